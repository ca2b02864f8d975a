"""Seeded synthetic inputs shared by the CPU oracle and the HIP path (random draws only)."""
from .gen import *  # noqa: F401,F403
