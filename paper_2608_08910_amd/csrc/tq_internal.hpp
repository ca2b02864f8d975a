// Host-side internals shared by the library's translation units (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <cstdarg>
#include <string>

#include "../../include/tq.h"

namespace tq {

// Records a thread-local error message and returns `st`.
tq_status fail(tq_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();
tq_status check_launch(const char* what);

inline bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

constexpr int kMaxK = 16384;

// Internal launchers (arguments already validated).
hipError_t launch_quantize(const float* x, int64_t t, int32_t k, int8_t* q, float* d, int32_t* bsum,
                           hipStream_t st);

}  // namespace tq
