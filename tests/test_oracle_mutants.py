"""Plant plausible mistakes in copies of the CPU oracle and check the pins catch each.

Every mutant is built from a patched copy of ``oracle/tq_oracle.c`` in a temporary
directory (or is a Python subclass of the oracle); the committed oracle is untouched.
A mutant that no pin rejects would mean the pins leave that part of the oracle
unchecked.
"""
import os

import numpy as np
import pytest

import oracle as oracle_pkg
from oracle import build as obuild
from oracle_pins import PINS

SRC = open(obuild.SRC).read()

C_MUTANTS = {
    "fold_planes_transposed": ("c[i] = (int8_t)(3 * t1[i] + t2[i]);", "c[i] = (int8_t)(t1[i] + 3 * t2[i]);"),
    "unfold_off_by_one": ("int a = (v + 4) / 3 - 1;", "int a = (v + 3) / 3 - 1;"),
    "two_plane_alpha_swapped": ("w[i] = alpha1 * (double)t1[i] + alpha2 * (double)t2[i];", "w[i] = alpha2 * (double)t1[i] + alpha1 * (double)t2[i];"),
    "f16_exponent_bias": ("ldexp((double)(1024 + f), e - 25)", "ldexp((double)(1024 + f), e - 24)"),
    "f16_subnormal_scale": ("v = ldexp((double)f, -24);", "v = ldexp((double)f, -25);"),
    "f16_sign_dropped": ("    v = ldexp((double)(1024 + f), e - 25); /* (1 + f/1024) * 2^(e-15) */\n  }\n  return sign ? -v : v;",
                         "    v = ldexp((double)(1024 + f), e - 25); /* (1 + f/1024) * 2^(e-15) */\n  }\n  return v;"),
    "quant_round_half_away": ("float r = rintf(y);", "float r = roundf(y);"),
    "quant_scale_128": ("float inv = 127.0f / amax;", "float inv = 128.0f / amax;"),
    "quant_d_128": ("*d = amax / 127.0f;", "*d = amax / 128.0f;"),
    "quant_signed_max": ("float a = fabsf(x[i]);", "float a = x[i];"),
    "quant_bsum_sign": ("s += (int32_t)r;", "s -= (int32_t)r;"),
    "quant_truncate": ("float r = rintf(y);", "float r = truncf(y);"),
    "quant_block_stride": ("d + tt * nb + b,", "d + b,"),
    "quant_tiny_threshold": ("if (amax < 0x1p-100f) {", "if (amax == 0.0f) {"),
    "dot_int8_wrap": ("s += (int64_t)a[i] * (int64_t)b[i];", "s += (int8_t)(a[i] * b[i]);"),
    "gemv_token_index_dropped": ("q + tt * k + b * 256, 256)", "q + b * 256, 256)"),
    "gemv_row_index_dropped": ("orc_dot_i8(c + r * k + b * 256,", "orc_dot_i8(c + b * 256,"),
    "gemv_scale_transposed": ("orc_f16_to_f64(s[r * kb + b])", "orc_f16_to_f64(s[b * n + r])"),
    "gemv_act_scale_dropped": ("* (double)d[tt * kb + b] * (double)v;", "* (double)v;"),
    "gemv_block_offset": ("q + tt * k + b * 256, 256)", "q + tt * k + b * 255, 256)"),
    "gemv_absref_signed": ("(double)d[tt * kb + b] * (double)v;\n        acc += term;\n        aacc += fabs(term);",
                           "(double)d[tt * kb + b] * (double)v;\n        acc += term;\n        aacc += term;"),
    "synth_field_swap": ("int sh = (e & 1) ? 32 : 0;", "int sh = (e & 1) ? 0 : 32;"),
    "synth_trit_shift": ("((f * 3u) >> 16) - 1", "((f * 3u) >> 15) - 1"),
    "synth_scale_counter": ("sm64_word(key, (uint64_t)(n * k / 2) + j)", "sm64_word(key, j)"),
    "synth_gamma": ("z = key + (i + 1) * 0x9E3779B97F4A7C15ull;", "z = key + i * 0x9E3779B97F4A7C15ull;"),
    "f16_encode_truncates": ("double r = nearbyint(q);", "double r = trunc(q);"),
    "f16_no_saturation": ("if (v > 65504.0) v = 65504.0;", "if (v > 65536.0) v = 65536.0;"),
    "tied_start_amax_over_3": ("float s = amax / 4.0f;", "float s = amax / 3.0f;"),
    "tied_clamp_3": ("if (r > 4.0f) r = 4.0f;", "if (r > 3.0f) r = 3.0f;"),
    "tied_round_half_away": ("float r = nearbyintf(t);", "float r = roundf(t);"),
    "tied_no_scale_step": ("s = (float)(pairwise_sum256(v) / (double)cc);", "(void)pairwise_sum256(v);"),
    "tied_scale_over_count": ("s = (float)(pairwise_sum256(v) / (double)cc);", "s = (float)(pairwise_sum256(v) / 256.0);"),
    "tied_final_codes_fp32_scale": ("code_step(wb, sd, cb);", "code_step(wb, s, cb);"),
    "tied_no_zero_floor": ("if (!(amax >= 0x1p-100f)) {", "if (amax == 0.0f) {"),
    "e2m1_subnormal_step": ("double v = (e == 0) ? 0.5 * m : ldexp(1.0 + 0.5 * m, e - 1);", "double v = (e == 0) ? 1.0 * m : ldexp(1.0 + 0.5 * m, e - 1);"),
    "e2m1_exponent_bias": ("double v = (e == 0) ? 0.5 * m : ldexp(1.0 + 0.5 * m, e - 1);", "double v = (e == 0) ? 0.5 * m : ldexp(1.0 + 0.5 * m, e);"),
    "e2m1_doubled_shift": ("int v = (e == 0) ? m : (2 + m) << (e - 1);", "int v = (e == 0) ? m : (2 + m) << e;"),
    "e2m1_doubled_mantissa": ("int v = (e == 0) ? m : (2 + m) << (e - 1);", "int v = (e == 0) ? m : (2 + 2 * m) << (e - 1);"),
    "e2m1_doubled_unsigned": ("int v = (e == 0) ? m : (2 + m) << (e - 1);\n  return sign ? -v : v;", "int v = (e == 0) ? m : (2 + m) << (e - 1);\n  return sign ? v : v;"),
    "e8m0_bias": ("return e == 255 ? NAN : ldexp(1.0, (int)e - 127);", "return e == 255 ? NAN : ldexp(1.0, (int)e - 128);"),
    "mx_half_not_absorbed": ("ldexp(1.0, (int)e8[r * k32 + j] - 128)", "ldexp(1.0, (int)e8[r * k32 + j] - 127)"),
    "mx_scale_index": ("ldexp(1.0, (int)e8[r * k32 + j] - 128)", "ldexp(1.0, (int)e8[j] - 128)"),
    "mx_act_block_index": ("(double)d[tt * kb + j / 8]", "(double)d[tt * kb + j / 4]"),
    "mx_nan_scale_accepted": ("    if (e8[i] == 255) return ORC_BAD_INPUT;\n", ""),
    "mx_isum_token_dropped": ("(int64_t)q[tt * k + 32 * j + i];", "(int64_t)q[32 * j + i];"),
    "free_ls_sign": ("const double num1 = (double)sc * u - (double)sb * v;", "const double num1 = (double)sc * u + (double)sb * v;"),
    "free_ls_cross_terms": ("const double num2 = (double)sa * v - (double)sb * u;", "const double num2 = (double)sa * v - (double)sb * v;"),
    "free_no_scale_step": ("        if (det > 0) {\n          const double num1", "        if (det < 0) {\n          const double num1"),
    "free_no_final_plane_step": ("      free_plane_step(wb, (float)orc_f16_to_f64(ab[0]), (float)orc_f16_to_f64(ab[1]), p1, p2);\n", ""),
    "free_plane_error_signed": ("double e = fabs((double)w[i] - ((double)a1 * u1 + (double)a2 * u2));", "double e = (double)w[i] - ((double)a1 * u1 + (double)a2 * u2);"),
    "free_planes_swapped_in_fit": ("vv[i] = (double)wb[i] * (double)p2[i];", "vv[i] = (double)wb[i] * (double)p1[i];"),
    "free_zero_block_not_zero": ("        for (int i = 0; i < 256; ++i) p1[i] = p2[i] = 0;\n", ""),
    "gemv2_alpha2_from_alpha1": ("orc_f16_to_f64(a[(r * kb + b) * 2 + 1])", "orc_f16_to_f64(a[(r * kb + b) * 2 + 0])"),
    "gemv2_scale_stride": ("orc_f16_to_f64(a[(r * kb + b) * 2 + 0])", "orc_f16_to_f64(a[(r * kb + b) + 0])"),
    "gemv2_plane2_dropped": ("        acc += term2;\n", ""),
    "gemv2_plane2_reads_plane1": ("orc_dot_i8(t2 + r * k + b * 256, qb, 256)", "orc_dot_i8(t1 + r * k + b * 256, qb, 256)"),
    "gemv2_isum_planes_swapped": ("isum[((tt * n + r) * kb + b) * 2 + 0] = (int32_t)v1;", "isum[((tt * n + r) * kb + b) * 2 + 0] = (int32_t)v2;"),
    "gemv2_absref_plane1_only": ("aacc += fabs(term1) + fabs(term2);", "aacc += fabs(term1);"),
    "gemv2_token_index_dropped": ("const int8_t* qb = q + tt * k + b * 256;", "const int8_t* qb = q + b * 256;"),
    "gemv2_act_scale_dropped": ("double db = (double)d[tt * kb + b];", "double db = 1.0;"),
    "gemv2_trit_range_unchecked": ("if (t1[i] < -1 || t1[i] > 1 || t2[i] < -1 || t2[i] > 1) return ORC_BAD_INPUT;\n  for (int64_t tt", "(void)0;\n  for (int64_t tt"),
}


def _first_failure(o):
    for p in PINS:
        try:
            p(o)
        except Exception as e:  # noqa: BLE001 - any failure kills the mutant
            return f"{p.__name__}: {type(e).__name__}"
    return None


@pytest.mark.parametrize("name", sorted(C_MUTANTS))
def test_c_mutant_is_caught(name, tmp_path):
    old, new = C_MUTANTS[name]
    assert SRC.count(old) == 1, f"mutation anchor for {name} not unique"
    src = tmp_path / "mut.c"
    src.write_text(SRC.replace(old, new))
    lib = obuild.build(str(src), str(tmp_path / "libmut.so"), werror=False)
    killed = _first_failure(oracle_pkg.Oracle(lib))
    assert killed is not None, f"mutant {name} survived every pin"


class _SwapGateUp(oracle_pkg.Oracle):
    def expert_slot(self, ex, x_row):
        return super().expert_slot({"gate": ex["up"], "up": ex["gate"], "down": ex["down"]}, x_row)


class _SiluSign(oracle_pkg.Oracle):
    @staticmethod
    def silu(z):
        z = np.asarray(z, dtype=np.float64)
        return z / (1.0 + np.exp(z))


class _FirstWeightOnly(oracle_pkg.Oracle):
    def moe(self, x, idx, w, get_expert, tokens=None):
        w = np.repeat(np.asarray(w)[:, :1], w.shape[1], axis=1)
        return super().moe(x, idx, w, get_expert, tokens)


@pytest.mark.parametrize("cls", [_SwapGateUp, _SiluSign, _FirstWeightOnly], ids=lambda c: c.__name__)
def test_python_mutant_is_caught(cls):
    assert _first_failure(cls(oracle_pkg.oracle.DEFAULT_LIB)) is not None
