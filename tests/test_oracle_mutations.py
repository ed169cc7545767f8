"""Mutation check of the oracle pins (CPU only).

Each case plants one plausible mistake in a temporary copy of the oracle's C
source (a dropped term, a wrong sign, index or constant), compiles it, binds
the oracle front end to that copy and runs the pins of tests/test_oracle_pins.
The pins are only trustworthy if every planted mistake makes at least one of
them fail.  The committed oracle is never modified.
"""
import os
import subprocess

import pytest

import oracle
from oracle import build as oracle_build

from . import test_oracle_pins as pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "sq_oracle.c")

# (name, original text, planted text)
MUTATIONS = [
    ("philox multiplier", "(uint64_t)0xD2511F53u * x0", "(uint64_t)0xD2511F55u * x0"),
    ("philox key bump", "k1 += 0xBB67AE85u;", "k1 += 0xBB67AE84u;"),
    ("philox word select", "return (w[(idx >> 1) & 3u] >> (16u * (uint32_t)(idx & 1u))) & 0xFFFFu;",
     "return (w[(idx >> 1) & 3u] >> (16u * (uint32_t)((idx + 1) & 1u))) & 0xFFFFu;"),
    ("SR threshold width", "const float two16 = pow2f(16);", "const float two16 = pow2f(15);"),
    ("abs mask", "uint32_t a = f2u(x[m * ld + c]) & 0x7FFFFFFFu;", "uint32_t a = f2u(x[m * ld + c]);"),
    ("threshold index", "float tau_next = r_max * pow2f(-(g + 1));", "float tau_next = r_max * pow2f(-g);"),
    ("threshold closedness", "if (r_c > tau_next) return g;", "if (r_c >= tau_next) return g;"),
    ("Q off by one", "return (1 << (bits - 1)) - 1;", "return (1 << (bits - 1));"),
    ("group scale sign", "float s_c = scale->inv0 * pow2f(g[c]);", "float s_c = scale->inv0 * pow2f(-(int)g[c]);"),
    ("dropped group scale", "float s_c = scale->inv0 * pow2f(g[c]);", "float s_c = scale->inv0;"),
    ("truncation instead of rounding", "qf = rintf(v);", "qf = truncf(v);"),
    ("round half away", "qf = rintf(v);", "qf = roundf(v);"),
    ("SR comparison direction", "qf = ((float)u < f * two16) ? l + 1.0f : l;",
     "qf = ((float)u > f * two16) ? l + 1.0f : l;"),
    ("SR uses ceil", "float l = floorf(v);", "float l = ceilf(v);"),
    ("zero threshold", "else if (r_max < pow2f(-96)) scale->flags = SQO_FLAG_ZERO;",
     "else if (r_max <= pow2f(-96)) scale->flags = SQO_FLAG_ZERO;"),
    ("per-tensor scale", "scale->inv0 = (float)Q / a;", "scale->inv0 = (float)(Q + 1) / a;"),
    ("dgrad shift direction", "int shift = num_groups - 1 - (int)g[c];", "int shift = (int)g[c];"),
    ("dgrad dropped shift", "acc += prod * ((int64_t)1 << shift);", "acc += prod;"),
    ("wgrad channel index", "acc += (int64_t)q[m * C_out + c] * (int64_t)xq[m * C_in + k];",
     "acc += (int64_t)q[m * C_out + (C_out - 1 - c)] * (int64_t)xq[m * C_in + k];"),
    ("dgrad dequant exponent", "float alpha = (d_grad * d_w) * pow2f(-(num_groups - 1));",
     "float alpha = (d_grad * d_w) * pow2f(-num_groups);"),
    ("wgrad dequant sign", "float beta = (d_grad * d_x) * pow2f(-(int)g_rows[i]);",
     "float beta = (d_grad * d_x) * pow2f((int)g_rows[i]);"),
    ("conv output row of a tap", "int64_t oh = ih + PH - r;", "int64_t oh = ih - PH + r;"),
    ("conv tap order in the im2col column", "int64_t col = ((int64_t)r * KW + s) * C_in + ci;",
     "int64_t col = ((int64_t)s * KH + r) * C_in + ci;"),
    ("conv last output row dropped", "if (oh < 0 || oh >= Ho) continue;", "if (oh < 0 || oh >= Ho - 1) continue;"),
    ("conv dropped shift", "acc += ((int64_t)1 << shift) * prod;", "acc += prod;"),
    ("per-channel axis", "float x = axis == 0 ? T[ch * ld + e] : T[e * ld + ch];",
     "float x = axis == 1 ? T[ch * ld + e] : T[e * ld + ch];"),
    ("column dequant exponent", "float gamma = (d_a * d_w[k]) * pow2f(-(num_groups - 1));",
     "float gamma = (d_a * d_w[k]) * pow2f(-num_groups);"),
    ("int32 range check", "            if (acc > INT32_MAX || acc < INT32_MIN) {\n#pragma omp atomic write\n"
                          "                err = SQO_ERR_RANGE;\n            }\n            A[i * C_in + k]",
     "            A[i * C_in + k]"),
    ("L1BN mean truncated", "int64_t mc = div_round_even(S, M);", "int64_t mc = S / M;"),
    ("L1BN mean ties away", "if (2 * r > den || (2 * r == den && (q & 1))) q += 1;", "if (2 * r >= den) q += 1;"),
    ("L1BN sigma code floor", "if (k < 1) k = 1;", "if (k < 0) k = 0;"),
    ("L1BN kappa count", "double num = (double)gamma_q[c] * (127.0 * (double)M);",
     "double num = (double)gamma_q[c] * (127.0 * (double)(M - 1));"),
    ("L1BN sign-mean term", "e = (float)(lambda * (D * sbar - gbar));", "e = (float)(lambda * (-gbar));"),
    ("L1BN sign term sign", "b = (float)(-(lambda * D));", "b = (float)(lambda * D);"),
    ("L1BN dgamma xhat scale", "const double dg = (delta * (double)G2) * rho;", "const double dg = delta * (double)G2;"),
    ("L1BN lambda step", "const double lambda = ((double)gamma_q[c] * rho) / (double)x_step;",
     "const double lambda = ((double)gamma_q[c] * rho) * (double)x_step;"),
    ("L1BN sign of deviation", "float s = (float)((d > 0) - (d < 0));", "float s = (float)((d < 0) - (d > 0));"),
    ("conv wgrad input row of a tap", "int64_t ih = oh + r - PH;", "int64_t ih = oh - r + PH;"),
    ("conv wgrad tap order", "B[co * cols + ((int64_t)r * KW + s) * C_in + ci] = (int32_t)acc;",
     "B[co * cols + ((int64_t)s * KH + r) * C_in + ci] = (int32_t)acc;"),
    ("conv wgrad last column dropped", "if (iw < 0 || iw >= W) continue;\n                                acc",
     "if (iw < 0 || iw >= W - 1) continue;\n                                acc"),
]


def _pin_calls():
    """Every pin with fixed arguments (covering the parametrised ones)."""
    calls = [
        pins.test_philox_known_answers,
        pins.test_sr_uniform_is_uniform_and_keyed,
        pins.test_channel_range_matches_numpy,
        pins.test_grouping_hand_table,
        lambda: pins.test_grouping_closed_form_random(4),
        lambda: pins.test_grouping_boundaries_exact(4),
        pins.test_scale_invariance_power_of_two,
        pins.test_round_half_to_even_ties,
        pins.test_stochastic_rounding_unbiased_and_variance,
        pins.test_stochastic_rounding_reproducible,
        pins.test_flags_zero_tiny_nonfinite,
        pins.test_wgrad_equals_int64_matmul_and_dequantized_product,
        pins.test_gemm_brute_force_tiny,
        pins.test_int32_range_is_enforced,
        pins.test_dequant_wgrad_row_scale_direction,
        pins.test_full_small_workload_consistency,
    ]
    for bits in (2, 4, 8):
        for ng in (1, 4):
            for mode in (0, 1):
                calls.append(lambda b=bits, n=ng, m=mode: pins.test_codes_in_range_and_top_maps_to_Q(b, n, m))
    for bits, ng in [(4, 4), (8, 3)]:
        calls.append(lambda b=bits, n=ng: pins.test_rtn_half_step_error_bound(b, n))
    for bits in (4, 8):
        calls.append(lambda b=bits: pins.test_single_group_is_per_tensor_symmetric(b))
    for bits, ng in [(4, 4), (6, 4)]:
        calls.append(lambda b=bits, n=ng: pins.test_dgrad_equals_shifted_matmul_and_group_gemms(b, n))
        calls.append(lambda b=bits, n=ng: pins.test_dgrad_dequant_equals_dequantized_product(b, n))
    calls.append(lambda: pins.test_shiftquant_variance_bound(4))
    for case in pins.CONV_CASES:
        calls.append(lambda c=case: pins.test_conv_dgrad_is_transpose_of_forward_conv(c))
    calls.append(pins.test_conv_dgrad_1x1_is_dgrad_and_brute_force)
    for axis in (0, 1):
        calls.append(lambda a=axis: pins.test_quantize_channels_is_per_tensor_per_channel(a, 8))
    calls.append(pins.test_quantize_channels_degenerate_channels)
    calls.append(lambda: pins.test_forward_equals_dequantized_product(4, 4))
    for case in pins.CONV_CASES[:4]:
        calls.append(lambda c=case: pins.test_conv_wgrad_is_adjoint_of_forward_conv(c))
    calls.append(pins.test_conv_wgrad_equals_wgrad_of_im2col)
    calls.append(pins.test_l1bn_forward_matches_textbook_when_statistics_are_exact)
    calls.append(pins.test_l1bn_forward_statistics_bounds_random)
    calls.append(lambda: pins.test_l1bn_backward_matches_autograd_when_statistics_are_exact(8, 4, 0))
    calls.append(pins.test_l1bn_backward_is_shift_invariant_random)
    calls.append(pins.test_l1bn_constant_channels)
    return calls


def _some_pin_fails() -> bool:
    for call in _pin_calls():
        try:
            call()
        except (Exception, pytest.fail.Exception):   # assertion, RangeError, pytest.raises
            return True
    return False


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_planted_mistake_is_caught(name, old, new, tmp_path):
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor for '{name}' not unique in sq_oracle.c"
    mutated = tmp_path / "sq_oracle_mut.c"
    mutated.write_text(src.replace(old, new))
    so = tmp_path / "liboracle_mut.so"
    subprocess.run(["gcc", *oracle_build.CFLAGS, "-w", str(mutated), "-o", str(so), "-lm"], check=True)
    prev = oracle.oracle.use_library(str(so))
    try:
        caught = _some_pin_fails()
    finally:
        oracle.oracle.restore_library(prev)
    assert caught, f"no pin catches the planted mistake '{name}'"


def test_unmutated_oracle_passes_all_pins():
    for call in _pin_calls():
        call()
