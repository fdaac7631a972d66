"""The oracle's pins must catch plausible mistakes in the oracle itself.

Each case copies ``oracle/fwht_oracle.c``, plants one mistake (a flipped
butterfly sign, a dropped stage, a wrong pair index, an off-by-one exponent
bias, a missing scale, an ignored stride, a wrong FP8 or INT8 rounding rule
or scale constant ...), compiles the copy on the CPU
into a temporary library and runs the pin battery of ``test_oracle.py``
against it.  At least one pin must fail for every mutant.  The real oracle
source is never modified.
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle as oracle_pkg
import test_oracle as T
import test_oracle_fp8 as F
import test_oracle_int8 as I

MUTANTS = [
    ("butterfly_sign", "v[j + h] = a - b;", "v[j + h] = b - a;"),
    ("butterfly_sum_dropped_term", "v[j] = a + b;", "v[j] = a;"),
    ("first_stage_dropped", "for (int64_t h = 1; h < n; h *= 2)", "for (int64_t h = 2; h < n; h *= 2)"),
    ("last_stage_dropped", "for (int64_t h = 1; h < n; h *= 2)", "for (int64_t h = 1; 2 * h < n; h *= 2)"),
    ("block_step_wrong", "for (int64_t i = 0; i < n; i += 2 * h)", "for (int64_t i = 0; i + h < n; i += h)"),
    ("partner_index_wrong", "double b = v[j + h];", "double b = v[(j + h) ^ 1];"),
    ("fp16_exponent_bias", "expo - 25", "expo - 24"),
    ("fp16_subnormal_scale", "ldexp((double)frac, -24)", "ldexp((double)frac, -23)"),
    ("fp16_implicit_bit", "(1024 + frac)", "(frac)"),
    ("bf16_exponent_bias", "expo - 134", "expo - 133"),
    ("bf16_fraction_width", "(128 + frac)", "(256 + frac)"),
    ("scale_missing", "row[k] *= jb->scale;", "row[k] *= 1.0;"),
    ("stride_ignored", "const uint16_t *src = jb->in + i * jb->in_stride;",
     "const uint16_t *src = jb->in + i * jb->n;"),
    ("direct_sign_parity", "(uint64_t)(cols[t] & k)", "(uint64_t)(cols[t] | k)"),
    ("direct_scale_missing", "out[t] = acc * scale;", "out[t] = acc;"),
    ("thread_remainder_rows_dropped", "jobs[t].row1 = m * (t + 1) / nthreads;",
     "jobs[t].row1 = m * t / nthreads + m / nthreads;"),
    # fused FP8 quantization
    ("e4m3_ties_away", "if (r > 0.5 || (r == 0.5 && fmod(kf, 2.0) != 0.0)) kf += 1.0;",
     "if (r >= 0.5) kf += 1.0;"),
    ("e4m3_exponent_bias", "int biased = (e - 1) + 7;", "int biased = (e - 1) + 8;"),
    ("e4m3_overflow_threshold", "a > 464.0", "a > 448.0"),
    ("e4m3_subnormal_spacing", "spacing = ldexp(1.0, -9);", "spacing = ldexp(1.0, -10);"),
    ("e4m3_decode_bias", "expo - 10", "expo - 11"),
    ("fp8_scale_constant", "const float s = amax / 448.0f;", "const float s = amax / 480.0f;"),
    ("fp8_multiplier_guard", "const float inv = isfinite(q) ? q : 0.0f;", "const float inv = q;"),
    ("amax_without_abs", "amax = max_ignoring_nan(amax, fabsf(y[k]));",
     "amax = max_ignoring_nan(amax, y[k]);"),
    # fused INT8 quantization
    ("int8_ties_away", "if (r > 0.5 || (r == 0.5 && fmod(f, 2.0) != 0.0)) f += 1.0;",
     "if (r >= 0.5) f += 1.0;"),
    ("int8_truncation", "double f = floor((double)v);", "double f = trunc((double)v);"),
    ("int8_saturation", "if (f > 127.0) f = 127.0;", "if (f > 126.0) f = 126.0;"),
    ("int8_scale_constant", "*scale = amax / 127.0f;", "*scale = amax / 128.0f;"),
    ("int8_inv_constant", "const float q = 127.0f / amax;", "const float q = 128.0f / amax;"),
    ("int8_multiplier_overflow", "const int usable = isfinite(amax) && isfinite(q);",
     "const int usable = isfinite(amax) && amax > 0.0f;"),
    ("int8_nonfinite_rows", "usable ? oracle_encode_int8(y[k] * inv) : 0",
     "usable ? oracle_encode_int8(y[k] * inv) : 1"),
]


def _pins(o):
    """Callables that raise on failure; each is one pin of test_oracle.py."""
    return [
        lambda: T.test_decode_fp16_every_pattern(o),
        lambda: T.test_decode_bf16_every_pattern(o),
        lambda: T.test_matches_explicit_matrix_integers_exact(o, 4),
        lambda: T.test_matches_explicit_matrix_integers_exact(o, 9),
        lambda: T.test_matches_explicit_matrix_random(o, "bf16", 8),
        lambda: T.test_matches_explicit_matrix_random(o, "fp16", 7),
        lambda: T.test_matches_kronecker_factorisation(o, 8, 7),
        lambda: T.test_direct_definition_agrees_with_explicit_matrix(o),
        lambda: T.test_orthogonality_from_basis_vectors(o, 4),
        lambda: T.test_hand_derived_fixtures(o),
        lambda: T.test_strided_rows_ignore_gaps(o),
        lambda: T.test_scale_is_one_final_product(o),
        lambda: T.test_threads_do_not_change_results(o),
        lambda: F.test_decode_e4m3_every_code(o),
        lambda: F.test_encode_e4m3_matches_torch(o),
        lambda: F.test_hand_derived_fixtures(o),
        lambda: F.test_quantization_properties(o, "bf16", 10),
        lambda: F.test_special_rows(o),
        lambda: I.test_encode_int8_matches_numpy_rint(o),
        lambda: I.test_hand_derived_fixtures(o),
        lambda: I.test_quantization_properties(o, "fp16", 7),
        lambda: I.test_special_rows(o),
    ]


def test_pins_pass_on_the_real_oracle(oracle):
    for pin in _pins(oracle):
        pin()


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, name, old, new):
    src = oracle_pkg.SOURCE.read_text()
    assert old in src, f"mutation site for {name} not found in the oracle source"
    mutated = tmp_path / "fwht_oracle_mutant.c"
    mutated.write_text(src.replace(old, new, 1))
    lib = oracle_pkg.compile_library(mutated, tmp_path / "liboracle_mutant.so")
    o = oracle_pkg.Oracle(lib)
    failures = []
    with np.errstate(all="ignore"):
        for i, pin in enumerate(_pins(o)):
            try:
                pin()
            except (AssertionError, ValueError):
                failures.append(i)
    assert failures, f"mutant {name} passed every pin"
