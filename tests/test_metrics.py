"""The comparison metric: ulp spacing and the tolerance reading."""
from __future__ import annotations

import numpy as np
import pytest

from metrics import bits_to_f64, compare, ulp


def test_ulp_hand_picked_values():
    assert ulp(np.array([1.0]), "fp16")[0] == 2.0**-10
    assert ulp(np.array([1.5]), "fp16")[0] == 2.0**-10
    assert ulp(np.array([65504.0]), "fp16")[0] == 32.0
    assert ulp(np.array([2.0**-14]), "fp16")[0] == 2.0**-24      # smallest normal
    assert ulp(np.array([2.0**-20]), "fp16")[0] == 2.0**-24      # subnormal range
    assert ulp(np.array([0.0]), "fp16")[0] == 2.0**-24
    assert ulp(np.array([1.0]), "bf16")[0] == 2.0**-7
    assert ulp(np.array([-3.0]), "bf16")[0] == 2.0**-6
    assert ulp(np.array([2.0**-126]), "bf16")[0] == 2.0**-133
    assert ulp(np.array([2.0**-130]), "bf16")[0] == 2.0**-133


def test_bits_to_f64():
    assert bits_to_f64(np.array([0x3C00], np.uint16), "fp16")[0] == 1.0
    assert bits_to_f64(np.array([0x3F80], np.uint16), "bf16")[0] == 1.0
    assert bits_to_f64(np.array([0xC000], np.uint16), "bf16")[0] == -2.0


def test_compare_exact_and_off_by_ulps():
    rng = np.random.default_rng(0)
    ref = rng.standard_normal((8, 256))
    rounded = ref.astype(np.float16).astype(np.float64)
    c = compare(rounded, ref, "fp16")
    assert c.ok and c.max_ulp_floored <= 0.5 + 1e-12
    bumped = rounded + 5 * ulp(rounded, "fp16")
    assert not compare(bumped, ref, "fp16").ok


def test_compare_nonfinite_classes():
    ref = np.array([[np.nan, np.inf, -np.inf, 1.0]])
    assert compare(np.array([[np.nan, np.inf, -np.inf, 1.0]]), ref, "bf16").ok
    assert not compare(np.array([[0.0, np.inf, -np.inf, 1.0]]), ref, "bf16").ok
    assert not compare(np.array([[np.nan, -np.inf, -np.inf, 1.0]]), ref, "bf16").ok
    assert not compare(np.array([[np.nan, np.inf, -np.inf, np.inf]]), ref, "bf16").ok


def test_compare_zero_rows_need_exact_zeros():
    ref = np.zeros((2, 16))
    assert compare(np.zeros((2, 16)), ref, "fp16").ok
    bad = np.zeros((2, 16))
    bad[1, 3] = 2.0**-24
    assert not compare(bad, ref, "fp16").ok


def test_floor_rejects_a_16bit_intermediate_rounding():
    """One rounding of the intermediate to 16 bits mid-transform must fail the floored-ulp clause."""
    from scipy.linalg import hadamard
    rng = np.random.default_rng(1)
    n = 1024
    x = rng.standard_normal((16, n)).astype(np.float16).astype(np.float64)
    H = hadamard(n).astype(np.float64)
    ref = x @ H / np.sqrt(n)
    # half the stages, round to fp16, the other half (H_n = H_32 (x) H_32)
    h32 = hadamard(32).astype(np.float64)
    half = np.stack([(r.reshape(32, 32) @ h32.T).reshape(-1) for r in x]) / np.sqrt(32)
    half = half.astype(np.float16).astype(np.float64)
    full = np.stack([(h32 @ r.reshape(32, 32)).reshape(-1) for r in half]) / np.sqrt(32)
    out = full.astype(np.float16).astype(np.float64)
    c = compare(out, ref, "fp16")
    assert c.rel_l2 <= 1e-3          # the L2 clause alone would accept it
    assert c.max_ulp_floored > 4.0   # the floored ulp clause does not


def test_ulp_reads_the_exponent_exactly():
    """Just below a power of two the spacing is that of the binade below (no
    rounding of a logarithm); zero and fp64 subnormals take the subnormal spacing."""
    below = np.nextafter(2.0, 0.0)
    assert ulp(np.array([below]), "fp16")[0] == 2.0**-10
    assert ulp(np.array([2.0]), "fp16")[0] == 2.0**-9
    assert ulp(np.array([5e-324, -0.0]), "bf16").tolist() == [2.0**-133] * 2


def test_blocked_comparison_equals_one_block():
    """Statistics merged over row blocks (any block size, any thread count) equal
    those of one comparison of the whole matrix."""
    from metrics import Accumulator
    rng = np.random.default_rng(3)
    ref = rng.standard_normal((40, 64)) * np.exp2(rng.integers(-30, 30, (40, 1)))
    ref[5] = 0.0
    gpu = ref.astype(np.float16).astype(np.float64)
    gpu[7, 3] += 3 * ulp(gpu[7:8, 3], "fp16")[0]
    ref[9, 1] = np.nan
    gpu[9, 1] = np.nan
    whole = compare(gpu, ref, "fp16")
    acc = Accumulator("fp16")
    for r0 in range(0, 40, 7):
        acc.merge(Accumulator("fp16").add(gpu[r0:r0 + 7], ref[r0:r0 + 7]))
    parts = acc.result()
    for f in ("count", "max_ulp_floored", "max_ulp_unfloored", "n_above_4ulp_unfloored",
              "nonfinite_mismatch", "zero_row_mismatch"):
        assert getattr(parts, f) == getattr(whole, f), f
    assert parts.rel_l2 == pytest.approx(whole.rel_l2, rel=1e-12)
