"""Pins of the oracle's fused transform + symmetric per-row INT8 quantization.

The integer rounding is pinned against numpy's round-half-to-even (a library
routine); the quantizer against hand-derived fixtures and the properties that
round-half-to-even at the per-row maximum scale guarantees.
"""
from __future__ import annotations

import json
from pathlib import Path

import numpy as np
import pytest

from paper_2412_08832_amd import workloads as W

GOLDEN = Path(__file__).resolve().parent / "golden" / "fwht_int8_small.json"


def test_encode_int8_matches_numpy_rint(oracle):
    ties = np.arange(-128, 128) + 0.5
    t32 = ties.astype(np.float32)
    rng = np.random.default_rng(0)
    x = np.concatenate([
        ties, np.nextafter(t32, np.float32(np.inf)), np.nextafter(t32, np.float32(-np.inf)),
        np.arange(-127, 128), rng.uniform(-127.4, 127.4, 20000), rng.uniform(-2, 2, 5000),
        [0.0, -0.0, 127.49, -127.49, 128.0, 200.0, -1e9, 3e38],
    ]).astype(np.float32)
    got = oracle.encode_int8(x)
    want = np.clip(np.rint(x.astype(np.float64)), -127, 127).astype(np.int8)
    assert np.array_equal(got, want), x[got != want][:10]


def test_hand_derived_fixtures(oracle):
    for c in json.loads(GOLDEN.read_text())["cases"]:
        bits = np.array(c["x"], dtype=np.float16).view(np.uint16)[None, :]
        codes, scales = oracle.fwht_int8(bits, "fp16", c["scale"])
        assert list(codes[0]) == c["codes"], c
        assert scales[0] == np.float32(c["scale_out"]), (scales[0], c)


@pytest.mark.parametrize("dtype", ["fp16", "bf16"])
@pytest.mark.parametrize("k", [7, 10, 13])
def test_quantization_properties(oracle, dtype, k):
    n = 1 << k
    bits = W.random_rows(17, n, dtype, seed=k)
    s = W.default_scale(n)
    y = oracle.fwht(bits, dtype, s).astype(np.float32).astype(np.float64)
    codes, scales = oracle.fwht_int8(bits, dtype, s)
    q = codes.astype(np.float64)
    for i in range(bits.shape[0]):
        amax = np.abs(y[i]).max()
        j = int(np.argmax(np.abs(y[i])))
        # the largest element lands on +-127 with its sign
        assert q[i, j] == 127.0 * np.sign(y[i, j])
        assert abs(scales[i] - amax / 127.0) <= 2.0 ** -23 * amax / 127.0
        # round to nearest: |q - v| <= 1/2 (plus fp32 slack), v = y * 127 / amax
        v = y[i] * (127.0 / amax)
        assert np.all(np.abs(q[i] - v) <= 0.5 + 2.0 ** -16)
        # dequantized error within half a scale step
        assert np.all(np.abs(q[i] * scales[i] - y[i]) <= 0.5 * scales[i] * (1 + 2.0 ** -16))
    # negating the input negates every code
    neg = bits ^ np.uint16(0x8000)
    cn, sn = oracle.fwht_int8(neg, dtype, s)
    assert np.array_equal(cn, -codes) and np.array_equal(sn, scales)


def test_special_rows(oracle):
    n = 128
    bits = W.random_rows(4, n, "bf16", seed=1)
    bits[0] = 0                      # zero row
    bits[1, 3] = 0x7FC0              # NaN -> the whole transformed row is NaN
    bits[2, 5] = 0x7F80              # +Inf -> every transformed value is +-Inf
    tiny = np.random.default_rng(5).integers(1, 0x7F, n).astype(np.uint16)
    bits = np.vstack([bits, tiny | (np.arange(n, dtype=np.uint16) % 2 << 15)])
    # row 4: bf16 subnormals; 127/amax overflows fp32, so the codes are all zero
    codes, scales = oracle.fwht_int8(bits, "bf16", W.default_scale(n))
    amax4 = np.float32(np.abs(oracle.fwht(bits[4:5], "bf16", W.default_scale(n))
                              .astype(np.float32)).max())
    assert 0 < amax4 < np.float32(127.0) * np.float32(2.0 ** -128)
    assert scales[4] == amax4 / np.float32(127.0) and (codes[4] == 0).all()
    assert scales[0] == 0 and (codes[0] == 0).all()
    assert np.isnan(scales[1]) and (codes[1] == 0).all()
    assert np.isinf(scales[2]) and (codes[2] == 0).all()
    assert np.isfinite(scales[3]) and np.abs(codes[3]).max() == 127


def test_power_of_two_scale_equivariance(oracle):
    bits = W.random_rows(9, 512, "fp16", seed=3)
    c1, s1 = oracle.fwht_int8(bits, "fp16", 0.0625)
    c2, s2 = oracle.fwht_int8(bits, "fp16", 0.125)
    assert np.array_equal(c1, c2)
    assert np.array_equal(s2, 2 * s1)


def test_plain_row_quantizer_on_fixture_rows(oracle):
    """Without the transform the same quantizer maps the fixtures' y rows to their codes."""
    for c in json.loads(GOLDEN.read_text())["cases"]:
        codes, scales = oracle.quantize_int8(np.array([c["y"]], dtype=np.float32))
        assert list(codes[0]) == c["codes"], c
        assert scales[0] == np.float32(c["scale_out"]), (scales[0], c)
