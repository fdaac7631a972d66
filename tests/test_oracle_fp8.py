"""Pins of the oracle's fused transform + FP8 (e4m3) quantization.

The e4m3 encoder and decoder are pinned against torch's float8_e4m3fn
conversion (a library routine); the quantizer against hand-derived fixtures
and the properties that round-to-nearest-even at the per-row maximum scale
guarantees.
"""
from __future__ import annotations

import json
from pathlib import Path

import numpy as np
import pytest
import torch

from paper_2412_08832_amd import workloads as W

GOLDEN = Path(__file__).resolve().parent / "golden" / "fwht_fp8_small.json"


def _torch_e4m3(values: np.ndarray) -> np.ndarray:
    return torch.from_numpy(np.asarray(values, dtype=np.float32)).to(torch.float8_e4m3fn) \
        .view(torch.uint8).numpy()


def _all_e4m3_values() -> np.ndarray:
    v = torch.from_numpy(np.arange(256, dtype=np.uint8)).view(torch.float8_e4m3fn).float().numpy()
    return np.sort(np.unique(v[np.isfinite(v)])).astype(np.float64)


def spacing_e4m3(a: np.ndarray) -> np.ndarray:
    """Distance between neighbouring e4m3 values around |a| (subnormal spacing below 2^-6)."""
    a = np.abs(np.asarray(a, dtype=np.float64))
    with np.errstate(divide="ignore"):
        e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    return np.where(a < 2.0 ** -6, 2.0 ** -9, np.exp2(e - 3))


def test_decode_e4m3_every_code(oracle):
    codes = np.arange(256, dtype=np.uint8)
    got = oracle.decode_e4m3(codes)
    want = torch.from_numpy(codes).view(torch.float8_e4m3fn).float().numpy().astype(np.float64)
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], want[~nan])


def test_encode_e4m3_matches_torch(oracle):
    fin = _all_e4m3_values()
    mids = (fin[1:] + fin[:-1]) / 2
    m32 = mids.astype(np.float32)
    rng = np.random.default_rng(0)
    x = np.concatenate([
        fin, mids, np.nextafter(m32, np.float32(np.inf)), np.nextafter(m32, np.float32(-np.inf)),
        [448.0, 449.0, 463.99, 464.0, 464.01, 470.0, 1e4, 3e38, np.inf, np.nan, 0.0, 2.0 ** -10,
         2.0 ** -11, 1.5 * 2.0 ** -10, 0.75 * 2.0 ** -9],
        rng.standard_normal(20000) * 60, rng.uniform(-2 ** -6, 2 ** -6, 5000)]).astype(np.float32)
    x = np.concatenate([x, -x])
    got = oracle.encode_e4m3(x)
    want = _torch_e4m3(x)
    gv = oracle.decode_e4m3(got)
    wv = oracle.decode_e4m3(want)
    same = (got == want) | (np.isnan(gv) & np.isnan(wv))
    assert same.all(), x[~same][:10]


def test_hand_derived_fixtures(oracle):
    for c in json.loads(GOLDEN.read_text())["cases"]:
        bits = np.array(c["x"], dtype=np.float16).view(np.uint16)[None, :]
        codes, scales = oracle.fwht_fp8(bits, "fp16", c["scale"])
        assert list(codes[0]) == c["codes"], c
        assert scales[0] == np.float32(c["scale_out"]), (scales[0], c)


@pytest.mark.parametrize("dtype", ["fp16", "bf16"])
@pytest.mark.parametrize("k", [7, 10, 13])
def test_quantization_properties(oracle, dtype, k):
    n = 1 << k
    bits = W.random_rows(17, n, dtype, seed=k)
    s = W.default_scale(n)
    y = oracle.fwht(bits, dtype, s).astype(np.float32).astype(np.float64)
    codes, scales = oracle.fwht_fp8(bits, dtype, s)
    deq = oracle.decode_e4m3(codes)
    for i in range(bits.shape[0]):
        amax = np.abs(y[i]).max()
        # the largest element lands on +-448 exactly
        j = int(np.argmax(np.abs(y[i])))
        assert abs(deq[i, j]) == 448.0
        assert np.sign(deq[i, j]) == np.sign(y[i, j])
        # scale is amax / 448 within fp32 rounding
        assert abs(scales[i] - amax / 448.0) <= 2.0 ** -23 * amax / 448.0
        # round-to-nearest: |deq - v| <= half a step (plus fp32 slack), v = y / s
        v = y[i] * (448.0 / amax)
        assert np.all(np.abs(deq[i] - v) <= 0.5 * spacing_e4m3(v) + 2.0 ** -20 * np.abs(v) + 1e-30)


def test_special_rows(oracle):
    n = 128
    bits = W.random_rows(4, n, "bf16", seed=1)
    bits[0] = 0                      # zero row
    bits[1, 3] = 0x7FC0              # NaN -> the whole transformed row is NaN
    bits[2, 5] = 0x7F80              # +Inf -> every transformed value is +-Inf
    tiny = np.random.default_rng(5).integers(1, 0x7F, n).astype(np.uint16)
    bits = np.vstack([bits, tiny | (np.arange(n, dtype=np.uint16) % 2 << 15)])
    # row 4: bf16 subnormals; 448/amax overflows fp32, so the codes are all zero
    codes, scales = oracle.fwht_fp8(bits, "bf16", W.default_scale(n))
    amax4 = np.float32(np.abs(oracle.fwht(bits[4:5], "bf16", W.default_scale(n))
                              .astype(np.float32)).max())
    assert 0 < amax4 < np.float32(448.0) * np.float32(2.0 ** -128)
    assert scales[4] == amax4 / np.float32(448.0) and ((codes[4] & 0x7F) == 0).all()  # +-0
    assert scales[0] == 0 and (codes[0] == 0).all()
    assert np.isnan(scales[1]) and np.isnan(oracle.decode_e4m3(codes[1])).all()
    assert np.isinf(scales[2]) and np.isnan(oracle.decode_e4m3(codes[2])).all()
    assert np.isfinite(scales[3]) and np.isfinite(oracle.decode_e4m3(codes[3])).all()


def test_power_of_two_scale_equivariance(oracle):
    bits = W.random_rows(9, 512, "fp16", seed=3)
    c1, s1 = oracle.fwht_fp8(bits, "fp16", 0.0625)
    c2, s2 = oracle.fwht_fp8(bits, "fp16", 0.125)
    assert np.array_equal(c1, c2)
    assert np.array_equal(s2, 2 * s1)


def test_plain_row_quantizer_on_fixture_rows(oracle):
    """Without the transform the same quantizer maps the fixtures' y rows to their codes."""
    for c in json.loads(GOLDEN.read_text())["cases"]:
        codes, scales = oracle.quantize_fp8(np.array([c["y"]], dtype=np.float32))
        assert list(codes[0]) == c["codes"], c
        assert scales[0] == np.float32(c["scale_out"]), (scales[0], c)
