"""Seeded input generators: determinism, rounding, and workload structure."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from paper_2412_08832_amd import workloads as W


def test_same_seed_same_bytes():
    a = W.random_rows(33, 256, "bf16", seed=7)
    b = W.random_rows(33, 256, "bf16", seed=7)
    assert a.tobytes() == b.tobytes()
    assert a.tobytes() != W.random_rows(33, 256, "bf16", seed=8).tobytes()


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    vals = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 1e3,
                           np.array([0.0, -0.0, 1.0 + 2**-8, 1.0 + 3 * 2**-8, 3.4e38, 1e-40],
                                    dtype=np.float32)])
    ours = W.round_to_bits(vals, "bf16")
    ref = torch.from_numpy(vals).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_fp16_rounding_is_numpy_rne():
    vals = np.array([1.0 + 2**-11, 1.0 + 3 * 2**-11, 65519.0, 65520.0], dtype=np.float32)
    bits = W.round_to_bits(vals, "fp16")
    assert list(bits.view(np.float16).astype(np.float64)) == [1.0, 1.0 + 2**-9, 65504.0, np.inf]


def test_truncated_draw_is_prefix_of_full_draw():
    for w in (W.WORKLOADS["fp16_1024x256"], W.WORKLOADS["fp16_16384x4096"], W.sweep_point(12, "bf16", True)):
        small = W.generate(w, rows=5)
        # the full recipe at a reduced row count must start with the same rows
        bigger = W.generate(w, rows=9)
        assert np.array_equal(small, bigger[:5])


def test_outlier_workloads():
    w2 = W.WORKLOADS["bf16_1048576x128_inplace"]
    assert (w2.m, w2.n, w2.inplace) == (1 << 20, 128, True)
    x3 = W.generate(W.WORKLOADS["fp16_16384x4096"], rows=64).view(np.float16).astype(np.float64)
    cols = W.hidden_outlier_columns()
    assert len(cols) == 16
    big = np.abs(x3[:, cols]).mean()
    rest = np.abs(np.delete(x3, cols, axis=1)).mean()
    assert 30 < big / rest < 70


def test_default_scale_is_fp32_rounded():
    for k in range(7, 16):
        n = 1 << k
        s = W.default_scale(n)
        assert s == float(np.float32(s))
        assert abs(s * np.sqrt(n) - 1.0) < 1e-7


def test_strided_canary_fill():
    bits = W.random_rows(4, 128, "fp16", seed=1, stride=136, fill_bits=0xBEEF)
    assert bits.shape == (4, 136)
    assert (bits[:, 128:] == 0xBEEF).all()


def test_small_sweep_points():
    for k in range(0, 7):
        w = W.sweep_point(k, "bf16", False)
        assert (w.m, w.n) == (1 << (28 - k), 1 << k)
        head = W.generate(w, rows=16)
        assert head.shape == (16, 1 << k) and np.array_equal(head, W.generate(w, rows=16))
    assert W.sweep_point(20, "fp16", True).m == 256
    with pytest.raises(ValueError):
        W.sweep_point(21, "fp16", True)
