"""Rotation versus quantization error on the outlier workloads (synthetic study).

The transform exists to spread outliers before low-precision quantization
(Sec. 1; rotations precede FP8 attention in Sec. 4.2).  This measures that on
the two synthetic outlier workloads, standing in for the paper's Llama
activations: per-row FP8 (e4m3) and symmetric INT8 quantization error of the
inputs themselves ("plain"), against that of the rotated inputs, rotated back
exactly before comparing ("rotated").  y = s H x, so x = H y / (n s); the
normalized rotation is orthogonal and leaves the squared error unchanged.

Findings the CPU tests pin (oracle only):
  * INT8: the rotation raises the signal-to-quantization-noise ratio by more
    than 10 dB on both workloads (one uniform step per row is set by the
    largest element, and the rotation shrinks it).
  * FP8 e4m3: the rotation lowers the worst-case error, but not the mean
    squared error -- e4m3 keeps a relative precision per element, and
    spreading a sparse outlier over the row gives every element a large
    absolute error.
The GPU tests check that the fused GPU kernels' codes give the oracle's
errors, and print the table.
"""
from __future__ import annotations

import numpy as np
import pytest

from paper_2412_08832_amd import workloads as W

SAMPLES = {"bf16_1048576x128_inplace": 4096, "fp16_16384x4096": 256}


def _inputs(oracle, name):
    w = W.WORKLOADS[name]
    bits = W.generate(w, rows=SAMPLES[name])
    return w, bits, oracle.decode(bits, w.dtype)


def _dequant(oracle, fmt, codes, scales):
    q = oracle.decode_e4m3(codes) if fmt == "fp8" else codes.astype(np.float64)
    return q * scales.astype(np.float64)[:, None]


def _plain(oracle, fmt, x):
    quant = oracle.quantize_fp8 if fmt == "fp8" else oracle.quantize_int8
    return _dequant(oracle, fmt, *quant(x.astype(np.float32)))


def _rotated_back(oracle, fmt, codes, scales, n, scale):
    return oracle.fwht_vec(_dequant(oracle, fmt, codes, scales)) / (n * float(scale))


def error_stats(x: np.ndarray, xhat: np.ndarray) -> dict:
    e = xhat - x
    se, sx = float(np.sum(e * e)), float(np.sum(x * x))
    return {"rel_mse": se / sx, "max_abs": float(np.abs(e).max()),
            "sqnr_db": 10.0 * np.log10(sx / se)}


def study_row(oracle, name, fmt):
    """Plain and rotated error of the oracle's quantizers on one workload sample."""
    w, bits, x = _inputs(oracle, name)
    fused = oracle.fwht_fp8 if fmt == "fp8" else oracle.fwht_int8
    codes, scales = fused(bits, w.dtype, w.scale)
    return (error_stats(x, _plain(oracle, fmt, x)),
            error_stats(x, _rotated_back(oracle, fmt, codes, scales, w.n, w.scale)))


@pytest.mark.parametrize("name", sorted(SAMPLES))
def test_rotation_helps_int8(oracle, name):
    plain, rot = study_row(oracle, name, "int8")
    assert rot["sqnr_db"] > plain["sqnr_db"] + 10.0, (plain, rot)
    assert rot["max_abs"] < plain["max_abs"], (plain, rot)


@pytest.mark.parametrize("name", sorted(SAMPLES))
def test_rotation_and_fp8(oracle, name):
    plain, rot = study_row(oracle, name, "fp8")
    assert rot["max_abs"] < plain["max_abs"] / 1.5, (plain, rot)
    assert rot["rel_mse"] > plain["rel_mse"], (plain, rot)


def test_rotating_back_is_exact_without_quantization(oracle):
    """The inverse used above undoes the transform to fp64 rounding."""
    w, bits, x = _inputs(oracle, "fp16_16384x4096")
    y = oracle.fwht(bits[:8], w.dtype, w.scale)
    back = oracle.fwht_vec(y) / (w.n * float(w.scale))
    assert np.allclose(back, x[:8], rtol=0, atol=1e-12 * np.abs(x[:8]).max())


@pytest.mark.gpu
@pytest.mark.parametrize("fmt", ["fp8", "int8"])
@pytest.mark.parametrize("name", sorted(SAMPLES))
def test_gpu_rotation_study(oracle, name, fmt):
    """The GPU's fused codes give the oracle's errors; prints one row of the table."""
    import torch
    from gpu_util import say, to_device
    from paper_2412_08832_amd import hadacore as H
    w, bits, x = _inputs(oracle, name)
    m, n = bits.shape
    dev = to_device(bits, w.dtype)
    code = H.FP16 if w.dtype == "fp16" else H.BF16
    codes = torch.empty((m, n), dtype=torch.uint8 if fmt == "fp8" else torch.int8, device="cuda")
    scales = torch.empty((m,), dtype=torch.float32, device="cuda")
    entry = H.hadamard_transform_fp8 if fmt == "fp8" else H.hadamard_transform_int8
    entry(dev.data_ptr(), n, codes.data_ptr(), n, scales.data_ptr(), m, n, code, w.scale,
          torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    gpu = error_stats(x, _rotated_back(oracle, fmt, codes.cpu().numpy(), scales.cpu().numpy(),
                                       n, w.scale))
    plain, rot = study_row(oracle, name, fmt)
    say(f"study {name} {fmt}: plain sqnr={plain['sqnr_db']:.2f} dB max={plain['max_abs']:.4g} | "
        f"rotated (oracle) sqnr={rot['sqnr_db']:.2f} dB max={rot['max_abs']:.4g} | "
        f"rotated (GPU) sqnr={gpu['sqnr_db']:.2f} dB max={gpu['max_abs']:.4g}")
    assert abs(gpu["rel_mse"] / rot["rel_mse"] - 1.0) < 0.01, (gpu, rot)
    assert abs(gpu["max_abs"] / rot["max_abs"] - 1.0) < 0.05, (gpu, rot)
