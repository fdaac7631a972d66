"""Seeded synthetic inputs for the batched Walsh-Hadamard transform.

This module holds no transform arithmetic.  It only draws seeded random
numbers (numpy PCG64), rounds them once to the 16-bit storage dtype with
round-to-nearest-even, and returns the raw uint16 bit patterns, so that the
GPU path and the CPU oracle consume the identical input.

The named workloads stand in for the paper's end-to-end use (rotations of
Llama-3.1 8B activations before FP8 attention, paper Sec. 4.2): head_dim 128
and hidden size 4096 shapes with outlier structure, plus the paper's size
range 2^7..2^15 at a fixed element count (Sec. 4.1 varies element count per
Hadamard size).
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

FP16 = "fp16"
BF16 = "bf16"


def round_to_bits(values: np.ndarray, dtype: str) -> np.ndarray:
    """Round float32 values to fp16/bf16 (round-to-nearest-even); return uint16 bits."""
    values = np.asarray(values, dtype=np.float32)
    if dtype == FP16:
        return values.astype(np.float16).view(np.uint16)
    if dtype == BF16:
        u = values.view(np.uint32)
        # round-to-nearest-even on the upper 16 bits of the fp32 pattern
        bias = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
        out = ((u + bias) >> np.uint32(16)).astype(np.uint16)
        nan = np.isnan(values)
        if nan.any():
            out[nan] = ((u[nan] >> np.uint32(16)) | np.uint32(0x40)).astype(np.uint16)
        return out
    raise ValueError(f"unknown dtype {dtype!r}")


def default_scale(n: int) -> float:
    """The normalized transform's scale 1/sqrt(n), computed in double and rounded to fp32."""
    return float(np.float32(1.0 / math.sqrt(n)))


def random_rows(m: int, n: int, dtype: str, seed: int, dist: str = "normal",
                stride: int | None = None, fill_bits: int = 0xDEAD) -> np.ndarray:
    """m rows of n seeded values, stored with row stride ``stride`` (>= n) elements.

    Gap elements between n and the stride are set to ``fill_bits`` (a canary).
    Returns a (m, stride) uint16 array.
    """
    rng = np.random.default_rng(seed)
    if dist == "normal":
        vals = rng.standard_normal((m, n), dtype=np.float32)
    elif dist == "uniform":
        vals = rng.uniform(-1.0, 1.0, (m, n)).astype(np.float32)
    elif dist == "integer":
        vals = rng.integers(-8, 9, (m, n)).astype(np.float32)
    else:
        raise ValueError(f"unknown distribution {dist!r}")
    bits = round_to_bits(vals, dtype)
    stride = n if stride is None else int(stride)
    if stride == n:
        return bits
    out = np.full((m, stride), fill_bits, dtype=np.uint16)
    out[:, :n] = bits
    return out


@dataclass(frozen=True)
class Workload:
    name: str
    dtype: str
    m: int
    n: int
    inplace: bool
    scale: float
    description: str


def _fp16_1024x256() -> Workload:
    return Workload("fp16_1024x256", FP16, 1024, 256, False, 1.0 / 16,
                    "fp16 1024x256, N(0,1) seed 0, out-of-place, scale 1/16")


def _bf16_1048576x128_inplace() -> Workload:
    return Workload("bf16_1048576x128_inplace", BF16, 1 << 20, 128, True, default_scale(128),
                    "bf16 head_dim rotation: 8x32x4096 rows of 128, N(0,1) with 0.1% of entries "
                    "x100, in-place, scale fp32(1/sqrt(128))")


def _fp16_16384x4096() -> Workload:
    return Workload("fp16_16384x4096", FP16, 16384, 4096, False, 1.0 / 64,
                    "fp16 hidden-dim rotation 16384x4096, N(0,1) with 16 fixed columns x50, "
                    "out-of-place, scale 1/64")


def _bf16_4096x32768_inplace() -> Workload:
    return Workload("bf16_4096x32768_inplace", BF16, 4096, 32768, True, default_scale(32768),
                    "bf16 largest size 4096x32768, U(-1,1), in-place, scale fp32(1/sqrt(32768))")


WORKLOADS = {w.name: w for w in (_fp16_1024x256(), _bf16_1048576x128_inplace(), _fp16_16384x4096(),
                                  _bf16_4096x32768_inplace())}


def sweep_point(k: int, dtype: str, inplace: bool, total_log2: int = 28) -> Workload:
    """Sweep point n = 2^k, m = 2^(total_log2 - k), N(0,1).  The paper's sizes are
    k = 7..15; k = 0..6 and k = 16..20 extend the sweep below and above them."""
    if not 0 <= k <= 20:
        raise ValueError("sweep covers n = 2^0 .. 2^20")
    n = 1 << k
    m = 1 << (total_log2 - k)
    mode = "inplace" if inplace else "outofplace"
    return Workload(f"sweep_{dtype}_n{n}_{mode}", dtype, m, n, inplace, default_scale(n),
                    f"{dtype} {m}x{n}, N(0,1) seed {_sweep_seed(k, dtype)}, {mode}, "
                    "scale fp32(1/sqrt(n))")


def _sweep_seed(k: int, dtype: str) -> int:
    return (100 if dtype == FP16 else 200) + k


def generate(w: Workload, rows: int | None = None) -> np.ndarray:
    """The workload's input bits, (m, n) uint16.

    ``rows`` keeps only the first rows.  numpy fills draws in row-major order, so
    a draw of fewer rows equals the first rows of the full draw; the
    bf16_1048576x128_inplace recipe draws its outlier mask after all values and therefore always draws in full.
    """
    m = w.m if rows is None else min(int(rows), w.m)
    n = w.n
    if w.name == "fp16_1024x256":
        rng = np.random.default_rng(0)
        vals = rng.standard_normal((m, n), dtype=np.float32)
    elif w.name == "bf16_1048576x128_inplace":
        rng = np.random.default_rng(2)
        vals = rng.standard_normal((w.m, n), dtype=np.float32)
        mask = rng.random((w.m, n), dtype=np.float32) < 1e-3
        vals[mask] *= np.float32(100.0)
        vals = vals[:m]
    elif w.name == "fp16_16384x4096":
        rng = np.random.default_rng(3)
        cols = rng.choice(n, 16, replace=False)
        vals = rng.standard_normal((m, n), dtype=np.float32)
        vals[:, cols] *= np.float32(50.0)
    elif w.name == "bf16_4096x32768_inplace":
        rng = np.random.default_rng(4)
        vals = rng.uniform(-1.0, 1.0, (m, n)).astype(np.float32)
    elif w.name.startswith("sweep"):
        k = int(math.log2(n))
        rng = np.random.default_rng(_sweep_seed(k, w.dtype))
        vals = rng.standard_normal((m, n), dtype=np.float32)
    else:
        raise ValueError(f"unknown workload {w.name!r}")
    return round_to_bits(np.ascontiguousarray(vals), w.dtype)


def hidden_outlier_columns() -> np.ndarray:
    """The 16 columns scaled x50 in the fp16_16384x4096 workload (drawn first from seed 3)."""
    return np.sort(np.random.default_rng(3).choice(4096, 16, replace=False))
