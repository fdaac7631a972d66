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
import os
from concurrent.futures import ThreadPoolExecutor
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


# Draws are made in slabs of SLAB_ELEMS elements (whole rows): slab s of a
# workload seeded with `seed` takes its numbers from the child seed sequence
# SeedSequence(seed, spawn_key=(s,)), filling its rows in row-major order.  The
# slab layout depends only on the shape, never on the thread count, so any
# number of threads gives the same bits, and a draw of fewer rows is a prefix
# of the full draw.
SLAB_ELEMS = 1 << 22


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    env = os.environ.get("OMP_NUM_THREADS", "")
    if env.isdigit() and int(env) > 0:
        n = min(n, int(env))
    return max(1, min(n, 16))


def _slab_values(w: Workload, seed: int, s: int, rows: int) -> np.ndarray:
    """float32 values of `rows` rows of slab s, by the workload's distribution."""
    rng = np.random.default_rng(np.random.SeedSequence(seed, spawn_key=(s,)))
    n = w.n
    if w.name == "bf16_1048576x128_inplace":
        # N(0,1) values, then (after all of the slab's values) a Bernoulli(1e-3)
        # mask of entries scaled x100
        vals = rng.standard_normal((rows, n), dtype=np.float32)
        mask = rng.random((rows, n), dtype=np.float32) < np.float32(1e-3)
        np.multiply(vals, np.float32(100.0), out=vals, where=mask)
        return vals
    if w.name == "bf16_4096x32768_inplace":
        # U[-1, 1) in fp32 steps of 2^-23
        vals = rng.random((rows, n), dtype=np.float32)
        vals *= np.float32(2.0)
        vals -= np.float32(1.0)
        return vals
    return rng.standard_normal((rows, n), dtype=np.float32)


def _seed(w: Workload) -> int:
    if w.name == "fp16_1024x256":
        return 0
    if w.name == "bf16_1048576x128_inplace":
        return 2
    if w.name == "fp16_16384x4096":
        return 3
    if w.name == "bf16_4096x32768_inplace":
        return 4
    if w.name.startswith("sweep"):
        return _sweep_seed(int(math.log2(w.n)), w.dtype)
    raise ValueError(f"unknown workload {w.name!r}")


def generate(w: Workload, rows: int | None = None) -> np.ndarray:
    """The workload's input bits, (m, n) uint16 (the first ``rows`` rows if given).

    Recipes: fp16_1024x256 N(0,1), seed 0; bf16_1048576x128_inplace N(0,1) with
    0.1% of entries x100, seed 2; fp16_16384x4096 N(0,1) with 16 columns x50 (the
    columns drawn first from default_rng(3), see hidden_outlier_columns), seed 3;
    bf16_4096x32768_inplace U(-1,1), seed 4; sweep points N(0,1), seed 100 + k
    (fp16) or 200 + k (bf16) for n = 2^k.  Values are drawn in fp32 slab by slab
    (see SLAB_ELEMS) and rounded once to the 16-bit dtype.
    """
    m = w.m if rows is None else max(0, min(int(rows), w.m))
    n = w.n
    seed = _seed(w)
    cols = hidden_outlier_columns() if w.name == "fp16_16384x4096" else None
    per = max(1, SLAB_ELEMS // n)
    out = np.empty((m, n), dtype=np.uint16)

    def fill(s: int) -> None:
        r0 = s * per
        r1 = min(m, r0 + per)
        if w.name == "bf16_1048576x128_inplace":
            # its mask follows all of the slab's values: draw the whole slab
            vals = _slab_values(w, seed, s, min(w.m, r0 + per) - r0)[: r1 - r0]
        else:
            vals = _slab_values(w, seed, s, r1 - r0)
        if cols is not None:
            vals[:, cols] *= np.float32(50.0)
        out[r0:r1] = round_to_bits(vals, w.dtype)

    slabs = range((m + per - 1) // per)
    if len(slabs) <= 1:
        for s in slabs:
            fill(s)
    else:
        # numpy's generators and ufuncs release the GIL for bulk work
        with ThreadPoolExecutor(max_workers=_threads()) as ex:
            list(ex.map(fill, slabs))
    return out


def hidden_outlier_columns() -> np.ndarray:
    """The 16 columns scaled x50 in the fp16_16384x4096 workload (drawn first from seed 3)."""
    return np.sort(np.random.default_rng(3).choice(4096, 16, replace=False))
