"""Comparison metrics between a 16-bit GPU result and the fp64 oracle.

Tolerance (the reading of "relative L2 <= 1e-3 (fp16) / 8e-3 (bf16) and max
elementwise error <= 4 ulp of the output dtype"):

* rel_l2 = ||gpu - ref||_F / ||ref||_F over finite reference entries;
* err_ulp[i, j] = |gpu - ref| / ulp(max(|ref|, tau_i)), tau_i = 2^-8 * rms_i,
  rms_i the root-mean-square of reference row i; ulp(v) = 2^(floor(log2 v) - p)
  with p = 10 (fp16) or 7 (bf16), floored at the dtype's subnormal spacing;
* non-finite references must be matched by class (NaN with NaN, +-Inf with the
  same-signed Inf); rows whose reference is all zero need exact zeros.

The floor keeps the per-element ulp well conditioned where a row's output
crosses zero: there the correctly rounded 16-bit value itself has relative
error far above 4 ulp of |ref|, whatever the kernel does.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

PRECISION_BITS = {"fp16": 10, "bf16": 7}
MIN_SPACING_LOG2 = {"fp16": -24, "bf16": -133}
REL_L2_LIMIT = {"fp16": 1e-3, "bf16": 8e-3}
MAX_ULP_LIMIT = 4.0
FLOOR_LOG2 = -8


def bits_to_f64(bits: np.ndarray, dtype: str) -> np.ndarray:
    """Decode fp16/bf16 bit patterns with numpy (fp16 view, bf16 as the top half of fp32)."""
    bits = np.asarray(bits, dtype=np.uint16)
    if dtype == "fp16":
        return bits.view(np.float16).astype(np.float64)
    if dtype == "bf16":
        return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    raise ValueError(dtype)


def ulp(values: np.ndarray, dtype: str) -> np.ndarray:
    """Spacing of the dtype's representable numbers at |values| (binade-wise), floored."""
    v = np.abs(np.asarray(values, dtype=np.float64))
    p = PRECISION_BITS[dtype]
    lo = MIN_SPACING_LOG2[dtype]
    with np.errstate(divide="ignore"):
        e = np.floor(np.log2(np.where(v > 0, v, 1.0)))
    e = np.where(v > 0, e, lo + p)
    return np.exp2(np.maximum(e - p, lo))


@dataclass
class Comparison:
    dtype: str
    count: int
    rel_l2: float
    max_ulp_floored: float
    max_ulp_unfloored: float
    n_above_4ulp_unfloored: int
    nonfinite_mismatch: int
    zero_row_mismatch: int

    @property
    def ok(self) -> bool:
        return (self.rel_l2 <= REL_L2_LIMIT[self.dtype]
                and self.max_ulp_floored <= MAX_ULP_LIMIT
                and self.nonfinite_mismatch == 0
                and self.zero_row_mismatch == 0)

    def __str__(self) -> str:
        return (f"{self.dtype}: n={self.count} rel_l2={self.rel_l2:.3e} "
                f"max_ulp_floored={self.max_ulp_floored:.3f} "
                f"max_ulp_unfloored={self.max_ulp_unfloored:.3g} "
                f"above4={self.n_above_4ulp_unfloored} nonfinite_mismatch={self.nonfinite_mismatch} "
                f"zero_row_mismatch={self.zero_row_mismatch}")


class Accumulator:
    """Accumulates the comparison over row blocks so that large matrices never
    need all of their float64 temporaries at once."""

    def __init__(self, dtype: str):
        self.dtype = dtype
        self.count = 0
        self.num = 0.0
        self.den = 0.0
        self.max_floored = 0.0
        self.max_unfloored = 0.0
        self.above = 0
        self.mismatch = 0
        self.zero_mismatch = 0

    def add(self, gpu: np.ndarray, ref: np.ndarray) -> "Accumulator":
        gpu = np.asarray(gpu, dtype=np.float64)
        ref = np.asarray(ref, dtype=np.float64)
        if gpu.shape != ref.shape:
            raise ValueError(f"shape mismatch {gpu.shape} vs {ref.shape}")
        if ref.ndim == 1:
            gpu = gpu[None, :]
            ref = ref[None, :]
        if ref.size == 0:
            return self
        fin = np.isfinite(ref)
        gfin = np.isfinite(gpu)
        self.mismatch += int(np.count_nonzero(np.isnan(ref) & ~np.isnan(gpu)))
        self.mismatch += int(np.count_nonzero(np.isinf(ref) & (gpu != ref)))
        self.mismatch += int(np.count_nonzero(fin & ~gfin))
        both = fin & gfin
        r = np.where(fin, ref, 0.0)
        diff = np.where(both, gpu - r, 0.0)
        self.den += float(np.sum(r * r))
        self.num += float(np.sum(diff * diff))
        rms = np.sqrt(np.mean(r * r, axis=1, keepdims=True))
        absdiff = np.abs(diff)
        floored = absdiff / ulp(np.maximum(np.abs(r), rms * 2.0 ** FLOOR_LOG2), self.dtype)
        unfloored = absdiff / ulp(np.abs(r), self.dtype)
        self.max_floored = max(self.max_floored, float(floored.max()))
        self.max_unfloored = max(self.max_unfloored, float(unfloored.max()))
        self.above += int(np.count_nonzero(unfloored > MAX_ULP_LIMIT))
        zero_rows = np.all(r == 0, axis=1) & np.all(fin, axis=1)
        if zero_rows.any():
            g = np.where(gfin, gpu, 1.0)
            self.zero_mismatch += int(np.count_nonzero(np.any(g[zero_rows] != 0, axis=1)))
        self.count += int(ref.size)
        return self

    def result(self) -> Comparison:
        if self.den > 0:
            rel = float(np.sqrt(self.num / self.den))
        else:
            rel = 0.0 if self.num == 0 else float("inf")
        return Comparison(self.dtype, self.count, rel, self.max_floored, self.max_unfloored,
                          self.above, self.mismatch, self.zero_mismatch)


def compare(gpu: np.ndarray, ref: np.ndarray, dtype: str) -> Comparison:
    """Compare decoded GPU values ``gpu`` with oracle values ``ref`` (both (m, n) float64)."""
    return Accumulator(dtype).add(gpu, ref).result()
