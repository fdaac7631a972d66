"""Comparison metrics between a 16-bit GPU result and the fp64 oracle.

Tolerance (the reading of "relative L2 <= 1e-3 (fp16) / 8e-3 (bf16) and max
elementwise error <= 4 ulp of the output dtype"):

* rel_l2 = ||gpu - ref||_F / ||ref||_F over finite reference entries;
* err_ulp[i, j] = |gpu - ref| / ulp(max(|ref|, tau_i)), tau_i = 2^-8 * rms_i,
  rms_i the root-mean-square of reference row i; ulp(v) = 2^(floor(log2 v) - p)
  with p = 10 (fp16) or 7 (bf16), floored at the dtype's subnormal spacing;
* non-finite references must be matched by class (NaN with NaN, +-Inf with the
  same-signed Inf); rows whose reference is all zero need exact zeros.

Why the floor.  A correctly rounded 16-bit output is within 0.5 ulp(|ref|) of
ref wherever ref is, so the floor is not about the final rounding.  It is about
the fp32 partial sums before it.  Each of the log2(n) butterfly levels rounds
values of the size of the row's outputs, so the fp32 result carries an absolute
error of about c * log2(n) * 2^-24 * rms (rms: the row's root-mean-square
output, c a small constant), whatever |ref| is.  Near a zero crossing |ref| is
far below rms, and that error divided by ulp(|ref|) grows without bound as
|ref| -> 0: the unfloored 4-ulp bound is out of reach of any fp32 kernel.  At
the floor |ref| = 2^-8 * rms the same error is c * log2(n) * 2^-16 of the value,
i.e. c * log2(n) / 64 fp16 ulps (0.23 c at n = 2^15) or c * log2(n) / 512 bf16
ulps, well inside 4 ulp; a 16-bit rounding of an intermediate (about 2^-11 * rms
absolute for fp16) is 2^7 floored ulps there and fails.  The unfloored maximum
and the count of elements above 4 unfloored ulps are reported beside it.
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
    """Spacing of the dtype's representable numbers at |values| (binade-wise), floored
    at the subnormal spacing: 2^max(floor(log2 |v|) - p, lo), read exactly from the
    fp64 exponent field (zero and fp64 subnormals, all below every floor, give 2^lo)."""
    v = np.abs(np.asarray(values, dtype=np.float64))
    p = PRECISION_BITS[dtype]
    lo = MIN_SPACING_LOG2[dtype]
    biased = (v.view(np.uint64) >> np.uint64(52)).astype(np.int64)  # floor(log2 v) + 1023
    e = np.maximum(biased - (1023 + p), lo)
    return ((e + 1023).astype(np.uint64) << np.uint64(52)).view(np.float64)


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
        if fin.all() and gfin.all():
            return self._add_finite(gpu, ref)
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

    def _add_finite(self, gpu: np.ndarray, ref: np.ndarray) -> "Accumulator":
        """add() for blocks whose entries are all finite (the common case)."""
        diff = gpu - ref
        sq = ref * ref
        self.den += float(sq.sum())
        self.num += float(np.vdot(diff, diff).real) if diff.flags.c_contiguous \
            else float((diff * diff).sum())
        rms = np.sqrt(sq.mean(axis=1, keepdims=True))
        absdiff = np.abs(diff)
        absref = np.abs(ref)
        floored = absdiff / ulp(np.maximum(absref, rms * 2.0 ** FLOOR_LOG2), self.dtype)
        unfloored = absdiff / ulp(absref, self.dtype)
        self.max_floored = max(self.max_floored, float(floored.max()))
        self.max_unfloored = max(self.max_unfloored, float(unfloored.max()))
        self.above += int(np.count_nonzero(unfloored > MAX_ULP_LIMIT))
        zero_rows = ~np.any(ref != 0, axis=1)
        if zero_rows.any():
            self.zero_mismatch += int(np.count_nonzero(np.any(gpu[zero_rows] != 0, axis=1)))
        self.count += int(ref.size)
        return self

    def merge(self, other: "Accumulator") -> "Accumulator":
        """Combine the statistics of another accumulator of the same dtype."""
        if other.dtype != self.dtype:
            raise ValueError("dtype mismatch")
        self.count += other.count
        self.num += other.num
        self.den += other.den
        self.max_floored = max(self.max_floored, other.max_floored)
        self.max_unfloored = max(self.max_unfloored, other.max_unfloored)
        self.above += other.above
        self.mismatch += other.mismatch
        self.zero_mismatch += other.zero_mismatch
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
