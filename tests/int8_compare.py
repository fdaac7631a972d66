"""Comparison of fused INT8 results with the oracle.

Codes are judged in the oracle's own decision variable v = y32 * (127/amax),
y32 being the exact transform rounded once to fp32.  A GPU code must equal the
oracle's code, or -- where the GPU's fp32 transform (whose error is a small
multiple of 2^-24 of the row's magnitudes) can land on the other side of a
rounding boundary -- lie within one half plus that error of v.  Rows without a
usable scale (amax 0, Inf or NaN, or 127/amax overflowing fp32) must have
all-zero codes.  Scales must agree
within a few fp32 ulps (two subnormal steps for scales below 2^-126).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

REL_FP32_SLACK = 2.0 ** -17      # fp32 transform error allowance, relative to the row maximum
SCALE_RTOL = 2.0 ** -19          # a few fp32 ulps
# plus two fp32 subnormal steps: a row scale below 2^-126 has fewer significant
# bits, and the fp32 transform's error in amax can move its last one
SCALE_ATOL = 2.0 * 2.0 ** -149
MAX_MISMATCH_FRACTION = 1e-3


@dataclass
class Int8Comparison:
    count: int
    mismatches: int
    invalid: int
    scale_bad: int

    @property
    def ok(self) -> bool:
        return (self.invalid == 0 and self.scale_bad == 0
                and self.mismatches <= MAX_MISMATCH_FRACTION * max(self.count, 1))

    def __str__(self) -> str:
        return (f"int8: n={self.count} code_mismatches={self.mismatches} invalid={self.invalid} "
                f"scale_bad={self.scale_bad}")


def compare_int8(oracle, codes_gpu: np.ndarray, scales_gpu: np.ndarray, bits: np.ndarray,
                 dtype: str, scale: float, n: int) -> Int8Comparison:
    codes_o, scales_o = oracle.fwht_int8(bits, dtype, scale, n=n)
    y32 = oracle.fwht(bits, dtype, scale, n=n).astype(np.float32)
    with np.errstate(all="ignore"):
        amax = np.where(np.isnan(y32).all(axis=1), np.nan, np.nanmax(np.abs(y32), axis=1))
        amax = amax.astype(np.float32)
        q = (np.float32(127.0) / amax).astype(np.float32)
        usable = np.isfinite(amax) & np.isfinite(q)
        inv = np.where(usable, q, np.float32(0.0)).astype(np.float32)
        v = (y32 * inv[:, None]).astype(np.float64)
    cg = codes_gpu[:, :n].astype(np.int8).astype(np.float64)
    co = codes_o.astype(np.float64)
    exact = cg == co
    with np.errstate(all="ignore"):
        near = np.abs(cg - v) <= 0.5 + REL_FP32_SLACK * 127.0
    valid = np.where(usable[:, None], exact | near, cg == 0)
    sg = scales_gpu.astype(np.float64)
    so = scales_o.astype(np.float64)
    same_class = (np.isnan(sg) == np.isnan(so)) & (np.isinf(sg) == np.isinf(so))
    with np.errstate(all="ignore"):
        close = np.where(np.isfinite(so), np.abs(sg - so) <= SCALE_RTOL * np.abs(so) + SCALE_ATOL,
                         sg == so)
    close = close | (np.isnan(sg) & np.isnan(so))
    return Int8Comparison(count=int(cg.size), mismatches=int(np.count_nonzero(~exact)),
                          invalid=int(np.count_nonzero(~valid)),
                          scale_bad=int(np.count_nonzero(~(same_class & close))))
