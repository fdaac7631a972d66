"""Helpers for GPU tests: move 16-bit bit patterns to and from the device, run
the library through its C ABI, and compare with the oracle block by block."""
from __future__ import annotations

import os
import sys

import numpy as np

from metrics import Accumulator, bits_to_f64

TORCH_DTYPE = None


def torch_dtype(dtype: str):
    import torch
    return {"fp16": torch.float16, "bf16": torch.bfloat16}[dtype]


def to_device(bits: np.ndarray, dtype: str):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to("cuda")
    return t.view(torch_dtype(dtype))


def to_host(t) -> np.ndarray:
    import torch
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def oracle_threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def say(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def compare_with_oracle(oracle, out_bits: np.ndarray, in_bits: np.ndarray, dtype: str,
                        scale: float, n: int, rows=None, block_elems: int = 1 << 23):
    """Compare out_bits[:, :n] with the oracle transform of in_bits[:, :n].

    ``rows`` restricts the comparison to the given row indices (sampled check).
    """
    acc = Accumulator(dtype)
    if rows is not None:
        rows = np.asarray(rows, dtype=np.int64)
        ref = oracle.fwht(np.ascontiguousarray(in_bits[rows]), dtype, scale, n=n,
                          nthreads=oracle_threads())
        acc.add(bits_to_f64(out_bits[rows, :n], dtype), ref)
        return acc.result()
    m = in_bits.shape[0]
    step = max(1, block_elems // max(n, 1))
    for r0 in range(0, m, step):
        r1 = min(m, r0 + step)
        ref = oracle.fwht(np.ascontiguousarray(in_bits[r0:r1]), dtype, scale, n=n,
                          nthreads=oracle_threads())
        acc.add(bits_to_f64(out_bits[r0:r1, :n], dtype), ref)
    return acc.result()
