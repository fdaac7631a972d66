"""Helpers for GPU tests: move 16-bit bit patterns to and from the device, run
the library through its C ABI, and compare with the oracle block by block."""
from __future__ import annotations

import os
import sys
from concurrent.futures import ThreadPoolExecutor

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
    """Host threads for oracle checks: the CPUs this process may run on, capped by
    OMP_NUM_THREADS when it is set (the GPU machine sets it to its CPU share)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    env = os.environ.get("OMP_NUM_THREADS", "")
    if env.isdigit() and int(env) > 0:
        n = min(n, int(env))
    return max(1, n)


def say(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def compare_with_oracle(oracle, out_bits: np.ndarray, in_bits: np.ndarray, dtype: str,
                        scale: float, n: int, rows=None, block_elems: int = 1 << 18,
                        threads: int | None = None):
    """Compare out_bits[:, :n] with the oracle transform of in_bits[:, :n].

    ``rows`` restricts the comparison to the given row indices (sampled check).
    Row blocks of about ``block_elems`` elements are transformed by the oracle and
    compared in a pool of ``threads`` host threads (the oracle's C code and numpy
    release the GIL); the per-block statistics are merged, so the result does not
    depend on the block size or the thread count.
    """
    if rows is not None:
        rows = np.asarray(rows, dtype=np.int64)
        in_bits = in_bits[rows]
        out_bits = out_bits[rows]
    m = in_bits.shape[0]
    step = max(1, block_elems // max(n, 1))

    def block(r0: int) -> Accumulator:
        r1 = min(m, r0 + step)
        ref = oracle.fwht(np.ascontiguousarray(in_bits[r0:r1]), dtype, scale, n=n, nthreads=1)
        return Accumulator(dtype).add(bits_to_f64(out_bits[r0:r1, :n], dtype), ref)

    starts = range(0, m, step)
    t = oracle_threads() if threads is None else max(1, int(threads))
    acc = Accumulator(dtype)
    if t == 1 or len(starts) == 1:
        for r0 in starts:
            acc.merge(block(r0))
    else:
        with ThreadPoolExecutor(max_workers=t) as ex:
            for a in ex.map(block, starts):
                acc.merge(a)
    return acc.result()
