"""hadamard_transform_ws_noalloc against hadamard_transform_ws, through the C ABI.

The allocation-free entry point runs the same two-pass kernels as
hadamard_transform_ws with the workspace taken from the library's fixed device
array, so its output must equal the workspace call's bit for bit.  Two calls in
a row, the second on a smaller problem, check that the array's leftover
contents from the first call do not leak into the second.  A problem whose
workspace would exceed the array is rejected before anything is enqueued.
"""
from __future__ import annotations

import numpy as np
import pytest

from gpu_util import compare_with_oracle, say, to_device, to_host
from paper_2412_08832_amd import hadacore as H
from paper_2412_08832_amd import workloads as W

pytestmark = pytest.mark.gpu

CODE = {"fp16": H.FP16, "bf16": H.BF16}


def _pair(oracle, m, n, dtype, inplace, seed):
    """Run both entry points on the same input; return (noalloc bits, ws bits, input bits)."""
    import torch
    bits = W.random_rows(m, n, dtype, seed=seed)
    s = W.default_scale(n)
    stream = torch.cuda.current_stream().cuda_stream
    outs = []
    for entry in ("ws", "noalloc"):
        x = to_device(bits, dtype)
        y = x if inplace else torch.empty_like(x)
        if entry == "ws":
            need = H.hadamard_transform_workspace_size(m, n)
            ws = torch.empty(need, dtype=torch.uint8, device="cuda")
            H.hadamard_transform_ws(x.data_ptr(), n, y.data_ptr(), n, m, n, CODE[dtype], s,
                                    ws.data_ptr(), need, stream)
        else:
            H.hadamard_transform_ws_noalloc(x.data_ptr(), n, y.data_ptr(), n, m, n, CODE[dtype], s,
                                            stream)
        torch.cuda.synchronize()
        outs.append(to_host(y))
    c = compare_with_oracle(oracle, outs[1], bits, dtype, s, n, rows=[0, m // 2, m - 1])
    say(f"  noalloc m={m} n={n} {dtype} inplace={inplace}: {c}")
    assert c.ok, str(c)
    return outs[1], outs[0]


@pytest.mark.parametrize("inplace", [False, True], ids=["out", "inplace"])
@pytest.mark.parametrize("dtype", ["fp16", "bf16"])
def test_noalloc_equals_workspace_call_twice(oracle, dtype, inplace):
    # first call: the largest problem the array holds at n = 2^17 (64 rows =
    # 32 MiB of fp32 workspace); second: a smaller one at n = 2^18 (5 rows)
    first = (H.NOALLOC_SCRATCH_BYTES // (4 << 17), 1 << 17)
    assert H.hadamard_transform_workspace_size(*first) == H.NOALLOC_SCRATCH_BYTES
    for (m, n), seed in ((first, 17), ((5, 1 << 18), 18)):
        say(f"noalloc vs ws: m={m} n={n} {dtype} inplace={inplace}")
        a, b = _pair(oracle, m, n, dtype, inplace, seed)
        assert np.array_equal(a, b)


def test_noalloc_one_pass_sizes_need_no_scratch(oracle):
    """n <= 2^16 is the one-pass transform: any m, no scratch limit."""
    import torch
    m, n = 3000, 4096     # 12M elements: beyond the scratch array, fine for one pass
    bits = W.random_rows(m, n, "bf16", seed=4096)
    x = to_device(bits, "bf16")
    y = torch.empty_like(x)
    s = W.default_scale(n)
    H.hadamard_transform_ws_noalloc(x.data_ptr(), n, y.data_ptr(), n, m, n, H.BF16, s,
                                    torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    c = compare_with_oracle(oracle, to_host(y), bits, "bf16", s, n)
    assert c.ok, str(c)


def test_noalloc_rejects_problems_beyond_the_array():
    import torch
    n = 1 << 17
    m = H.NOALLOC_SCRATCH_BYTES // (4 * n) + 1
    x = torch.zeros((m, n), dtype=torch.bfloat16, device="cuda")
    st = H.hadamard_transform_ws_noalloc(x.data_ptr(), n, x.data_ptr(), n, m, n, H.BF16, 1.0,
                                         torch.cuda.current_stream().cuda_stream, check=False)
    assert H.STATUS_NAMES[st] == "SCRATCH"
    torch.cuda.synchronize()
    assert int(x.view(torch.int16).abs().sum()) == 0   # nothing was enqueued
