"""The entry points inside a captured HIP graph, and on concurrent streams.

The C ABI enqueues kernel launches only: no allocation, no memset, no
synchronization.  So a caller can capture it into a graph, for example a
serving loop, and replay it.  Each replay here follows eager work that
rewrites the inputs, and every replay is checked against the eager call on
the same inputs.
"""
from __future__ import annotations

import pytest

from paper_2412_08832_amd import hadacore as H

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _device():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    H.library()
    yield
    torch.cuda.synchronize()


CASES = [  # (n, m, dtype, in place): wave kernel, block kernel, persistent loop
    (128, 4099, "bf16", True),
    (32768, 37, "fp16", False),
    (65536, 300, "bf16", False),
]


@pytest.mark.parametrize("n,m,dtype,inplace", CASES)
def test_graph_replays_match_eager(n, m, dtype, inplace):
    import torch
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float16
    code = H.BF16 if dtype == "bf16" else H.FP16
    scale = 1.0 / n ** 0.5
    x = torch.empty(m, n, dtype=tdt, device="cuda")
    out = x if inplace else torch.empty_like(x)
    codes = torch.empty(m, n, dtype=torch.uint8, device="cuda")
    scales = torch.empty(m, dtype=torch.float32, device="cuda")
    src = torch.empty_like(x)      # the graph's input for the 16-bit call when in place

    def enqueue(stream):
        # FP8 codes of x, then the 16-bit transform (in place when asked)
        H.hadamard_transform_fp8(x.data_ptr(), n, codes.data_ptr(), n, scales.data_ptr(), m, n,
                                 code, scale, stream)
        H.hadamard_transform(x.data_ptr(), out.data_ptr(), m, n, code, scale, stream)

    # one eager call first: the library's one-time device check happens outside capture
    gen = torch.Generator(device="cuda").manual_seed(n)
    src.copy_(torch.randn(m, n, device="cuda", generator=gen).to(tdt))
    x.copy_(src)
    enqueue(torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()

    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            enqueue(side.cuda_stream)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()

    for replay in range(4):
        # eager work between replays: new inputs, then the eager reference
        src.copy_(torch.randn(m, n, device="cuda", generator=gen).to(tdt))
        x.copy_(src)
        enqueue(torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        ref_out, ref_codes, ref_scales = out.clone(), codes.clone(), scales.clone()
        x.copy_(src)
        if not inplace:
            out.zero_()
        codes.zero_()
        scales.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref_out), f"replay {replay}: transform differs from eager"
        assert torch.equal(codes, ref_codes), f"replay {replay}: FP8 codes differ from eager"
        assert torch.equal(scales, ref_scales), f"replay {replay}: scales differ from eager"


def test_concurrent_streams_match_serial():
    """Calls on two streams at once (different buffers, different sizes) give the
    same bits as the same calls one after the other."""
    import torch
    gen = torch.Generator(device="cuda").manual_seed(7)
    a = torch.randn(8192, 4096, device="cuda", generator=gen).to(torch.bfloat16)
    b = torch.randn(1 << 16, 128, device="cuda", generator=gen).to(torch.float16)
    ra, rb = torch.empty_like(a), torch.empty_like(b)
    s0 = torch.cuda.current_stream().cuda_stream
    H.hadamard_transform(a.data_ptr(), ra.data_ptr(), 8192, 4096, H.BF16, 1 / 64, s0)
    H.hadamard_transform(b.data_ptr(), rb.data_ptr(), 1 << 16, 128, H.FP16, 0.125, s0)
    torch.cuda.synchronize()
    oa, ob = torch.empty_like(a), torch.empty_like(b)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    for _ in range(3):
        oa.zero_()
        ob.zero_()
        torch.cuda.synchronize()
        for i in range(4):   # interleave several launches on both streams
            H.hadamard_transform(a.data_ptr(), oa.data_ptr(), 8192, 4096, H.BF16, 1 / 64,
                                 s1.cuda_stream)
            H.hadamard_transform(b.data_ptr(), ob.data_ptr(), 1 << 16, 128, H.FP16, 0.125,
                                 s2.cuda_stream)
        torch.cuda.synchronize()
        assert torch.equal(oa, ra) and torch.equal(ob, rb)
