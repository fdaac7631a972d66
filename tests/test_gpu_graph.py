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


CASES = [  # (n, m, dtype, in place): wave kernel, block kernel, persistent loops
    (128, 4099, "bf16", True),
    (32768, 37, "fp16", False),
    (32768, 4100, "bf16", True),
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


def test_host_threads_match_serial():
    """Calls from four host threads at once, each on its own stream and buffers
    (wave kernel, block kernel, persistent loop, FP8 output), give the same bits
    as the same calls made one after the other from one thread."""
    import threading
    import torch
    gen = torch.Generator(device="cuda").manual_seed(11)
    jobs = [  # (m, n, torch dtype, library dtype, fp8 output)
        (8192, 4096, torch.bfloat16, H.BF16, False),
        (1 << 16, 128, torch.float16, H.FP16, False),
        (300, 1 << 16, torch.bfloat16, H.BF16, False),
        (4096, 1024, torch.float16, H.FP16, True),
    ]
    xs = [torch.randn(m, n, device="cuda", generator=gen).to(dt) for m, n, dt, _, _ in jobs]

    def outputs(i):
        m, n, dt, _, q = jobs[i]
        if q:
            return (torch.empty(m, n, dtype=torch.uint8, device="cuda"),
                    torch.empty(m, dtype=torch.float32, device="cuda"))
        return (torch.empty(m, n, dtype=dt, device="cuda"),)

    def call(i, outs, stream):
        m, n, _, code, q = jobs[i]
        x = xs[i]
        if q:
            H.hadamard_transform_fp8(x.data_ptr(), n, outs[0].data_ptr(), n, outs[1].data_ptr(),
                                     m, n, code, n ** -0.5, stream)
        else:
            H.hadamard_transform(x.data_ptr(), outs[0].data_ptr(), m, n, code, n ** -0.5, stream)

    s0 = torch.cuda.current_stream().cuda_stream
    refs = [outputs(i) for i in range(len(jobs))]
    for i in range(len(jobs)):
        call(i, refs[i], s0)
    torch.cuda.synchronize()

    streams = [torch.cuda.Stream() for _ in jobs]
    for _ in range(2):
        got = [outputs(i) for i in range(len(jobs))]
        for o in got:
            for t in o:
                t.zero_()
        torch.cuda.synchronize()
        errors = []
        start = threading.Barrier(len(jobs))

        def worker(i):
            try:
                start.wait()
                for _ in range(5):
                    call(i, got[i], streams[i].cuda_stream)
            except Exception as e:  # reported below, in the main thread
                errors.append(e)

        threads = [threading.Thread(target=worker, args=(i,)) for i in range(len(jobs))]
        for t in threads:
            t.start()
        for t in threads:
            t.join(timeout=120)
        assert not any(t.is_alive() for t in threads), "a host thread did not finish"
        assert not errors, errors
        torch.cuda.synchronize()
        for i in range(len(jobs)):
            for a, b in zip(got[i], refs[i]):
                assert torch.equal(a, b), f"job {i} differs from the serial result"


def test_graph_replays_two_pass_size():
    """n = 2^17 runs two kernels through the caller's workspace; captured and
    replayed, each replay equals the eager call on the same input."""
    import torch
    m, n = 24, 1 << 17
    gen = torch.Generator(device="cuda").manual_seed(17)
    x = torch.empty(m, n, dtype=torch.bfloat16, device="cuda")
    out = torch.empty_like(x)
    ws = torch.empty(H.hadamard_transform_workspace_size(m, n), dtype=torch.uint8, device="cuda")

    def enqueue(stream):
        H.hadamard_transform_ws(x.data_ptr(), n, out.data_ptr(), n, m, n, H.BF16, n ** -0.5,
                                ws.data_ptr(), ws.numel(), stream)

    x.copy_(torch.randn(m, n, device="cuda", generator=gen).to(torch.bfloat16))
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
    for replay in range(3):
        x.copy_(torch.randn(m, n, device="cuda", generator=gen).to(torch.bfloat16))
        enqueue(torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        ref = out.clone()
        out.zero_()
        ws.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref), f"replay {replay}: two-pass transform differs from eager"
