"""GPU parity: libhadacore (through its C ABI) against the fp64 oracle.

Tolerance (written here, derived in the design notes): rel-L2 <= 1e-3 (fp16)
or 8e-3 (bf16) and max error <= 4 ulp of the output dtype with the ulp taken
at max(|ref|, 2^-8 * row RMS); non-finite outputs must match by class.
"""
from __future__ import annotations

import numpy as np
import pytest

from gpu_util import compare_with_oracle, say, to_device, to_host
from metrics import bits_to_f64
from paper_2412_08832_amd import hadacore as H
from paper_2412_08832_amd import workloads as W

pytestmark = pytest.mark.gpu

DTYPES = ["fp16", "bf16"]
CODE = {"fp16": H.FP16, "bf16": H.BF16}


VARIANTS = ["auto", "valu", "mfma"]


@pytest.fixture(scope="module", autouse=True)
def _device():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    H.library()  # fail loudly if the HIP library is missing
    yield
    torch.cuda.synchronize()


@pytest.fixture(params=VARIANTS)
def variant(request, monkeypatch):
    """Front end of the transform: the per-size table ("auto") or forced VALU / matrix-core."""
    if request.param == "auto":
        monkeypatch.delenv("HADACORE_VARIANT", raising=False)
    else:
        monkeypatch.setenv("HADACORE_VARIANT", request.param)
    return request.param


def _run(bits: np.ndarray, dtype: str, scale: float, n: int, inplace: bool,
         out_stride: int | None = None, out_fill: int = 0xAAAA):
    """Transform on the GPU through hadamard_transform_strided; returns output bits."""
    import torch
    m, in_stride = bits.shape
    x = to_device(bits, dtype)
    if inplace:
        out, out_stride = x, in_stride
    else:
        out_stride = n if out_stride is None else out_stride
        out = to_device(np.full((m, out_stride), out_fill, np.uint16), dtype)
    H.hadamard_transform_strided(x.data_ptr(), in_stride, out.data_ptr(), out_stride, m, n,
                                 CODE[dtype], scale, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    return to_host(out)


def _ragged_rows(L: int) -> int:
    # n <= 4096 spans many workgroups and leaves a ragged tail (multi-row tiles for
    # n <= 256, one row per thread for n <= 8); larger n run one row per workgroup
    return (1 << 21 >> L) + 3 if L <= 12 else 37


@pytest.mark.parametrize("inplace", [False, True], ids=["out", "inplace"])
@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("L", range(0, 17))
def test_every_size_ragged(oracle, L, dtype, inplace, variant):
    n = 1 << L
    m = _ragged_rows(L)
    say(f"every_size n={n} m={m} {dtype} inplace={inplace} variant={variant}")
    bits = W.random_rows(m, n, dtype, seed=1000 + L)
    s = W.default_scale(n)
    out = _run(bits, dtype, s, n, inplace)
    c = compare_with_oracle(oracle, out, bits, dtype, s, n)
    say(f"  {c}")
    assert c.ok, str(c)


@pytest.mark.parametrize("name", ["fp16_1024x256", "bf16_1048576x128_inplace", "fp16_16384x4096", "bf16_4096x32768_inplace"])
def test_configs_full_size(oracle, name):
    w = W.WORKLOADS[name]
    say(f"config {w.name}: {w.description}")
    bits = W.generate(w)
    out = _run(bits, w.dtype, w.scale, w.n, w.inplace)
    c = compare_with_oracle(oracle, out, bits, w.dtype, w.scale, w.n)
    say(f"  {c}")
    assert c.ok, str(c)


@pytest.mark.parametrize("name", ["fp16_1024x256", "bf16_1048576x128_inplace", "fp16_16384x4096", "bf16_4096x32768_inplace"])
def test_configs_other_mode_bitwise(name):
    """Each named workload in the other mode (in place <-> out of place) gives the
    same bits as its stated mode, which test_configs_full_size checks against the oracle."""
    w = W.WORKLOADS[name]
    bits = W.generate(w)
    a = _run(bits, w.dtype, w.scale, w.n, w.inplace)
    b = _run(bits, w.dtype, w.scale, w.n, not w.inplace)
    assert np.array_equal(a, b)


# Sweep points (2^28 elements) compared in full where the dispatch changes shape
# and above: n = 2048 (two-wave block kernel), 4096 (matrix-core front),
# 8192-32768 (block kernels; n = 32768 at 8192 rows runs the persistent loop) and 65536 (the
# persistent loop); elsewhere about 2^20 elements of sampled rows.
FULL_SWEEP_L = (11, 12, 13, 14, 15, 16)


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("L", [1, 4, 6] + list(range(7, 17)))
def test_sweep_full_size(oracle, L, dtype):
    w = W.sweep_point(L, dtype, inplace=True)
    bits = W.generate(w)
    rows = None
    if L not in FULL_SWEEP_L:
        rng = np.random.default_rng(L)
        rows = np.unique(np.r_[0, w.m - 1, rng.integers(0, w.m, max(256, (1 << 20) >> L))])
    for inplace in (True, False):
        say(f"sweep {dtype} n={w.n} m={w.m} inplace={inplace} "
            f"({'all rows' if rows is None else f'{len(rows)} sampled rows'})")
        out = _run(bits, dtype, w.scale, w.n, inplace)
        c = compare_with_oracle(oracle, out, bits, dtype, w.scale, w.n, rows=rows)
        say(f"  {c}")
        assert c.ok, str(c)
        del out


@pytest.mark.parametrize("inplace", [False, True], ids=["out", "inplace"])
@pytest.mark.parametrize("dtype", DTYPES)
def test_n65536_several_rows_per_workgroup(oracle, dtype, inplace, variant):
    """n = 65536 runs one persistent workgroup per CU (matrix-core front): with
    m = 2 * CUs + 37 rows each workgroup takes two or three rows in turn."""
    import torch
    n = 1 << 16
    m = 2 * torch.cuda.get_device_properties(0).multi_processor_count + 37
    say(f"n=65536 m={m} {dtype} inplace={inplace} variant={variant}")
    bits = W.random_rows(m, n, dtype, seed=616)
    s = W.default_scale(n)
    out = _run(bits, dtype, s, n, inplace)
    c = compare_with_oracle(oracle, out, bits, dtype, s, n)
    say(f"  {c}")
    assert c.ok, str(c)


@pytest.mark.parametrize("inplace", [False, True], ids=["out", "inplace"])
@pytest.mark.parametrize("dtype", DTYPES)
def test_n65536_nonfinite_rows_between_ordinary_rows(oracle, dtype, inplace, variant):
    """NaN, Inf and zero rows handled by a persistent n = 65536 workgroup before
    and after ordinary rows: nothing carries over to the rows that follow."""
    import torch
    n = 1 << 16
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    m = 2 * cus + 5
    say(f"n=65536 nonfinite rows m={m} {dtype} inplace={inplace} variant={variant}")
    bits = W.random_rows(m, n, dtype, seed=67)
    nan = 0x7E00 if dtype == "fp16" else 0x7FC0
    inf = 0x7C00 if dtype == "fp16" else 0x7F80
    bits[0, 11] = nan
    bits[cus + 1, 5] = nan
    bits[1, 3] = inf
    bits[2 * cus, 1] = inf | 0x8000
    bits[2] = 0
    bits[cus + 3] = 0
    s = W.default_scale(n)
    out = _run(bits, dtype, s, n, inplace)
    c = compare_with_oracle(oracle, out, bits, dtype, s, n)
    say(f"  {c}")
    assert c.ok, str(c)


@pytest.mark.parametrize("inplace", [False, True], ids=["out", "inplace"])
@pytest.mark.parametrize("dtype,m", [("bf16", 4095), ("bf16", 4096), ("fp16", 4095), ("fp16", 4096),
                                     ("bf16", 4099)])
def test_n32768_either_side_of_the_loop_switch(oracle, dtype, m, inplace):
    """16-bit n = 32768 runs the persistent loop (one workgroup per CU) from 4096
    rows and the block kernel below; both sides of the switch against the oracle
    on sampled rows (first, last, random; 4099 rows leave a few workgroups a
    seventeenth row)."""
    n = 1 << 15
    say(f"{dtype} n=32768 m={m} inplace={inplace}")
    bits = W.random_rows(m, n, dtype, seed=m)
    s = W.default_scale(n)
    out = _run(bits, dtype, s, n, inplace)
    rng = np.random.default_rng(m)
    rows = np.unique(np.r_[0, 1, m - 2, m - 1, rng.integers(0, m, 128)])
    c = compare_with_oracle(oracle, out, bits, dtype, s, n, rows=rows)
    say(f"  {c}")
    assert c.ok, str(c)


def _loop_rows(m: int, cus: int, special) -> np.ndarray:
    """Rows to compare in an n = 32768 loop test: the special rows, the rows the
    same workgroups take next (row + CUs, + 2 CUs), the first and last rows, and
    random ones."""
    rng = np.random.default_rng(m)
    picks = [r + k * cus for r in special for k in (0, 1, 2)]
    return np.unique(np.clip(np.r_[0, 1, m - 2, m - 1, picks, rng.integers(0, m, 96)], 0, m - 1))


@pytest.mark.parametrize("inplace", [False, True], ids=["out", "inplace"])
@pytest.mark.parametrize("dtype", DTYPES)
def test_n32768_loop_nonfinite_rows_between_ordinary_rows(oracle, dtype, inplace):
    """NaN, Inf and zero rows in the persistent n = 32768 loop (4096 + 5 rows, so
    each workgroup takes ~16 rows): nothing carries over to the rows a workgroup
    takes after them."""
    import torch
    n = 1 << 15
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    m = 4096 + 5
    say(f"n=32768 loop nonfinite rows m={m} {dtype} inplace={inplace}")
    bits = W.random_rows(m, n, dtype, seed=3277)
    nan = 0x7E00 if dtype == "fp16" else 0x7FC0
    inf = 0x7C00 if dtype == "fp16" else 0x7F80
    special = [0, 1, 2, cus + 1, cus + 3, 2 * cus, m - 1]
    bits[0, 11] = nan
    bits[cus + 1, 5] = nan
    bits[1, 3] = inf
    bits[2 * cus, 1] = inf | 0x8000
    bits[2] = 0
    bits[cus + 3] = 0
    bits[m - 1, 7] = nan
    s = W.default_scale(n)
    out = _run(bits, dtype, s, n, inplace)
    c = compare_with_oracle(oracle, out, bits, dtype, s, n, rows=_loop_rows(m, cus, special))
    say(f"  {c}")
    assert c.ok, str(c)


@pytest.mark.parametrize("dtype", DTYPES)
def test_n32768_loop_strided_rows_keep_gaps(oracle, dtype):
    """The n = 32768 loop on strided rows (4099 rows, input stride n + 24, output
    stride n + 40): the gaps keep their canaries in both modes, and the rows
    match the oracle and each other."""
    import torch
    n = 1 << 15
    m = 4099
    in_stride, out_stride = n + 24, n + 40
    say(f"n=32768 loop strided {dtype} m={m}")
    bits = W.random_rows(m, n, dtype, seed=3299, stride=in_stride, fill_bits=0x7FC1)
    s = W.default_scale(n)
    out = _run(bits, dtype, s, n, False, out_stride=out_stride, out_fill=0x5A5A)
    assert (out[:, n:] == 0x5A5A).all(), "out-of-place write touched the row gap"
    rows = _loop_rows(m, torch.cuda.get_device_properties(0).multi_processor_count, [3, 4000])
    c = compare_with_oracle(oracle, out, bits, dtype, s, n, rows=rows)
    say(f"  {c}")
    assert c.ok, str(c)
    out2 = _run(bits, dtype, s, n, True)
    assert (out2[:, n:] == 0x7FC1).all(), "in-place write touched the row gap"
    assert np.array_equal(out2[:, :n], out[:, :n])


@pytest.mark.parametrize("dtype,scale", [("bf16", 0.0), ("bf16", -1.0), ("bf16", 1e30), ("fp16", 3.0),
                                         ("fp16", -0.0078125)])
def test_n32768_loop_unusual_scales(oracle, dtype, scale):
    """The n = 32768 loop with scales other than 1/sqrt(n) (zero, negative, far
    from 1): the scale split into the matrix-core operand and the final factor."""
    import torch
    n = 1 << 15
    m = 4096
    say(f"n=32768 loop scale={scale} {dtype}")
    bits = W.random_rows(m, n, dtype, seed=3300)   # N(0,1): |y| * 1e30 stays inside bf16's range
    out = _run(bits, dtype, scale, n, False)
    rows = _loop_rows(m, torch.cuda.get_device_properties(0).multi_processor_count, [7])
    c = compare_with_oracle(oracle, out, bits, dtype, scale, n, rows=rows)
    say(f"  {c}")
    assert c.ok, str(c)


# scales beyond 1/sqrt(n): zero, negative, not a power of two, far from 1 (kept
# where the outputs stay inside the dtype's range, so that the comparison with
# the unrounded oracle is meaningful)
SCALES = {"fp16": [0.0, -1.0, -0.0078125, 3.0, 1e-3], "bf16": [0.0, -1.0, -0.0078125, 3.0, 1e-30, 1e30]}


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("L", [2, 5, 7, 12, 15, 16])
def test_unusual_scales(oracle, L, dtype, variant):
    n = 1 << L
    m = 19
    bits = W.random_rows(m, n, dtype, seed=900 + L)
    for s in SCALES[dtype]:
        s32 = float(np.float32(s))
        out = _run(bits, dtype, s32, n, False)
        c = compare_with_oracle(oracle, out, bits, dtype, s32, n)
        assert c.ok, f"scale {s32}: {c}"


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("L", [0, 2, 5, 7, 8, 11, 12, 13, 15, 16])
def test_single_row(oracle, L, dtype, variant):
    n = 1 << L
    bits = W.random_rows(1, n, dtype, seed=7 + L)
    out = _run(bits, dtype, 0.5, n, False)
    c = compare_with_oracle(oracle, out, bits, dtype, 0.5, n)
    assert c.ok, str(c)


def test_zero_rows_leaves_output_untouched():
    import torch
    x = to_device(np.full((4, 256), 0x3C00, np.uint16), "fp16")
    H.hadamard_transform(x.data_ptr(), x.data_ptr(), 0, 256, H.FP16, 1.0,
                         torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert (to_host(x) == 0x3C00).all()


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("L", [0, 1, 2, 3, 5, 7, 9, 12, 14, 16])
def test_strided_rows_keep_gaps(oracle, L, dtype, variant):
    n = 1 << L
    m = 19
    in_stride, out_stride = n + 24, n + 40
    bits = W.random_rows(m, n, dtype, seed=L, stride=in_stride, fill_bits=0x7FC1)
    s = W.default_scale(n)
    out = _run(bits, dtype, s, n, False, out_stride=out_stride, out_fill=0x5A5A)
    assert (out[:, n:] == 0x5A5A).all(), "out-of-place write touched the row gap"
    c = compare_with_oracle(oracle, out, bits, dtype, s, n)
    assert c.ok, str(c)
    # in place on the strided buffer: gap canaries stay, rows transform
    out2 = _run(bits, dtype, s, n, True)
    assert (out2[:, n:] == 0x7FC1).all(), "in-place write touched the row gap"
    assert np.array_equal(out2[:, :n], out[:, :n])


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("n", [256, 4096, 65536])
def test_large_offsets(oracle, n, dtype):
    """Rows 2^26 elements apart (the largest stride): row offsets past 2^32 bytes."""
    import torch
    m, stride = 40, 1 << 26
    say(f"large offsets {dtype} n={n}: {m} rows, stride 2^26 elements")
    buf = torch.zeros(m * stride, dtype=torch.int16, device="cuda")
    bits = W.random_rows(m, n, dtype, seed=77)
    for i in range(m):
        buf[i * stride:i * stride + n] = torch.from_numpy(bits[i].view(np.int16)).cuda()
    x = buf.view(torch.float16 if dtype == "fp16" else torch.bfloat16)
    s = W.default_scale(n)
    H.hadamard_transform_strided(x.data_ptr(), stride, x.data_ptr(), stride, m, n, CODE[dtype],
                                 s, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    out = np.stack([buf[i * stride:i * stride + n].cpu().numpy().view(np.uint16) for i in range(m)])
    c = compare_with_oracle(oracle, out, bits, dtype, s, n)
    assert c.ok, str(c)
    del buf


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("L", [0, 1, 3, 5, 7, 10, 13, 15, 16])
def test_special_vectors(L, dtype, variant):
    n = 1 << L
    one = W.round_to_bits(np.array([1.0], np.float32), dtype)[0]
    rows = np.zeros((4, n), np.uint16)
    rows[0, 0] = one                       # delta -> all ones
    rows[1, :] = one                       # ones -> n e_0
    k = (n // 2 + 5) % n                   # a Walsh row -> n e_k
    parity = np.array([bin(k & j).count("1") & 1 for j in range(n)])
    rows[2] = W.round_to_bits(np.where(parity == 1, -1.0, 1.0).astype(np.float32), dtype)
    # row 3 stays zero
    s = 2.0 ** -(L // 2)
    out = bits_to_f64(_run(rows, dtype, s, n, False), dtype)
    assert np.array_equal(out[0], np.full(n, s))
    e0 = np.zeros(n)
    e0[0] = n * s
    assert np.array_equal(out[1], e0)
    ek = np.zeros(n)
    ek[k] = n * s
    assert np.array_equal(out[2], ek)
    assert np.array_equal(out[3], np.zeros(n))


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("L", [1, 2, 5, 7, 12, 15, 16])
def test_nonfinite_and_subnormal_inputs(oracle, L, dtype, variant):
    n = 1 << L
    bits = W.random_rows(6, n, dtype, seed=3)
    nan = 0x7E00 if dtype == "fp16" else 0x7FC0
    inf = 0x7C00 if dtype == "fp16" else 0x7F80
    bits[0, n // 3] = nan
    bits[1, 5 % n] = inf
    bits[2, 1] = inf
    bits[2, n - 2] = inf | 0x8000
    # row 3: subnormals only
    rng = np.random.default_rng(5)
    sub = rng.integers(1, 0x3FF if dtype == "fp16" else 0x7F, n).astype(np.uint16)
    bits[3] = sub | (rng.integers(0, 2, n).astype(np.uint16) << 15)
    s = W.default_scale(n)
    out = _run(bits, dtype, s, n, False)
    c = compare_with_oracle(oracle, out, bits, dtype, s, n)
    assert c.ok, str(c)


@pytest.mark.parametrize("L", [7, 12, 15, 16])
def test_bf16_huge_values_do_not_overflow(oracle, L, variant):
    n = 1 << L
    rng = np.random.default_rng(L)
    vals = (rng.choice([-1.0, 1.0], (8, n)) * rng.uniform(1e36, 3e37, (8, n))).astype(np.float32)
    bits = W.round_to_bits(vals, "bf16")
    s = W.default_scale(n)
    out = _run(bits, "bf16", s, n, False)
    assert np.isfinite(bits_to_f64(out, "bf16")).all()
    c = compare_with_oracle(oracle, out, bits, "bf16", s, n)
    assert c.ok, str(c)


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("L", range(0, 17))
def test_deterministic_and_inplace_equals_out_of_place(L, dtype, variant):
    n = 1 << L
    m = 4096 >> max(0, L - 10) if L <= 12 else 9
    bits = W.random_rows(m, n, dtype, seed=L + 50)
    s = W.default_scale(n)
    a = _run(bits, dtype, s, n, False)
    b = _run(bits, dtype, s, n, False)
    c = _run(bits, dtype, s, n, True)
    assert np.array_equal(a, b)
    assert np.array_equal(a, c)


def test_python_wrapper_errors_and_stream():
    import torch
    x = torch.randn(64, 256, device="cuda").to(torch.float16)
    with pytest.raises(TypeError):
        H.transform(x.float())
    with pytest.raises(ValueError):
        H.transform(x.t())
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        y = H.transform(x)
    side.synchronize()
    ref = H.transform(x)
    torch.cuda.synchronize()
    assert torch.equal(y, ref)


def test_stream_copy():
    import torch
    src = torch.randint(-30000, 30000, (1 << 22,), dtype=torch.int16, device="cuda")
    dst = torch.zeros_like(src)
    H.hadacore_stream_copy(src.data_ptr(), dst.data_ptr(), src.numel() * 2,
                           torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert torch.equal(src, dst)


# Output stores take the SC1 cache bit only where every store writes whole
# 128-byte lines (output 128-byte aligned, rows contiguous or 128-byte pitched);
# elsewhere plain nontemporal stores.  The two paths must give the same bytes
# and write nothing outside the output.
ALIGN_CASES = [(2, "bf16", 4099), (4, "bf16", 4099), (8, "fp16", 4099), (32, "bf16", 1001), (128, "bf16", 1001),
               (128, "fp16", 64), (1024, "fp16", 37), (4096, "bf16", 37), (8192, "bf16", 21),
               (16384, "bf16", 5)]


@pytest.mark.parametrize("n,dtype,m", ALIGN_CASES)
def test_output_alignment_picks_store_path_not_result(oracle, n, dtype, m):
    import torch
    s = W.default_scale(n)
    bits = W.random_rows(m, n, dtype, seed=n + m)
    x = to_device(bits, dtype)
    outs = {}
    for off in (0, 16, 64):  # bytes past a 256-byte aligned allocation
        pad = 256 // 2
        buf = torch.full((pad + m * n + pad,), -1, dtype=torch.int16, device="cuda")
        out = buf[pad + off // 2: pad + off // 2 + m * n]
        H.hadamard_transform(x.data_ptr(), out.data_ptr(), m, n, CODE[dtype], s,
                             torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        host = buf.cpu().numpy()
        lo, hi = pad + off // 2, pad + off // 2 + m * n
        assert (host[:lo] == -1).all() and (host[hi:] == -1).all(), f"write outside the output (offset {off})"
        outs[off] = host[lo:hi].copy()
    assert np.array_equal(outs[0], outs[16]) and np.array_equal(outs[0], outs[64])
    c = compare_with_oracle(oracle, outs[0].view(np.uint16).reshape(m, n), bits, dtype, s, n)
    say(f"  n={n} {dtype} m={m}: {c}")
    assert c.ok, str(c)


@pytest.mark.parametrize("n,m", [(1, 4099), (2, 4099), (4, 4099), (8, 4099), (128, 1001), (16384, 5)])
@pytest.mark.parametrize("fmt", ["fp8", "int8"])
def test_code_and_scale_alignment_picks_store_path_not_result(n, m, fmt):
    import torch
    s = W.default_scale(n)
    bits = W.random_rows(m, n, "bf16", seed=3 * n + m)
    x = to_device(bits, "bf16")
    fn = H.hadamard_transform_fp8 if fmt == "fp8" else H.hadamard_transform_int8
    got = []
    for coff, soff in ((0, 0), (16, 4), (64, 16)):
        cbuf = torch.full((256 + m * n + 256,), 0x5A, dtype=torch.uint8, device="cuda")
        sbuf = torch.full((64 + m + 64,), -7.0, dtype=torch.float32, device="cuda")
        codes = cbuf[256 + coff: 256 + coff + m * n]
        scales = sbuf[64 + soff // 4: 64 + soff // 4 + m]
        fn(x.data_ptr(), n, codes.data_ptr(), n, scales.data_ptr(), m, n, H.BF16, s,
           torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        ch, sh = cbuf.cpu().numpy(), sbuf.cpu().numpy()
        c0, s0 = 256 + coff, 64 + soff // 4
        assert (ch[:c0] == 0x5A).all() and (ch[c0 + m * n:] == 0x5A).all()
        assert (sh[:s0] == -7.0).all() and (sh[s0 + m:] == -7.0).all()
        got.append((ch[c0:c0 + m * n].copy(), sh[s0:s0 + m].view(np.uint32).copy()))
    for c, sc in got[1:]:
        assert np.array_equal(c, got[0][0]) and np.array_equal(sc, got[0][1])


def test_stream_copy_unaligned_destination():
    import torch
    src = torch.randint(-30000, 30000, (1 << 20,), dtype=torch.int16, device="cuda")
    for off in (0, 8, 32):  # 16-bit elements: 0, 16 and 64 bytes
        buf = torch.full((src.numel() + 256,), 7, dtype=torch.int16, device="cuda")
        dst = buf[128 + off: 128 + off + src.numel()]
        H.hadacore_stream_copy(src.data_ptr(), dst.data_ptr(), src.numel() * 2,
                               torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        assert torch.equal(src, dst)
        assert (buf[:128 + off] == 7).all() and (buf[128 + off + src.numel():] == 7).all()
