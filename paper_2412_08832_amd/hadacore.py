"""ctypes binding of libhadacore (``include/hadacore.h``).

Argument marshalling only: every step of the transform runs in the HIP
kernels of ``libhadacore.so``.  The library is loaded from this package
directory; if it is missing, every call raises (there is no fallback).

The raw entry points take device addresses as integers and keep the C names:
``hadamard_transform``, ``hadamard_transform_strided``, ``hadamard_transform_ws``,
``hadamard_transform_ws_noalloc``, ``hadamard_transform_workspace_size``, ``hadamard_transform_fp8``,
``hadamard_transform_int8``, ``hadacore_stream_copy``, ``hadacore_status_string``,
``hadacore_version``.  ``transform``, ``transform_fp8`` and ``transform_int8`` are
convenience wrappers for 2-D torch tensors on a ROCm device.
"""
from __future__ import annotations

import ctypes
import math
from pathlib import Path

LIBRARY = Path(__file__).resolve().parent / "libhadacore.so"

FP16 = 0
BF16 = 1
SUCCESS = 0
STATUS_NAMES = {
    0: "SUCCESS", 1: "INVALID_VALUE", 2: "INVALID_SIZE", 3: "INVALID_DTYPE",
    4: "INVALID_STRIDE", 5: "MISALIGNED", 6: "OVERLAP", 7: "LAUNCH",
    8: "UNSUPPORTED_DEVICE", 9: "TOO_LARGE", 10: "WORKSPACE", 11: "SCRATCH",
}
NOALLOC_SCRATCH_BYTES = 32 << 20  # HADACORE_NOALLOC_SCRATCH_BYTES
EXPORTS = ("hadamard_transform", "hadamard_transform_strided", "hadamard_transform_ws",
           "hadamard_transform_ws_noalloc", "hadamard_transform_workspace_size", "hadamard_transform_fp8",
           "hadamard_transform_int8", "hadacore_stream_copy", "hadacore_status_string",
           "hadacore_version")


class HadacoreError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {STATUS_NAMES.get(status, status)} "
                         f"({hadacore_status_string(status)})")


_lib = None


def _load_torch_runtime() -> None:
    """Import torch, if it is installed, before the library is loaded.

    The device pointers and streams passed to the library come from torch, which
    ships its own copy of the HIP runtime.  libhadacore.so needs libamdhip64.so.7:
    if torch's copy is already loaded, that need is met by it; if the library were
    loaded first, the dynamic loader would map the system ROCm runtime instead and
    torch would then map its own, leaving two runtimes in one process -- the
    library's would see none of torch's memory or streams (and reports no device).
    """
    try:
        import torch  # noqa: F401
    except ImportError:
        pass


def library() -> ctypes.CDLL:
    """The loaded libhadacore.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not LIBRARY.exists():
            raise RuntimeError(f"{LIBRARY} is missing: build it with "
                               "`python -m paper_2412_08832_amd.build`")
        _load_torch_runtime()
        lib = ctypes.CDLL(str(LIBRARY))
        i64, vp, f32, i32 = ctypes.c_int64, ctypes.c_void_p, ctypes.c_float, ctypes.c_int32
        lib.hadamard_transform.argtypes = [vp, vp, i64, i64, i32, f32, vp]
        lib.hadamard_transform.restype = i32
        lib.hadamard_transform_strided.argtypes = [vp, i64, vp, i64, i64, i64, i32, f32, vp]
        lib.hadamard_transform_strided.restype = i32
        lib.hadamard_transform_ws.argtypes = [vp, i64, vp, i64, i64, i64, i32, f32, vp, i64, vp]
        lib.hadamard_transform_ws.restype = i32
        lib.hadamard_transform_ws_noalloc.argtypes = [vp, i64, vp, i64, i64, i64, i32, f32, vp]
        lib.hadamard_transform_ws_noalloc.restype = i32
        lib.hadamard_transform_workspace_size.argtypes = [i64, i64]
        lib.hadamard_transform_workspace_size.restype = i64
        lib.hadamard_transform_fp8.argtypes = [vp, i64, vp, i64, vp, i64, i64, i32, f32, vp]
        lib.hadamard_transform_fp8.restype = i32
        lib.hadamard_transform_int8.argtypes = [vp, i64, vp, i64, vp, i64, i64, i32, f32, vp]
        lib.hadamard_transform_int8.restype = i32
        lib.hadacore_stream_copy.argtypes = [vp, vp, i64, vp]
        lib.hadacore_stream_copy.restype = i32
        lib.hadacore_status_string.argtypes = [i32]
        lib.hadacore_status_string.restype = ctypes.c_char_p
        lib.hadacore_version.argtypes = []
        lib.hadacore_version.restype = i32
        _lib = lib
    return _lib


def _check(status: int, where: str) -> None:
    if status != SUCCESS:
        raise HadacoreError(status, where)


def hadamard_transform(in_ptr: int, out_ptr: int, m: int, n: int, dtype: int, scale: float,
                       stream: int = 0, check: bool = True) -> int:
    st = library().hadamard_transform(in_ptr, out_ptr, m, n, dtype, scale, stream)
    if check:
        _check(st, "hadamard_transform")
    return st


def hadamard_transform_strided(in_ptr: int, in_row_stride: int, out_ptr: int,
                               out_row_stride: int, m: int, n: int, dtype: int, scale: float,
                               stream: int = 0, check: bool = True) -> int:
    st = library().hadamard_transform_strided(in_ptr, in_row_stride, out_ptr, out_row_stride,
                                              m, n, dtype, scale, stream)
    if check:
        _check(st, "hadamard_transform_strided")
    return st


def hadamard_transform_ws(in_ptr: int, in_row_stride: int, out_ptr: int, out_row_stride: int,
                          m: int, n: int, dtype: int, scale: float, workspace_ptr: int,
                          workspace_bytes: int, stream: int = 0, check: bool = True) -> int:
    st = library().hadamard_transform_ws(in_ptr, in_row_stride, out_ptr, out_row_stride, m, n,
                                         dtype, scale, workspace_ptr, workspace_bytes, stream)
    if check:
        _check(st, "hadamard_transform_ws")
    return st


def hadamard_transform_ws_noalloc(in_ptr: int, in_row_stride: int, out_ptr: int,
                                  out_row_stride: int, m: int, n: int, dtype: int, scale: float,
                                  stream: int = 0, check: bool = True) -> int:
    st = library().hadamard_transform_ws_noalloc(in_ptr, in_row_stride, out_ptr, out_row_stride,
                                                 m, n, dtype, scale, stream)
    if check:
        _check(st, "hadamard_transform_ws_noalloc")
    return st


def hadamard_transform_workspace_size(m: int, n: int) -> int:
    return int(library().hadamard_transform_workspace_size(m, n))


def hadamard_transform_fp8(in_ptr: int, in_row_stride: int, codes_ptr: int, codes_row_stride: int,
                           scales_ptr: int, m: int, n: int, dtype: int, scale: float,
                           stream: int = 0, check: bool = True) -> int:
    st = library().hadamard_transform_fp8(in_ptr, in_row_stride, codes_ptr, codes_row_stride,
                                          scales_ptr, m, n, dtype, scale, stream)
    if check:
        _check(st, "hadamard_transform_fp8")
    return st


def hadamard_transform_int8(in_ptr: int, in_row_stride: int, codes_ptr: int,
                            codes_row_stride: int, scales_ptr: int, m: int, n: int, dtype: int,
                            scale: float, stream: int = 0, check: bool = True) -> int:
    st = library().hadamard_transform_int8(in_ptr, in_row_stride, codes_ptr, codes_row_stride,
                                           scales_ptr, m, n, dtype, scale, stream)
    if check:
        _check(st, "hadamard_transform_int8")
    return st


def hadacore_stream_copy(src_ptr: int, dst_ptr: int, nbytes: int, stream: int = 0,
                         check: bool = True) -> int:
    st = library().hadacore_stream_copy(src_ptr, dst_ptr, nbytes, stream)
    if check:
        _check(st, "hadacore_stream_copy")
    return st


def hadacore_status_string(status: int) -> str:
    return library().hadacore_status_string(status).decode()


def hadacore_version() -> int:
    return int(library().hadacore_version())


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.float16:
        return FP16
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"expected float16 or bfloat16, got {t.dtype}")


def transform(x, out=None, scale: float | None = None, n: int | None = None, stream=None,
              workspace=None):
    """out = scale * x @ H_n over the first ``n`` columns of each row of a 2-D tensor.

    ``x`` and ``out`` are 2-D float16/bfloat16 ROCm tensors with unit column
    stride; ``out=None`` allocates a new tensor, ``out=x`` runs in place.  The
    default scale is fp32(1/sqrt(n)); the default stream is torch's current one.
    n above 2^16 runs through ``hadamard_transform_ws``; ``workspace`` (a
    contiguous ROCm tensor of at least hadamard_transform_workspace_size(m, n)
    bytes) is allocated here when not given.
    """
    import torch
    if x.dim() != 2 or not x.is_cuda:
        raise ValueError("expected a 2-D tensor on a ROCm device")
    if x.stride(1) != 1:
        raise ValueError("rows must be contiguous (column stride 1)")
    code = _dtype_code(x)
    n = x.shape[1] if n is None else int(n)
    if out is None:
        out = torch.empty((x.shape[0], n), dtype=x.dtype, device=x.device)
    if out.dtype != x.dtype or out.device != x.device or out.dim() != 2 or out.stride(1) != 1:
        raise ValueError("out must be a 2-D tensor of the same dtype/device with column stride 1")
    if out.shape[0] != x.shape[0] or out.shape[1] < n or x.shape[1] < n:
        raise ValueError("shape mismatch between x, out and n")
    if scale is None:
        scale = float(ctypes.c_float(1.0 / math.sqrt(n)).value)
    if stream is None:
        stream = torch.cuda.current_stream(x.device).cuda_stream
    elif hasattr(stream, "cuda_stream"):
        stream = stream.cuda_stream
    # a single row's stride is never used to address anything; report n
    in_stride = x.stride(0) if x.shape[0] > 1 else n
    out_stride = out.stride(0) if out.shape[0] > 1 else n
    with torch.cuda.device(x.device):
        if n > 1 << 16:
            need = hadamard_transform_workspace_size(x.shape[0], n)
            if workspace is None:
                workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=x.device)
            wbytes = workspace.numel() * workspace.element_size()
            hadamard_transform_ws(x.data_ptr(), in_stride, out.data_ptr(), out_stride,
                                  x.shape[0], n, code, scale, workspace.data_ptr(), wbytes,
                                  stream)
        else:
            hadamard_transform_strided(x.data_ptr(), in_stride, out.data_ptr(), out_stride,
                                       x.shape[0], n, code, scale, stream)
    return out


def _transform_quantized(x, codes, scales, scale, stream, entry, codes_dtype):
    import torch
    if x.dim() != 2 or not x.is_cuda or x.stride(1) != 1:
        raise ValueError("expected a 2-D ROCm tensor with contiguous rows")
    code = _dtype_code(x)
    m, n = x.shape
    if codes is None:
        codes = torch.empty((m, n), dtype=codes_dtype, device=x.device)
    if scales is None:
        scales = torch.empty((m,), dtype=torch.float32, device=x.device)
    if codes.dtype != codes_dtype or codes.dim() != 2 or codes.stride(1) != 1 \
            or tuple(codes.shape) != (m, n):
        raise ValueError(f"codes must be a (m, n) {codes_dtype} tensor with contiguous rows")
    if scales.dtype != torch.float32 or scales.numel() != m or not scales.is_contiguous():
        raise ValueError("scales must be a contiguous float32 tensor of m elements")
    if scale is None:
        scale = float(ctypes.c_float(1.0 / math.sqrt(n)).value)
    if stream is None:
        stream = torch.cuda.current_stream(x.device).cuda_stream
    elif hasattr(stream, "cuda_stream"):
        stream = stream.cuda_stream
    in_stride = x.stride(0) if m > 1 else n
    codes_stride = codes.stride(0) if m > 1 else ((n + 15) // 16) * 16
    with torch.cuda.device(x.device):
        entry(x.data_ptr(), in_stride, codes.data_ptr(), codes_stride, scales.data_ptr(), m, n,
              code, scale, stream)
    return codes, scales


def transform_fp8(x, codes=None, scales=None, scale: float | None = None, stream=None):
    """Fused transform + per-row e4m3 quantization of a 2-D float16/bfloat16 tensor.

    Returns (codes, scales): codes is a (m, n) torch.uint8 tensor of e4m3 bit
    patterns and scales a (m,) float32 tensor, so that
    x @ H_n * scale ~ codes.view(torch.float8_e4m3fn).float() * scales[:, None].
    """
    import torch
    return _transform_quantized(x, codes, scales, scale, stream, hadamard_transform_fp8,
                                torch.uint8)


def transform_int8(x, codes=None, scales=None, scale: float | None = None, stream=None):
    """Fused transform + symmetric per-row INT8 quantization of a 2-D float16/bfloat16
    tensor.  Returns (codes, scales): a (m, n) torch.int8 tensor and a (m,) float32
    tensor, so that x @ H_n * scale ~ codes.float() * scales[:, None].
    """
    import torch
    return _transform_quantized(x, codes, scales, scale, stream, hadamard_transform_int8,
                                torch.int8)
