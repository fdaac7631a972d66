"""fp64 CPU oracle for the batched normalized Walsh-Hadamard transform.

TEST INFRASTRUCTURE ONLY.  The product path (``paper_2412_08832_amd``) never
imports this package; only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may.  It shares nothing with the HIP library:
the arithmetic lives in ``fwht_oracle.c`` (plain C11, fp64), this module only
compiles it with gcc and marshals numpy arrays through ctypes.

What is computed (paper Sec. 2.1-2.2): for an m x n matrix of fp16/bf16 rows,
``y[i, j] = s * sum_k (-1)**popcount(j & k) * x[i, k]``, i.e. ``x @ H_n * s``
with ``H_n`` the Sylvester-ordered Walsh-Hadamard matrix.  ``fwht`` follows the
iterative radix-2 algorithm of Sec. 2.2; ``fwht_direct`` evaluates the plain
definition one output at a time; ``fwht_fp8`` and ``fwht_int8`` add per-row
FP8 (e4m3) or symmetric INT8 quantization of the transformed rows (the fused
transform + quantization the paper names as future work, Sec. 5).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from pathlib import Path

import numpy as np

HERE = Path(__file__).resolve().parent
SOURCE = HERE / "fwht_oracle.c"
LIBRARY = HERE / "liboracle_fwht.so"

FP16 = 0
BF16 = 1
DTYPES = {"fp16": FP16, "bf16": BF16}


def compile_library(source: Path = SOURCE, output: Path = LIBRARY) -> Path:
    """Compile the oracle C source into a shared library with gcc (-O2, no fast-math)."""
    tmp = output.with_name(output.name + f".tmp{os.getpid()}")
    cmd = ["gcc", "-std=c11", "-O2", "-fPIC", "-shared", "-pthread", "-Wall", "-Wextra",
           "-fno-fast-math", str(source), "-o", str(tmp), "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, output)
    return output


def build() -> Path:
    """Compile the oracle library in place (always recompiles)."""
    return compile_library()


def _dtype_code(dtype) -> int:
    if isinstance(dtype, str):
        return DTYPES[dtype]
    if dtype in (FP16, BF16):
        return int(dtype)
    raise ValueError(f"unknown dtype {dtype!r}")


class Oracle:
    """ctypes view of one compiled oracle library (the default one, or a test mutant)."""

    def __init__(self, path: Path | str = LIBRARY):
        self.path = Path(path)
        lib = ctypes.CDLL(str(self.path))
        u16p = ctypes.POINTER(ctypes.c_uint16)
        f64p = ctypes.POINTER(ctypes.c_double)
        i64p = ctypes.POINTER(ctypes.c_int64)
        i64 = ctypes.c_int64
        lib.oracle_decode_fp16.argtypes = [ctypes.c_uint16]
        lib.oracle_decode_fp16.restype = ctypes.c_double
        lib.oracle_decode_bf16.argtypes = [ctypes.c_uint16]
        lib.oracle_decode_bf16.restype = ctypes.c_double
        lib.oracle_fwht_vec_f64.argtypes = [f64p, i64]
        lib.oracle_fwht_vec_f64.restype = None
        lib.oracle_decode_rows.argtypes = [u16p, i64, i64, i64, ctypes.c_int, f64p]
        lib.oracle_decode_rows.restype = ctypes.c_int
        lib.oracle_fwht_f64.argtypes = [u16p, i64, i64, i64, ctypes.c_int, ctypes.c_double,
                                        f64p, ctypes.c_int]
        lib.oracle_fwht_f64.restype = ctypes.c_int
        lib.oracle_fwht_direct_f64.argtypes = [u16p, i64, i64, ctypes.c_int, ctypes.c_double,
                                               i64p, i64p, i64, f64p]
        lib.oracle_fwht_direct_f64.restype = ctypes.c_int
        u8p = ctypes.POINTER(ctypes.c_uint8)
        f32p = ctypes.POINTER(ctypes.c_float)
        lib.oracle_decode_e4m3.argtypes = [ctypes.c_uint8]
        lib.oracle_decode_e4m3.restype = ctypes.c_double
        lib.oracle_encode_e4m3.argtypes = [ctypes.c_float]
        lib.oracle_encode_e4m3.restype = ctypes.c_uint8
        lib.oracle_fwht_fp8.argtypes = [u16p, i64, i64, i64, ctypes.c_int, ctypes.c_double, u8p,
                                        i64, f32p]
        lib.oracle_fwht_fp8.restype = ctypes.c_int
        i8p = ctypes.POINTER(ctypes.c_int8)
        lib.oracle_encode_int8.argtypes = [ctypes.c_float]
        lib.oracle_encode_int8.restype = ctypes.c_int8
        lib.oracle_fwht_int8.argtypes = [u16p, i64, i64, i64, ctypes.c_int, ctypes.c_double, i8p,
                                         i64, f32p]
        lib.oracle_fwht_int8.restype = ctypes.c_int
        lib.oracle_quantize_fp8.argtypes = [f32p, i64, i64, u8p, f32p]
        lib.oracle_quantize_fp8.restype = ctypes.c_int
        lib.oracle_quantize_int8.argtypes = [f32p, i64, i64, i8p, f32p]
        lib.oracle_quantize_int8.restype = ctypes.c_int
        self.lib = lib

    # -- decoders ---------------------------------------------------------
    def decode(self, bits: np.ndarray, dtype) -> np.ndarray:
        """Exact decode of a 2-D (or 1-D) uint16 array of fp16/bf16 bit patterns to float64."""
        bits = np.ascontiguousarray(bits, dtype=np.uint16)
        shape = bits.shape
        flat = bits.reshape(1, -1) if bits.ndim != 2 else bits
        m, n = flat.shape
        out = np.empty((m, n), dtype=np.float64)
        rc = self.lib.oracle_decode_rows(_u16(flat), n, m, n, _dtype_code(dtype), _f64(out))
        if rc:
            raise ValueError("oracle_decode_rows rejected its arguments")
        return out.reshape(shape)

    # -- transforms ---------------------------------------------------------
    def fwht_vec(self, v: np.ndarray) -> np.ndarray:
        """Unscaled FWHT of float64 rows (last axis), returned as a new array."""
        out = np.array(v, dtype=np.float64, copy=True, order="C")
        rows = out.reshape(-1, out.shape[-1])
        n = rows.shape[1]
        for r in range(rows.shape[0]):
            self.lib.oracle_fwht_vec_f64(_f64(rows[r]), n)
        return out

    def fwht(self, bits: np.ndarray, dtype, scale: float, n: int | None = None,
             nthreads: int = 1) -> np.ndarray:
        """y = scale * x @ H_n per row of a 2-D uint16 array (row stride = bits.shape[1]).

        When ``n`` is given and smaller than the row stride, only the first ``n``
        columns of each row are transformed (strided rows).
        """
        bits = np.ascontiguousarray(bits, dtype=np.uint16)
        if bits.ndim != 2:
            raise ValueError("expected a 2-D array of bit patterns")
        m, stride = bits.shape
        n = stride if n is None else int(n)
        out = np.empty((m, n), dtype=np.float64)
        rc = self.lib.oracle_fwht_f64(_u16(bits), stride, m, n, _dtype_code(dtype),
                                      float(scale), _f64(out), int(nthreads))
        if rc:
            raise ValueError("oracle_fwht_f64 rejected its arguments")
        return out

    def fwht_direct(self, bits: np.ndarray, dtype, scale: float, rows, cols,
                    n: int | None = None) -> np.ndarray:
        """The plain definition at selected (row, col) outputs."""
        bits = np.ascontiguousarray(bits, dtype=np.uint16)
        m, stride = bits.shape
        n = stride if n is None else int(n)
        rows = np.ascontiguousarray(rows, dtype=np.int64)
        cols = np.ascontiguousarray(cols, dtype=np.int64)
        if rows.shape != cols.shape:
            raise ValueError("rows and cols must have the same shape")
        if rows.size and (rows.min() < 0 or rows.max() >= m):
            raise ValueError("row index out of range")
        out = np.empty(rows.shape, dtype=np.float64)
        rc = self.lib.oracle_fwht_direct_f64(_u16(bits), stride, n, _dtype_code(dtype),
                                             float(scale), _i64(rows), _i64(cols), rows.size,
                                             _f64(out))
        if rc:
            raise ValueError("oracle_fwht_direct_f64 rejected its arguments")
        return out

    # -- fused transform + FP8 quantization ----------------------------------
    def encode_e4m3(self, values) -> np.ndarray:
        """OCP e4m3 codes (round-to-nearest-even) of float32 values."""
        v = np.asarray(values, dtype=np.float32)
        f = self.lib.oracle_encode_e4m3
        return np.fromiter((f(float(x)) for x in v.ravel()), dtype=np.uint8,
                           count=v.size).reshape(v.shape)

    def decode_e4m3(self, codes) -> np.ndarray:
        """Exact values of OCP e4m3 codes."""
        c = np.asarray(codes, dtype=np.uint8)
        table = np.array([self.lib.oracle_decode_e4m3(i) for i in range(256)], dtype=np.float64)
        return table[c]

    def fwht_fp8(self, bits: np.ndarray, dtype, scale: float, n: int | None = None):
        """Fused transform + per-row e4m3 quantization: (codes (m, n) uint8, scales (m,) float32)."""
        bits = np.ascontiguousarray(bits, dtype=np.uint16)
        m, stride = bits.shape
        n = stride if n is None else int(n)
        codes = np.empty((m, n), dtype=np.uint8)
        scales = np.empty(m, dtype=np.float32)
        rc = self.lib.oracle_fwht_fp8(_u16(bits), stride, m, n, _dtype_code(dtype), float(scale),
                                      _u8(codes), n, _f32(scales))
        if rc:
            raise ValueError("oracle_fwht_fp8 rejected its arguments")
        return codes, scales

    # -- fused transform + INT8 quantization ---------------------------------
    def encode_int8(self, values) -> np.ndarray:
        """Round-half-to-even of float32 values to int8, saturated to [-127, 127]."""
        v = np.asarray(values, dtype=np.float32)
        f = self.lib.oracle_encode_int8
        return np.fromiter((f(float(x)) for x in v.ravel()), dtype=np.int8,
                           count=v.size).reshape(v.shape)

    def fwht_int8(self, bits: np.ndarray, dtype, scale: float, n: int | None = None):
        """Fused transform + per-row symmetric INT8 quantization: (codes (m, n) int8,
        scales (m,) float32)."""
        bits = np.ascontiguousarray(bits, dtype=np.uint16)
        m, stride = bits.shape
        n = stride if n is None else int(n)
        codes = np.empty((m, n), dtype=np.int8)
        scales = np.empty(m, dtype=np.float32)
        rc = self.lib.oracle_fwht_int8(_u16(bits), stride, m, n, _dtype_code(dtype), float(scale),
                                       _i8(codes), n, _f32(scales))
        if rc:
            raise ValueError("oracle_fwht_int8 rejected its arguments")
        return codes, scales

    # -- the same quantizers on plain fp32 rows (no transform) ----------------
    def quantize_fp8(self, rows: np.ndarray):
        """Per-row e4m3 quantization of a 2-D float32 array: (codes uint8, scales float32)."""
        y = np.ascontiguousarray(rows, dtype=np.float32)
        m, n = y.shape
        codes = np.empty((m, n), dtype=np.uint8)
        scales = np.empty(m, dtype=np.float32)
        if self.lib.oracle_quantize_fp8(_f32(y), m, n, _u8(codes), _f32(scales)):
            raise ValueError("oracle_quantize_fp8 rejected its arguments")
        return codes, scales

    def quantize_int8(self, rows: np.ndarray):
        """Per-row symmetric INT8 quantization of a 2-D float32 array: (codes int8, scales)."""
        y = np.ascontiguousarray(rows, dtype=np.float32)
        m, n = y.shape
        codes = np.empty((m, n), dtype=np.int8)
        scales = np.empty(m, dtype=np.float32)
        if self.lib.oracle_quantize_int8(_f32(y), m, n, _i8(codes), _f32(scales)):
            raise ValueError("oracle_quantize_int8 rejected its arguments")
        return codes, scales


def _i8(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int8))


def _u8(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8))


def _f32(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_float))


def _u16(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_uint16))


def _f64(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _i64(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))


_DEFAULT: Oracle | None = None


def get() -> Oracle:
    """The oracle built from ``fwht_oracle.c`` (compiled on first use if missing or stale)."""
    global _DEFAULT
    if _DEFAULT is None:
        if not LIBRARY.exists() or LIBRARY.stat().st_mtime < SOURCE.stat().st_mtime:
            compile_library()
        _DEFAULT = Oracle(LIBRARY)
    return _DEFAULT
