"""The C ABI on the CPU: the library loads, exports what the header declares,
and rejects bad arguments synchronously, before any HIP call.

No call here passes arguments that validation would accept: on a GPU machine
that would launch a kernel on fake pointers.
"""
from __future__ import annotations

import math
import re
import subprocess
from pathlib import Path

import pytest

from paper_2412_08832_amd import hadacore as H

ROOT = Path(__file__).resolve().parent.parent
HEADER = ROOT / "include" / "hadacore.h"

# fake, never-dereferenced device addresses (16-byte aligned, far apart)
A = 1 << 32
B = 1 << 33

# A mistaken case here that validation accepted would launch a kernel on the fake
# addresses above; on a machine with a GPU that faults, so these run GPU-less only.
cpu_only = pytest.mark.skipif(Path("/dev/kfd").exists(),
                                reason="fake-pointer validation tests run only without a GPU")


def _declared_functions() -> set[str]:
    text = re.sub(r"/\*.*?\*/", "", HEADER.read_text(), flags=re.S)
    return set(re.findall(r"^\s*[A-Za-z_][\w\s\*]*?\b([a-z_][a-z0-9_]*)\s*\(", text, flags=re.M))


def _header_defines() -> dict[str, int]:
    return {k: int(v) for k, v in re.findall(r"#define\s+(HADACORE_\w+)\s+(\d+)", HEADER.read_text())}


def test_library_exports_every_declared_function():
    declared = _declared_functions()
    assert declared == set(H.EXPORTS)
    nm = subprocess.run(["nm", "-D", "--defined-only", str(H.LIBRARY)], capture_output=True,
                        text=True, check=True).stdout
    exported = set(re.findall(r"\bT\s+(\w+)$", nm, flags=re.M))
    missing = declared - exported
    assert not missing, f"declared but not exported: {missing}"
    lib = H.library()
    for name in declared:
        assert hasattr(lib, name)


def test_binding_constants_match_header():
    d = _header_defines()
    assert H.hadacore_version() == d["HADACORE_VERSION"]
    assert d["HADACORE_FP16"] == H.FP16 and d["HADACORE_BF16"] == H.BF16
    for code, name in H.STATUS_NAMES.items():
        key = "HADACORE_SUCCESS" if name == "SUCCESS" else f"HADACORE_ERROR_{name}"
        assert d[key] == code


def test_status_strings():
    for code in H.STATUS_NAMES:
        s = H.hadacore_status_string(code)
        assert s and s != "unknown status"
    assert H.hadacore_status_string(99) == "unknown status"


def _st(*args):
    return H.hadamard_transform_strided(*args, check=False)


@cpu_only
@pytest.mark.parametrize("n", [0, 3, 6, 100, 127, 129, 3 * 1024, 3 << 15, 1 << 17, -128])
def test_invalid_size(n):
    assert _st(A, 1 << 17, B, 1 << 17, 4, n, H.FP16, 1.0, 0) == 2


@cpu_only
@pytest.mark.parametrize("dtype", [-1, 2, 7])
def test_invalid_dtype(dtype):
    assert _st(A, 128, B, 128, 4, 128, dtype, 1.0, 0) == 3


@cpu_only
def test_invalid_values():
    assert _st(A, 128, B, 128, -1, 128, H.FP16, 1.0, 0) == 1
    assert _st(0, 128, B, 128, 4, 128, H.FP16, 1.0, 0) == 1
    assert _st(A, 128, 0, 128, 4, 128, H.BF16, 1.0, 0) == 1
    for bad in (math.nan, math.inf, -math.inf):
        assert _st(A, 128, B, 128, 4, 128, H.FP16, bad, 0) == 1


@cpu_only
def test_invalid_strides():
    assert _st(A, 120, B, 128, 4, 128, H.FP16, 1.0, 0) == 4     # in stride < n
    assert _st(A, 128, B, 64, 4, 128, H.FP16, 1.0, 0) == 4      # out stride < n
    assert _st(A, 132, B, 128, 4, 128, H.FP16, 1.0, 0) == 4     # not a multiple of 8
    assert _st(A, 20, B, 16, 4, 16, H.FP16, 1.0, 0) == 4        # n = 16: multiple of 8
    assert _st(A, 6, B, 4, 4, 4, H.FP16, 1.0, 0) == 4           # n = 4: multiple of 4
    assert _st(A, 2, B, 3, 4, 2, H.BF16, 1.0, 0) == 4           # n = 2: multiple of 2
    big = (1 << 26) + 8                                          # above the 2^26 stride limit
    assert _st(A, big, B, 128, 4, 128, H.FP16, 1.0, 0) == 4
    assert _st(A, 128, B, big, 4, 128, H.BF16, 1.0, 0) == 4
    assert _st(A, big, A, big, 4, 128, H.BF16, 1.0, 0) == 4     # in place too


@cpu_only
def test_misaligned_pointers():
    assert _st(A + 2, 128, B, 128, 4, 128, H.FP16, 1.0, 0) == 5
    assert _st(A, 128, B + 8, 128, 4, 128, H.BF16, 1.0, 0) == 5


@cpu_only
def test_overlap_rules():
    # out starts inside in's rows
    assert _st(A, 128, A + 2 * 128, 128, 4, 128, H.FP16, 1.0, 0) == 6
    # same pointer, different strides: not the in-place layout
    assert _st(A, 256, A, 128, 4, 128, H.FP16, 1.0, 0) == 6
    # interleaved rows: in uses columns 0..127, out 128..255 of a 256-wide buffer
    assert _st(A, 256, A + 256, 256, 4, 128, H.FP16, 1.0, 0) == 6


@cpu_only
def test_zero_rows_is_a_no_op():
    assert _st(0, 128, 0, 128, 0, 128, H.FP16, 1.0, 0) == 0
    assert H.hadamard_transform(0, 0, 0, 4096, H.BF16, 0.5, 0, check=False) == 0


@cpu_only
def test_too_large():
    assert _st(A, 128, B, 128, 1 << 31, 128, H.FP16, 1.0, 0) == 9


@cpu_only
def test_unstrided_entry_validates_the_same():
    assert H.hadamard_transform(A, B, 4, 96, H.FP16, 1.0, 0, check=False) == 2
    assert H.hadamard_transform(A + 4, B, 4, 128, H.FP16, 1.0, 0, check=False) == 5


@cpu_only
def test_stream_copy_validation():
    assert H.hadacore_stream_copy(A, B, 17, 0, check=False) == 1
    assert H.hadacore_stream_copy(A, B, -16, 0, check=False) == 1
    assert H.hadacore_stream_copy(A, B, 0, 0, check=False) == 0
    assert H.hadacore_stream_copy(0, B, 32, 0, check=False) == 1
    assert H.hadacore_stream_copy(A + 8, B, 32, 0, check=False) == 5
    assert H.hadacore_stream_copy(A, A + 16, 64, 0, check=False) == 6


@cpu_only
def test_errors_raise_in_python():
    with pytest.raises(H.HadacoreError) as e:
        H.hadamard_transform(A, B, 4, 100, H.FP16, 1.0, 0)
    assert e.value.status == 2


C8 = 1 << 34   # fake codes buffer
S8 = 1 << 35   # fake scales buffer
QUANTIZED = {"fp8": "hadamard_transform_fp8", "int8": "hadamard_transform_int8"}


@cpu_only
@pytest.mark.parametrize("fmt", sorted(QUANTIZED))
def test_quantized_validation(fmt):
    entry = getattr(H, QUANTIZED[fmt])

    def _fp8(*args):
        return entry(*args, check=False)

    ok_args = (A, 128, C8, 128, S8, 4, 128, H.BF16, 1.0, 0)
    assert _fp8(A, 128, C8, 128, S8, 4, 100, H.BF16, 1.0, 0) == 2          # size
    assert _fp8(A, 1 << 17, C8, 1 << 17, S8, 4, 1 << 17, H.BF16, 1.0, 0) == 2  # above 2^16
    assert _fp8(A, 128, C8, 128, S8, 4, 128, 5, 1.0, 0) == 3                # dtype
    assert _fp8(A, 128, C8, 136, S8, 4, 128, H.BF16, 1.0, 0) == 4           # codes stride % 16
    assert _fp8(A, 8, C8, 12, S8, 4, 8, H.BF16, 1.0, 0) == 4                # n = 8: codes % 8
    assert _fp8(A, 6, C8, 4, S8, 4, 4, H.BF16, 1.0, 0) == 4                 # n = 4: input % 4
    assert _fp8(A, 128, C8, 120, S8, 4, 128, H.BF16, 1.0, 0) == 4           # codes stride < n
    assert _fp8(A, 120, C8, 128, S8, 4, 128, H.BF16, 1.0, 0) == 4           # input stride < n
    assert _fp8(A, (1 << 26) + 8, C8, 128, S8, 4, 128, H.BF16, 1.0, 0) == 4  # input stride > 2^26
    assert _fp8(A, 128, C8, (1 << 26) + 16, S8, 4, 128, H.BF16, 1.0, 0) == 4  # codes stride > 2^26
    assert _fp8(A, 128, C8 + 8, 128, S8, 4, 128, H.BF16, 1.0, 0) == 5       # codes alignment
    assert _fp8(A, 128, C8, 128, S8 + 2, 4, 128, H.BF16, 1.0, 0) == 5       # scales alignment
    assert _fp8(A, 128, 0, 128, S8, 4, 128, H.BF16, 1.0, 0) == 1            # null codes
    assert _fp8(A, 128, C8, 128, 0, 4, 128, H.BF16, 1.0, 0) == 1            # null scales
    assert _fp8(A, 128, C8, 128, S8, 4, 128, H.BF16, math.nan, 0) == 1      # scale
    assert _fp8(A, 128, A + 64, 128, S8, 4, 128, H.BF16, 1.0, 0) == 6       # codes inside input
    assert _fp8(A, 128, C8, 128, A + 16, 4, 128, H.BF16, 1.0, 0) == 6       # scales inside input
    assert _fp8(A, 128, C8, 128, C8 + 256, 4, 128, H.BF16, 1.0, 0) == 6     # scales inside codes
    assert _fp8(0, 128, 0, 128, 0, 0, 128, H.BF16, 1.0, 0) == 0             # m == 0
    assert _fp8(A, 128, C8, 128, S8, -1, 128, H.BF16, 1.0, 0) == 1
    assert len(ok_args) == 10


W8 = 1 << 36   # fake workspace


def _ws(*args):
    return H.hadamard_transform_ws(*args, check=False)


def test_workspace_size():
    assert H.hadamard_transform_workspace_size(4, 1 << 17) == 4 * 4 * (1 << 17)
    assert H.hadamard_transform_workspace_size(3, 1 << 20) == 4 * 3 * (1 << 20)
    assert H.hadamard_transform_workspace_size(4, 1 << 16) == 0     # one pass, no workspace
    assert H.hadamard_transform_workspace_size(4, 1 << 15) == 0
    assert H.hadamard_transform_workspace_size(0, 1 << 17) == 0
    assert H.hadamard_transform_workspace_size(4, 1 << 21) == 0     # unsupported size
    assert H.hadamard_transform_workspace_size(4, 3 << 15) == 0


@cpu_only
def test_workspace_entry_validation():
    n = 1 << 17
    need = H.hadamard_transform_workspace_size(4, n)
    assert H.hadamard_transform(A, B, 4, n, H.FP16, 1.0, 0, check=False) == 2  # one-pass entry
    assert _ws(A, n, B, n, 4, 1 << 21, H.FP16, 1.0, W8, need, 0) == 2          # above 2^20
    assert _ws(A, n, B, n, 4, n, H.FP16, 1.0, 0, need, 0) == 10                # no workspace
    assert _ws(A, n, B, n, 4, n, H.FP16, 1.0, W8, need - 16, 0) == 10          # too small
    assert _ws(A, n, B, n, 4, n, H.FP16, 1.0, W8 + 8, need, 0) == 5            # misaligned
    assert _ws(A, n, B, n, 4, n, H.FP16, 1.0, A + 64, need, 0) == 6            # overlaps in
    assert _ws(A, n, B, n, 4, n, H.FP16, 1.0, B - need + 2, need, 0) == 5      # misaligned first
    assert _ws(A, n, B, n, 4, n, H.FP16, 1.0, B - need + 16, need, 0) == 6     # overlaps out
    assert _ws(A, n + 4, B, n, 4, n, H.FP16, 1.0, W8, need, 0) == 4            # stride % 8
    assert _ws(0, n, 0, n, 0, n, H.FP16, 1.0, 0, 0, 0) == 0                    # m == 0
    assert _ws(A, n, B, n, 4, n, H.FP16, math.inf, W8, need, 0) == 1
