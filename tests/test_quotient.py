"""The multiply-and-correct quotient amax / Q of the row kernels' quantization
scale, checked on the CPU (tests/native/quotient_check.c).

The kernels use it where the check proves it exact (every finite amax for
Q = 127; every amax whose quotient is normal for Q = 448) and divide
otherwise.  The test runs the checker on a sample: every 4099th fp32 bit
pattern plus dense windows around the subnormal boundary and around Q * 2^-126.
HADACORE_QUOTIENT_EXHAUSTIVE=1 checks all 2^31 inputs (a few minutes).
"""
from __future__ import annotations

import os
import shutil
import subprocess
from pathlib import Path

import pytest

SRC = Path(__file__).resolve().parent / "native" / "quotient_check.c"


@pytest.fixture(scope="module")
def checker(tmp_path_factory):
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    exe = tmp_path_factory.mktemp("quotient") / "quotient_check"
    subprocess.run([cc, "-O2", "-mfma", "-ffp-contract=off", str(SRC), "-o", str(exe), "-lm"],
                   check=True)
    return exe


def test_quotient_by_constant_is_correctly_rounded_where_used(checker):
    stride = "1" if os.environ.get("HADACORE_QUOTIENT_EXHAUSTIVE") == "1" else "4099"
    out = subprocess.run([str(checker), stride], check=True, capture_output=True, text=True).stdout
    rows = {float(q): (int(n), int(bn), int(bs)) for q, n, bn, bs in
            (line.split() for line in out.strip().splitlines())}
    n127, bad_norm127, bad_sub127 = rows[127.0]
    n448, bad_norm448, bad_sub448 = rows[448.0]
    assert n127 > 500_000 and n448 > 500_000
    assert bad_norm127 == 0 and bad_sub127 == 0        # Q = 127: exact for every finite amax
    assert bad_norm448 == 0                            # Q = 448: exact whenever the quotient is normal
    assert bad_sub448 > 0                              # ... and not for subnormal quotients (hence the guard)
