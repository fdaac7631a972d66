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


def test_one_element_row_takes_the_largest_code(oracle):
    """A one-element row v with amax = |v| in [2^-100, inf): the quantization
    multiplier RN(Q / amax) times v, rounded to fp32, always encodes to the
    largest code of v's sign (the oracle's own encoders decide), so the dense
    kernel writes that code without the quotient.  Below the range Q / amax can
    overflow, which is why those rows keep the general path."""
    import numpy as np
    rng = np.random.default_rng(2024)
    e = rng.integers(-100, 128, 1_000_000)
    v = np.ldexp(1.0 + rng.random(e.size), e).astype(np.float32)
    fmax = np.finfo(np.float32).max
    edges = np.array([2.0 ** -100, np.nextafter(np.float32(2.0 ** -100), np.float32(1)),
                      1.0, 127.0, 448.0, 3.0, fmax, np.nextafter(fmax, np.float32(0))], np.float32)
    v = np.concatenate([v[np.isfinite(v)], edges])
    v = np.concatenate([v, -v])
    with np.errstate(over="ignore"):
        for q, encode, top in ((448.0, oracle.encode_e4m3, (0x7E, 0xFE)),
                               (127.0, oracle.encode_int8, (127, -127))):
            mul = np.float32(q) / np.abs(v)              # fp32, correctly rounded
            assert np.isfinite(mul).all()
            w = (v * mul).astype(np.float32)            # the fp32 product
            vals = np.unique(w)
            assert vals.size <= 16, vals                 # a few values next to +-Q
            codes = encode(vals)
            want = np.where(vals > 0, top[0], top[1])
            assert np.array_equal(codes.astype(np.int64), np.asarray(want, np.int64)), (q, vals, codes)
        # below the range the quotient can overflow: those rows take the division
        assert np.float32(448.0) / np.float32(2.0 ** -130) == np.inf
