"""Pins of the fp64 oracle against facts fixed by the paper and by mathematics.

Nothing here compares the oracle with itself: each check uses an independent
construction (scipy's Sylvester Hadamard matrix, Kronecker products built with
numpy, numpy's own 16-bit decoders, hand-derived fixtures, closed-form special
vectors, orthogonality, involution and Parseval).
"""
from __future__ import annotations

import json
import math
from pathlib import Path

import numpy as np
import pytest
import scipy.linalg

from paper_2412_08832_amd import workloads as W
from metrics import bits_to_f64

GOLDEN = Path(__file__).resolve().parent / "golden" / "fwht_small.json"


def _hadamard(n: int) -> np.ndarray:
    # scipy builds the Sylvester-ordered matrix by repeated Kronecker doubling
    return scipy.linalg.hadamard(n).astype(np.float64)


# --- 16-bit decoders -----------------------------------------------------------

def test_decode_fp16_every_pattern(oracle):
    bits = np.arange(1 << 16, dtype=np.uint16)
    got = oracle.decode(bits, "fp16")
    want = bits.view(np.float16).astype(np.float64)
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], want[~nan])
    # sign of zero survives
    assert math.copysign(1.0, got[0x8000]) == -1.0


def test_decode_bf16_every_pattern(oracle):
    bits = np.arange(1 << 16, dtype=np.uint16)
    got = oracle.decode(bits, "bf16")
    with np.errstate(invalid="ignore"):
        want = (bits.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], want[~nan])


# --- brute force against the explicit matrix (the paper's own unit test, Sec. 4.2) ---

@pytest.mark.parametrize("k", range(1, 11))
def test_matches_explicit_matrix_integers_exact(oracle, k):
    n = 1 << k
    bits = W.random_rows(5, n, "fp16", seed=k, dist="integer")
    x = bits_to_f64(bits, "fp16")
    want = x @ _hadamard(n)
    got = oracle.fwht(bits, "fp16", 1.0)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("dtype", ["fp16", "bf16"])
@pytest.mark.parametrize("k", [1, 3, 7, 8, 9, 10])
def test_matches_explicit_matrix_random(oracle, dtype, k):
    n = 1 << k
    bits = W.random_rows(7, n, dtype, seed=100 + k)
    x = bits_to_f64(bits, dtype)
    s = W.default_scale(n)
    want = (x @ _hadamard(n)) * s
    got = oracle.fwht(bits, dtype, s)
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12 * np.abs(want).max())


@pytest.mark.parametrize("a_log2,b_log2", [(6, 5), (8, 4), (8, 5), (7, 7), (8, 6), (8, 7)])
def test_matches_kronecker_factorisation(oracle, a_log2, b_log2):
    """H_{ab} = H_a (x) H_b: a row reshaped to an a x b matrix X transforms as H_a X H_b^T.

    This reaches n = 2^11 .. 2^15 without an n x n matrix (Sec. 3.4 relates the
    transform to Kronecker products of smaller Hadamard matrices).
    """
    a, b = 1 << a_log2, 1 << b_log2
    n = a * b
    bits = W.random_rows(2, n, "fp16", seed=n, dist="integer")
    x = bits_to_f64(bits, "fp16")
    ha, hb = _hadamard(a), _hadamard(b)
    want = np.stack([(ha @ row.reshape(a, b) @ hb.T).reshape(-1) for row in x])
    got = oracle.fwht(bits, "fp16", 1.0)
    assert np.array_equal(got, want)


def test_sixteen_by_sixteen_reshape_identity(oracle):
    """n = 256 as a 16 x 16 tile: H_16 applied on both sides of the reshaped row (Sec. 3.1)."""
    bits = W.random_rows(3, 256, "bf16", seed=5)
    x = bits_to_f64(bits, "bf16")
    h16 = _hadamard(16)
    want = np.stack([(h16 @ row.reshape(16, 16) @ h16).reshape(-1) for row in x])
    np.testing.assert_allclose(oracle.fwht(bits, "bf16", 1.0), want, rtol=1e-13, atol=1e-12)


def test_partial_last_tile_identity(oracle):
    """n = 2^a * 16^k: the last radix-16 step uses I_{16/2^a} (x) H_{2^a} (Sec. 3.3).

    n = 2048 = 8 * 256: transform the fast index with H_256, then view pairs of
    8-long columns as 16-vectors and apply the block-diagonal [[H_8, 0], [0, H_8]].
    """
    n = 2048
    bits = W.random_rows(2, n, "fp16", seed=9, dist="integer")
    x = bits_to_f64(bits, "fp16")
    h256 = _hadamard(256)
    tile = np.kron(np.eye(2), _hadamard(8))
    want = []
    for row in x:
        X = row.reshape(8, 256) @ h256.T              # H_256 along the fast index
        Z = X.T.reshape(128, 16) @ tile.T             # 16-vectors = two stacked columns
        want.append(Z.reshape(256, 8).T.reshape(-1))
    assert np.array_equal(oracle.fwht(bits, "fp16", 1.0), np.stack(want))


def test_direct_definition_agrees_with_explicit_matrix(oracle):
    n = 512
    bits = W.random_rows(4, n, "fp16", seed=11, dist="integer")
    x = bits_to_f64(bits, "fp16")
    want = (x @ _hadamard(n)) * 0.375   # integers times 3/8: exact in fp64
    rows = np.repeat(np.arange(4), 17)
    cols = np.tile(np.r_[0, 1, 2, 3, 255, 256, 257, 300, 311, 400, 444, 480, 500, 509, 510, 511, 128], 4)
    got = oracle.fwht_direct(bits, "fp16", 0.375, rows, cols)
    assert np.array_equal(got, want[rows, cols])


@pytest.mark.parametrize("k", [7, 12, 15])
def test_direct_definition_agrees_with_fast_transform_large(oracle, k):
    n = 1 << k
    bits = W.random_rows(2, n, "fp16", seed=k)
    s = W.default_scale(n)
    full = oracle.fwht(bits, "fp16", s)
    rng = np.random.default_rng(k)
    rows = rng.integers(0, 2, 64)
    cols = rng.integers(0, n, 64)
    got = oracle.fwht_direct(bits, "fp16", s, rows, cols)
    # fp16 inputs: both unscaled sums are exact in fp64, so only the final product rounds
    assert np.array_equal(got, full[rows, cols])


# --- structure: orthogonality, involution, Parseval ---------------------------------

@pytest.mark.parametrize("k", [1, 4, 7, 10])
def test_orthogonality_from_basis_vectors(oracle, k):
    """Transforming e_0..e_{n-1} yields H with H H^T = n I (Sec. 2.1: orthogonal, +-1)."""
    n = 1 << k
    H = oracle.fwht_vec(np.eye(n))
    assert np.array_equal(np.abs(H), np.ones((n, n)))
    assert np.array_equal(H @ H.T, n * np.eye(n))
    assert np.array_equal(H, _hadamard(n))


@pytest.mark.parametrize("k", [7, 11, 15])
def test_involution_integers_exact(oracle, k):
    n = 1 << k
    x = np.random.default_rng(k).integers(-8, 9, (3, n)).astype(np.float64)
    twice = oracle.fwht_vec(oracle.fwht_vec(x))
    assert np.array_equal(twice, n * x)


@pytest.mark.parametrize("k", [7, 13, 15])
def test_involution_and_parseval_random(oracle, k):
    n = 1 << k
    x = np.random.default_rng(k + 1).standard_normal((3, n))
    y = oracle.fwht_vec(x) / math.sqrt(n)
    np.testing.assert_allclose(np.linalg.norm(y, axis=1), np.linalg.norm(x, axis=1), rtol=1e-13)
    back = oracle.fwht_vec(y) / math.sqrt(n)
    np.testing.assert_allclose(back, x, rtol=0, atol=1e-12 * np.abs(x).max())


# --- closed-form special vectors and hand-derived fixtures --------------------------

@pytest.mark.parametrize("k", [7, 9, 15])
def test_special_vectors(oracle, k):
    n = 1 << k
    one = np.float16(1.0).view(np.uint16)
    delta = np.zeros((1, n), np.uint16)
    delta[0, 0] = one
    assert np.array_equal(oracle.fwht(delta, "fp16", 1.0), np.ones((1, n)))
    ones = np.full((1, n), one, np.uint16)
    e0 = np.zeros((1, n))
    e0[0, 0] = n
    assert np.array_equal(oracle.fwht(ones, "fp16", 1.0), e0)
    # a Walsh row (-1)^popcount(k & j) maps to n e_k
    for kk in (1, 5, n // 2 + 3, n - 1):
        j = np.arange(n)
        parity = np.array([bin(kk & int(v)).count("1") & 1 for v in j])
        row = np.where(parity == 1, -1.0, 1.0).astype(np.float16).view(np.uint16)[None, :]
        want = np.zeros((1, n))
        want[0, kk] = n
        assert np.array_equal(oracle.fwht(row, "fp16", 1.0), want)


def test_hand_derived_fixtures(oracle):
    cases = json.loads(GOLDEN.read_text())["cases"]
    for c in cases:
        x = np.array(c["x"], dtype=np.float64)
        got = oracle.fwht_vec(x[None, :])[0] * c["scale"]
        assert np.array_equal(got, np.array(c["y"], dtype=np.float64)), c
        bits = np.array(c["x"], dtype=np.float16).view(np.uint16)[None, :]
        assert np.array_equal(oracle.fwht(bits, "fp16", c["scale"])[0], np.array(c["y"], float)), c


# --- interface behaviour: strides, scale, threads, non-finite values ------------------

def test_strided_rows_ignore_gaps(oracle):
    n, stride = 256, 272
    bits = W.random_rows(6, n, "bf16", seed=3, stride=stride, fill_bits=0x7FC0)  # NaN canary
    dense = np.ascontiguousarray(bits[:, :n])
    got = oracle.fwht(bits, "bf16", 0.0625, n=n)
    assert np.array_equal(got, oracle.fwht(dense, "bf16", 0.0625))
    assert np.isfinite(got).all()


def test_scale_is_one_final_product(oracle):
    bits = W.random_rows(3, 1024, "fp16", seed=8)
    y1 = oracle.fwht(bits, "fp16", 1.0)
    s = W.default_scale(1024)  # 1/32, a power of two
    assert np.array_equal(oracle.fwht(bits, "fp16", s), y1 * s)
    s2 = float(np.float32(0.3))
    assert np.array_equal(oracle.fwht(bits, "fp16", s2), y1 * s2)


def test_threads_do_not_change_results(oracle):
    bits = W.random_rows(37, 2048, "bf16", seed=4)
    assert np.array_equal(oracle.fwht(bits, "bf16", 0.1, nthreads=1),
                          oracle.fwht(bits, "bf16", 0.1, nthreads=8))


def test_nonfinite_propagation(oracle):
    n = 128
    bits = W.random_rows(3, n, "fp16", seed=2)
    bits[0, 17] = 0x7E00                      # NaN: every output of row 0 is NaN
    bits[1, 5] = 0x7C00                       # +Inf alone: outputs are +-Inf, sign of H[j][5]
    y = oracle.fwht(bits, "fp16", W.default_scale(n))
    assert np.isnan(y[0]).all()
    signs = _hadamard(n)[:, 5]
    assert np.array_equal(y[1], signs * np.inf)
    assert np.isfinite(y[2]).all()


def test_rejects_bad_arguments(oracle):
    bits = np.zeros((2, 96), np.uint16)
    with pytest.raises(ValueError):
        oracle.fwht(bits, "fp16", 1.0)                       # n not a power of two
    with pytest.raises(ValueError):
        oracle.fwht(np.zeros((2, 64), np.uint16), "fp16", 1.0, n=128)  # stride < n
