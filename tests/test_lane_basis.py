"""The change of basis behind the matrix-core front's lane stages, checked on the CPU.

After the radix-32 matrix-core step, the vector bits sit on lane bits 0-3 and
each lane stage exchanges a value with a partner lane.  DPP reaches partners
l ^ 1, l ^ 2 (quad_perm), l ^ 7 (row_half_mirror) and l ^ 8 (row_ror:8), but
not l ^ 4.  The kernel therefore runs the butterflies along the basis
b = (1, 2, 7, 8) of GF(2)^4 instead of (1, 2, 4, 8), and in each stage treats
lane l as the "high" member of its pair when <psi_i, l> is odd, psi being the
dual basis (masks 5, 6, 4, 8).  This file emulates those twisted butterflies
(every lane forms self + sign * partner) and checks the claim the kernel's
store layout relies on:

    lane p holds (-1)^popcount(p) * y[j(p)],   j(p) = (p0^p2, p1^p2, p0^p1^p2, p3),

y being the Walsh-Hadamard transform (Sec. 2.1-2.2) of the 16 lane values.
"""
from __future__ import annotations

import itertools

import numpy as np
import pytest

PARTNERS = (1, 2, 7, 8)
DUAL_MASKS = (5, 6, 4, 8)


def sylvester(n: int) -> np.ndarray:
    return np.array([[(-1) ** bin(i & j).count("1") for j in range(n)] for i in range(n)],
                    dtype=np.float64)


def twisted_stages(x: np.ndarray, partners, masks) -> np.ndarray:
    """Each stage: v[l] <- v[l] + sign(l) * v[l ^ b], sign(l) = -1 iff <mask, l> is odd."""
    v = x.astype(np.float64).copy()
    lanes = np.arange(len(v))
    for b, mask in zip(partners, masks):
        sign = np.where(np.array([bin(int(l) & mask).count("1") & 1 for l in lanes]) == 1, -1.0, 1.0)
        v = v + sign * v[lanes ^ b]
    return v


def j_map(p: int) -> int:
    """The same bit formula as the kernel's lane_frequency on lane bits 0-3."""
    p2 = (p >> 2) & 1
    b0 = (p & 1) ^ p2
    b1 = ((p >> 1) & 1) ^ p2
    return b0 | (b1 << 1) | ((b0 ^ b1 ^ p2) << 2) | (p & 8)


def test_j_is_a_permutation_that_fixes_the_high_bit():
    images = [j_map(p) for p in range(16)]
    assert sorted(images) == list(range(16))
    assert all((j_map(p) ^ p) & 8 == 0 for p in range(16))


@pytest.mark.parametrize("order", list(itertools.permutations(range(4))))
def test_dual_basis_butterflies_give_the_transform_at_permuted_lanes(order):
    rng = np.random.default_rng(sum(o << (2 * i) for i, o in enumerate(order)))
    x = rng.standard_normal(16)
    y = sylvester(16) @ x
    v = twisted_stages(x, [PARTNERS[i] for i in order], [DUAL_MASKS[i] for i in order])
    for p in range(16):
        sign = -1.0 if bin(p).count("1") & 1 else 1.0
        assert v[p] == pytest.approx(sign * y[j_map(p)], rel=1e-12, abs=1e-12)


def test_standard_basis_is_the_identity_case():
    """Partners (1, 2, 4, 8) with their own bits as masks: lane p holds +-y[p]."""
    x = np.random.default_rng(3).standard_normal(16)
    y = sylvester(16) @ x
    v = twisted_stages(x, (1, 2, 4, 8), (1, 2, 4, 8))
    signs = np.array([-1.0 if bin(p).count("1") & 1 else 1.0 for p in range(16)])
    np.testing.assert_allclose(v, signs * y, rtol=1e-12, atol=1e-12)


def test_partner_seven_needs_the_dual_masks():
    """With partner l ^ 7 but the plain bit masks (1, 2, 4, 8), some lane holds no
    single +-y[k]: the dual masks are what make the stages a transform."""
    x = np.random.default_rng(4).standard_normal(16)
    y = sylvester(16) @ x
    v = twisted_stages(x, PARTNERS, (1, 2, 4, 8))
    clean = [any(abs(v[p] - s * y[k]) < 1e-9 for k in range(16) for s in (1.0, -1.0))
             for p in range(16)]
    assert not all(clean)
