"""Pins of the oracle's balanced stage partition (CPU only).

The balanced partition is the one whose slowest stage is fastest (Sec. 3.2:
a pipeline with a fixed degree is bottlenecked by its slowest stage).  The
oracle finds it with the textbook recursion over prefixes; these tests tie
that recursion and the canonical cut rule to things fixed outside it:
hand-worked examples, closed forms, and exhaustive enumeration of every
cut vector on small inputs.
"""
import math

import numpy as np
import pytest


def _U(o, u):
    return o.prefix(np.asarray(u, np.float64))


@pytest.mark.parametrize("u,pp,W,cuts", [
    ([1, 2, 3, 4, 5], 2, 9.0, [3]),          # [1 2 3 | 4 5]: max(6, 9)
    ([5, 1, 1, 1, 5], 3, 5.0, [1, 4]),       # [5 | 1 1 1 | 5]
    ([2] * 7, 3, 6.0, [1, 4]),               # sizes 1,3,3: short stages first
    ([7], 1, 7.0, []),
    ([0, 0, 3, 0], 2, 3.0, [1]),              # zero-cost layers: earliest optimal cut
    ([1, 1, 1, 100], 2, 100.0, [3]),          # one dominant layer alone at the end
    ([4, 4, 1, 1, 1, 1, 4, 4], 4, 6.0, [1, 4, 7]),  # each 4 alone or with half the 1s
])
def test_hand_worked(oracle, u, pp, W, cuts):
    U = _U(oracle, u)
    wb, cb = oracle.bottleneck_bruteforce(U, pp)
    assert wb == W and cb == cuts
    wd = oracle.bottleneck_dp(U, pp)
    assert wd == W
    assert oracle.canonical_cuts(U, pp, wd) == cuts


def test_closed_forms_pp1_and_ppL(oracle):
    rng = np.random.default_rng(1)
    for L in (1, 2, 17, 64, 128):
        u = rng.lognormal(0.0, 1.0, L)
        U = _U(oracle, u)
        assert oracle.bottleneck_dp(U, 1) == U[L]
        assert oracle.bottleneck_dp(U, L) == max(U[i + 1] - U[i] for i in range(L))
        assert oracle.canonical_cuts(U, L, oracle.bottleneck_dp(U, L)) == list(range(1, L))


@pytest.mark.parametrize("L,pp", [(10, 4), (12, 5), (128, 3), (128, 100), (97, 8), (6, 6)])
def test_closed_form_equal_costs(oracle, L, pp):
    c = 0.75                          # exact in binary: every prefix is exact
    U = _U(oracle, [c] * L)
    W = oracle.bottleneck_dp(U, pp)
    assert W == math.ceil(L / pp) * c
    cuts = oracle.canonical_cuts(U, pp, W)
    sizes = np.diff([0] + cuts + [L])
    big = math.ceil(L / pp)
    # lexicographically smallest: the short stages come first, then full ones
    assert list(sizes) == sorted(sizes)
    assert sizes.max() == big and sizes.sum() == L and sizes.min() >= 1
    if L % pp == 0:
        assert set(sizes) == {L // pp}


def _random_u(rng, L, kind):
    if kind == "int":
        return rng.integers(0, 4, L).astype(np.float64)       # many exact ties, zeros
    if kind == "dominant":
        u = rng.uniform(0.1, 1.0, L)
        u[rng.integers(0, L)] = 50.0
        return u
    if kind == "equal":
        return np.full(L, 1.5)
    return rng.lognormal(0.0, 0.8, L)


def test_dp_and_cuts_match_exhaustive_enumeration(oracle):
    rng = np.random.default_rng(2024)
    n = 0
    for kind in ("int", "dominant", "equal", "lognormal"):
        for _ in range(250):
            L = int(rng.integers(1, 12))
            pp = int(rng.integers(1, L + 1))
            u = _random_u(rng, L, kind)
            U = _U(oracle, u)
            wb, cb = oracle.bottleneck_bruteforce(U, pp)
            wd = oracle.bottleneck_dp(U, pp)
            assert wd == wb, (u, pp)
            assert oracle.canonical_cuts(U, pp, wd) == cb, (u, pp)
            n += 1
    assert n == 1000


def test_canonical_cuts_are_optimal_and_componentwise_smallest(oracle):
    """At sizes too large to enumerate: the cuts attain W*, and moving any one
    cut left breaks a segment (so no optimal vector is smaller anywhere)."""
    rng = np.random.default_rng(7)
    for _ in range(60):
        L = int(rng.integers(20, 129))
        pp = int(rng.integers(2, min(L, 40) + 1))
        u = rng.lognormal(0.0, 0.6, L)
        U = _U(oracle, u)
        W = oracle.bottleneck_dp(U, pp)
        cuts = oracle.canonical_cuts(U, pp, W)
        b = [0] + cuts + [L]
        segs = [U[b[k + 1]] - U[b[k]] for k in range(pp)]
        assert max(segs) == W
        assert all(b[k] < b[k + 1] for k in range(pp))
        for k in range(1, pp):
            if b[k] - 1 > b[k - 1]:
                assert U[b[k + 1]] - U[b[k] - 1] > W
        # lower bounds: every single layer lies in some stage, and pp stages
        # cover the total (up to rounding of the prefix)
        assert W >= max(U[i + 1] - U[i] for i in range(L))
        assert W >= U[L] / pp * (1 - 1e-12)


def test_dp_monotone_in_pp(oracle):
    rng = np.random.default_rng(3)
    for _ in range(30):
        L = int(rng.integers(2, 129))
        U = _U(oracle, rng.lognormal(0, 1, L))
        ws = [oracle.bottleneck_dp(U, pp) for pp in range(1, L + 1)]
        assert all(ws[i + 1] <= ws[i] for i in range(L - 1))
