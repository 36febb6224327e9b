"""Pins for the oracle's CDF-mode selection (Section 8.1).

Checked against a hand-worked row, brute force in exact rational arithmetic
(Python's sorted order and Fraction sums of the float64 weights, so no
rounding of a running total can decide a cut), peaked rows whose trailing
blocks carry less mass than float64 resolves next to the total, and
properties the rule must have: tau = 1 keeps every block (every block's
softmax mass is positive), the kept set grows with tau, the kept candidates
outscore the rest, and the forced blocks are always kept. A slip such as a
cumulative sum taken in index order, a missing normalisation, a strict
instead of a non-strict threshold, a reversed tie-break or a running total
that saturates at 1 fails here.
"""

import math
from fractions import Fraction

import numpy as np
import pytest

import oracle as orc


def test_hand_worked_row():
    # p = 4/8, 2/8, 1/8, 1/8 for blocks 0..3; blocks 2 and 3 tie (lower index first).
    s = np.array([[[math.log(4.0), math.log(2.0), 0.0, 0.0]]], dtype=np.float32)
    # the row is global block 0: the diagonal (block 0) is forced and also first
    for tau, want in [(0.5, [0]), (0.6, [0, 1]), (0.75, [0, 1]), (0.8, [0, 1, 2]),
                      (0.875, [0, 1, 2]), (0.9, [0, 1, 2, 3]), (1.0, [0, 1, 2, 3])]:
        mask, sel, counts = orc.select_cdf(s, tau, 0)
        assert np.nonzero(mask[0, 0])[0].tolist() == want, tau
        assert sel[0, 0, :counts[0, 0]].tolist() == want
        assert (sel[0, 0, counts[0, 0]:] == -1).all()
    # as global block 3 the diagonal adds block 3 to the 0.5 prefix
    mask, _, _ = orc.select_cdf(s, 0.5, 3)
    assert np.nonzero(mask[0, 0])[0].tolist() == [0, 3]


def brute_force_cut(row, tau):
    """Shortest prefix of the (score desc, index asc) order whose mass reaches tau,
    with every sum exact: the weights are the float64 values exp(s - max), taken
    as exact rationals."""
    n = len(row)
    order = sorted(range(n), key=lambda j: (-row[j], j))
    mx = max(row)
    w = [Fraction(math.exp(x - mx)) for x in row]
    z = sum(w)
    t = Fraction(tau)
    run = Fraction(0)
    for k, j in enumerate(order, start=1):
        run += w[j]
        if run >= t * z:
            return order, k
    return order, n


@pytest.mark.parametrize("seed", range(12))
def test_brute_force(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 40))
    nq = int(rng.integers(1, 5))
    i0 = int(rng.integers(0, n - nq + 1)) if n >= nq else 0
    nq = min(nq, n - i0)
    s = (rng.standard_normal((2, nq, n)) * rng.uniform(0.1, 4.0)).astype(np.float32)
    if n > 3:
        s[0, 0, 1] = s[0, 0, 2]  # a tie
    if seed % 3 == 2:
        s[1] -= np.float32(60.0) * (np.arange(n, dtype=np.float32) % 2)  # peaked row
    G = [int(x) for x in rng.choice(n, size=min(2, n), replace=False)] if seed % 2 else []
    tau = float(rng.uniform(0.05, 1.0)) if seed % 4 else 1.0 - 1e-13
    mask, sel, counts = orc.select_cdf(s, tau, i0, G)
    for h in range(2):
        for r in range(nq):
            order, k = brute_force_cut([float(x) for x in s[h, r]], tau)
            want = set(order[:k]) | {i0 + r} | set(G)
            assert set(np.nonzero(mask[h, r])[0].tolist()) == want
            assert counts[h, r] == len(want)


def test_peaked_row_keeps_blocks_below_float64_resolution():
    # p = 1, then seven blocks of e^-40 = 4.2e-18 each: their mass is below
    # half an ulp of the total, so a prefix sum reaches the total after the
    # first block; every block still carries mass, so tau = 1 keeps all eight.
    s = np.array([[[0.0] + [-40.0] * 7]], dtype=np.float32)
    mask, sel, counts = orc.select_cdf(s, 1.0, 0)
    assert mask[0, 0].all() and counts[0, 0] == 8
    assert sel[0, 0].tolist() == list(range(8))
    # tau = 1 - 1e-12 allows 1e-12 of the mass to be left out: the seven
    # trailing blocks (3e-17 together) go, and the diagonal (block 0) stays.
    mask, _, counts = orc.select_cdf(s, 1.0 - 1e-12, 0)
    assert np.nonzero(mask[0, 0])[0].tolist() == [0]
    # the cut runs through the tail at the right place: blocks e^-10, e^-20,
    # e^-30 leave out 4.5e-5, 2.1e-9 and 9.4e-14 after one, two and three blocks
    s = np.array([[[0.0, -10.0, -20.0, -30.0]]], dtype=np.float32)
    for tau, k in [(1.0 - 1e-4, 1), (1.0 - 1e-6, 2), (1.0 - 1e-9, 3), (1.0 - 1e-12, 3),
                   (1.0 - 1e-14, 4), (1.0, 4)]:
        mask, _, _ = orc.select_cdf(s, tau, 0)
        assert np.nonzero(mask[0, 0])[0].tolist() == list(range(k)), tau
    # a score spread beyond float64's exp range: the weight of the low block
    # underflows to 0, but its mass is positive, so tau = 1 still keeps it
    s = np.array([[[0.0, -800.0, -1000.0]]], dtype=np.float32)
    mask, _, _ = orc.select_cdf(s, 1.0, 2)
    assert mask[0, 0].all()
    mask, _, _ = orc.select_cdf(s, 0.999, 2)
    assert np.nonzero(mask[0, 0])[0].tolist() == [0, 2]  # block 0 and the diagonal


def test_left_out_mass_is_the_exact_suffix():
    rng = np.random.default_rng(7)
    row = (rng.standard_normal(50) * 3).astype(np.float32)
    order, left, Z = orc.cdf_order_and_mass(row)
    w = np.exp(row.astype(np.float64) - float(row.max()))
    assert left[-1] == 0.0 and left[0] == Z
    for k in range(51):
        assert math.isclose(left[k], float(sum(Fraction(float(x)) for x in w[order[k:]])),
                            rel_tol=1e-14, abs_tol=0.0)


def test_tau_one_keeps_everything_and_growth_is_monotone():
    rng = np.random.default_rng(3)
    s = rng.standard_normal((3, 6, 50)).astype(np.float32)
    s[2] *= np.float32(30.0)  # peaked rows
    full, _, _ = orc.select_cdf(s, 1.0, 10)
    assert full.all()
    prev = None
    for tau in (0.1, 0.3, 0.5, 0.7, 0.85, 0.9, 0.95, 0.99, 1 - 1e-9, 1 - 1e-15, 1.0):
        m, _, _ = orc.select_cdf(s, tau, 10)
        if prev is not None:
            assert (m | ~prev).all()  # prev is a subset of m
        prev = m


def test_kept_candidates_outscore_the_rest_and_forced_blocks_stay():
    rng = np.random.default_rng(4)
    s = rng.standard_normal((2, 8, 64)).astype(np.float32)
    G = [60, 61]
    mask, _, _ = orc.select_cdf(s, 0.6, 20, G)
    for h in range(2):
        for r in range(8):
            i = 20 + r
            assert mask[h, r, i] and mask[h, r, G].all()
            cand = np.ones(64, dtype=bool)
            cand[[i] + G] = False
            kept = s[h, r][cand & mask[h, r]]
            dropped = s[h, r][cand & ~mask[h, r]]
            if kept.size and dropped.size:
                assert kept.min() >= dropped.max()


def test_rejects_bad_tau_and_nan():
    s = np.zeros((1, 1, 4), dtype=np.float32)
    for tau in (0.0, -0.1, 1.5):
        with pytest.raises(ValueError):
            orc.select_cdf(s, tau, 0)
    for bad in (np.nan, np.inf, -np.inf):
        s[0, 0, 2] = bad
        with pytest.raises(ValueError):
            orc.select_cdf(s, 0.5, 0)
