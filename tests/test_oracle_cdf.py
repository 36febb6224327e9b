"""Pins for the oracle's CDF-mode selection (Section 8.1).

Checked against a hand-worked row, brute force in plain Python (sorted order,
running sum of exp), and properties the rule must have: tau = 1 keeps every
block, the kept set grows with tau, the kept candidates outscore the rest, and
the forced blocks are always kept. A slip such as a cumulative sum taken in
index order, a missing normalisation, a strict instead of a non-strict
threshold, or a reversed tie-break fails here.
"""

import math

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


@pytest.mark.parametrize("seed", range(10))
def test_brute_force(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 40))
    nq = int(rng.integers(1, 5))
    i0 = int(rng.integers(0, n - nq + 1)) if n >= nq else 0
    nq = min(nq, n - i0)
    s = (rng.standard_normal((2, nq, n)) * rng.uniform(0.1, 4.0)).astype(np.float32)
    if n > 3:
        s[0, 0, 1] = s[0, 0, 2]  # a tie
    G = [int(x) for x in rng.choice(n, size=min(2, n), replace=False)] if seed % 2 else []
    tau = float(rng.uniform(0.05, 1.0))
    mask, sel, counts = orc.select_cdf(s, tau, i0, G)
    for h in range(2):
        for r in range(nq):
            row = [float(x) for x in s[h, r]]
            order = sorted(range(n), key=lambda j: (-row[j], j))
            mx = max(row)
            e = [math.exp(x - mx) for x in row]
            z = sum(e)
            run, k = 0.0, 0
            for j in order:
                run += e[j]
                k += 1
                if run / z >= tau - 1e-12:
                    break
            want = set(order[:k]) | {i0 + r} | set(G)
            assert set(np.nonzero(mask[h, r])[0].tolist()) == want
            assert counts[h, r] == len(want)


def test_tau_one_keeps_everything_and_growth_is_monotone():
    rng = np.random.default_rng(3)
    s = rng.standard_normal((3, 6, 50)).astype(np.float32)
    full, _, _ = orc.select_cdf(s, 1.0, 10)
    assert full.all()
    prev = None
    for tau in (0.1, 0.3, 0.5, 0.7, 0.85, 0.9, 0.95, 0.99, 1.0):
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
    s[0, 0, 2] = np.nan
    with pytest.raises(ValueError):
        orc.select_cdf(s, 0.5, 0)
