"""Pins for the oracle's demand-directed routing (Section 5.1, Section 5.2).

The paper's own worked example (tests/golden/cross_ring_example.json: ring
forwarding moves 4 + 3 + 1 = 8 block-hops where direct delivery moves 4) is
reproduced; provide sets are checked against Eq. 2 written as loops, the
producer's packed layout against the consumer's own derivation from the same
mask (the metadata-free exchange), and the volume counts by brute force. A
slip such as a relay hop that forgets a downstream consumer, a provide set not
cut to the producer's shard, or a packing order that differs between the two
ends fails here.
"""

import json
import os

import numpy as np
import pytest

import oracle as orc

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "cross_ring_example.json")


def test_paper_cross_ring_example():
    ex = json.load(open(GOLDEN))
    R, p = ex["ranks"], ex["producer"]
    names = ex["blocks"]
    n = R * len(names)           # every rank owns len(names) blocks; p owns the first ones
    lo = p * len(names)
    demands = [np.zeros((1, n), dtype=bool) for _ in range(R)]
    for c, blocks in ex["demand"].items():
        for name in blocks:
            demands[int(c)][0, lo + names.index(name)] = True
    provides = orc.provide_masks(demands, R, p)
    assert [c for c, _ in provides] == [1, 2, 3]
    vol = orc.route_volume(provides, len(names))
    per_hop = [int(np.logical_or.reduce([m for _, m in provides[k:]]).sum()) for k in range(R - 1)]
    assert per_hop == ex["relay_blocks_per_hop"]
    assert vol["relay"] == ex["relay_block_hops"]
    assert vol["direct"] == ex["direct_blocks"]
    assert vol["dense"] == (R - 1) * len(names)


@pytest.mark.parametrize("seed", range(6))
def test_provide_sets_are_eq2_restricted_to_the_shard(seed):
    rng = np.random.default_rng(seed)
    H, n = int(rng.integers(1, 5)), int(rng.integers(4, 60))
    R = int(rng.integers(2, min(n, 8) + 1))
    p = int(rng.integers(0, R))
    mask_all = rng.random((H, n, n)) < 0.15
    owner = orc.contiguous_owner(n, R)
    demands = [orc.rank_demand(mask_all, owner, c) for c in range(R)]
    provides = orc.provide_masks(demands, R, p)
    for k, (c, m) in enumerate(provides):
        assert c == (p + k + 1) % R
        for h in range(H):
            for j in range(n):
                want = owner[j] == p and any(mask_all[h, i, j] for i in range(n) if owner[i] == c)
                assert m[h, j] == want


@pytest.mark.parametrize("seed", range(6))
def test_volumes_brute_force(seed):
    rng = np.random.default_rng(20 + seed)
    H, n = int(rng.integers(1, 5)), int(rng.integers(4, 60))
    R = int(rng.integers(2, min(n, 8) + 1))
    p = int(rng.integers(0, R))
    demands = [rng.random((H, n)) < 0.3 for _ in range(R)]
    provides = orc.provide_masks(demands, R, p)
    lo, hi = orc.local_range(n, R, p)
    vol = orc.route_volume(provides, hi - lo)
    direct = relay = 0
    for k in range(1, R):
        for h in range(H):
            for j in range(lo, hi):
                direct += int(demands[(p + k) % R][h, j])
                relay += int(any(demands[(p + m) % R][h, j] for m in range(k, R)))
    assert vol["direct"] == direct and vol["relay"] == relay
    assert vol["dense"] == (R - 1) * H * (hi - lo)
    assert vol["direct"] <= vol["relay"] <= vol["dense"]


def test_packing_is_derived_identically_on_both_ends():
    rng = np.random.default_rng(5)
    H, n, b, d, R, p = 3, 20, 4, 8, 4, 1
    L = n * b - 2
    K, V = rng.standard_normal((H, L, d)), rng.standard_normal((H, L, d))
    demands = [rng.random((H, n)) < 0.4 for _ in range(R)]
    provides = orc.provide_masks(demands, R, p)
    out = orc.pack_by_consumer(provides, K, V, L, b)
    lo, hi = orc.local_range(n, R, p)
    for idx, (c, m) in enumerate(provides):
        # the consumer derives its receive layout from its own demand cut to p's shard
        mine = np.zeros((H, n), dtype=bool)
        mine[:, lo:hi] = demands[c][:, lo:hi]
        c_off, c_blk, _ = orc.packing_plan(mine)
        s0 = out["cons_off"][idx]
        s1 = out["cons_off"][idx + 1]
        assert s1 - s0 == c_off[-1]
        np.testing.assert_array_equal(out["gather_blk"][s0:s1], c_blk)
        np.testing.assert_array_equal(out["head_off"][idx * H:(idx + 1) * H + 1] - s0, c_off)
        for t, slot in enumerate(range(s0, s1)):
            h = int(np.searchsorted(c_off, t, side="right") - 1)
            j = int(c_blk[t])
            cnt = min(b, L - j * b)
            np.testing.assert_array_equal(out["K_packed"][slot, :cnt], K[h, j * b:j * b + cnt])
            np.testing.assert_array_equal(out["V_packed"][slot][:, :cnt], V[h, j * b:j * b + cnt].T)
