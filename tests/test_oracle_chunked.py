"""Pins for the oracle's shard-by-shard attention (Section 2.3, Section 7).

The merged result is checked against attention over the union of the key sets
evaluated in one piece by a library routine (torch's scaled_dot_product_attention
in float64 on the CPU), and the chunk schedule against a hand-worked example and
brute-force invariants written with plain loops. A slip such as a missing
exp(lse) weight, a merge that ignores an empty side, a shard boundary off by
one, a chunk counted twice, or a schedule sorted the wrong way fails here.
"""

import itertools
import math

import numpy as np
import pytest
import torch

import oracle as orc


def _sdpa(q, k, v, scale):
    """Library reference: softmax(q k^T * scale) v and the row log-sum-exp, float64."""
    qt, kt, vt = (torch.from_numpy(x)[None, None] for x in (q, k, v))
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, scale=scale)[0, 0].numpy()
    lse = torch.logsumexp(torch.from_numpy(q @ k.T) * scale, dim=1).numpy()
    return o, lse


@pytest.mark.parametrize("seed", range(4))
def test_merge_of_two_key_sets_equals_attention_over_their_union(seed):
    rng = np.random.default_rng(seed)
    nq, nk, d = 5, 23, 8
    q, k, v = rng.standard_normal((nq, d)), rng.standard_normal((nk, d)), rng.standard_normal((nk, d))
    scale = 0.4
    split = rng.permutation(nk)
    a, b = np.sort(split[:9]), np.sort(split[9:])
    o_a, l_a = _sdpa(q, k[a], v[a], scale)
    o_b, l_b = _sdpa(q, k[b], v[b], scale)
    o, l = orc.lse_merge(o_a, l_a, o_b, l_b)
    o_ref, l_ref = _sdpa(q, k, v, scale)
    np.testing.assert_allclose(o, o_ref, rtol=0, atol=1e-12)
    np.testing.assert_allclose(l, l_ref, rtol=0, atol=1e-12)


def test_merge_with_an_empty_side_is_the_identity():
    rng = np.random.default_rng(7)
    o = rng.standard_normal((6, 4))
    l = rng.standard_normal(6)
    empty_o, empty_l = np.zeros((6, 4)), np.full(6, -np.inf)
    for got_o, got_l in (orc.lse_merge(o, l, empty_o, empty_l), orc.lse_merge(empty_o, empty_l, o, l)):
        np.testing.assert_array_equal(got_o, o)
        np.testing.assert_allclose(got_l, l, rtol=0, atol=1e-15)
    both_o, both_l = orc.lse_merge(empty_o, empty_l, empty_o, empty_l)
    assert (both_o == 0).all() and np.isneginf(both_l).all()


def test_merge_weights_by_exp_lse_hand_example():
    # Two one-key parts with scores s = 0 and s = log 3: weights 1/4 and 3/4.
    o, l = orc.lse_merge(np.array([[1.0, 0.0]]), np.array([0.0]),
                         np.array([[0.0, 2.0]]), np.array([math.log(3.0)]))
    np.testing.assert_allclose(o, [[0.25, 1.5]], rtol=0, atol=1e-15)
    np.testing.assert_allclose(l, [math.log(4.0)], rtol=0, atol=1e-15)


def test_merge_is_commutative_and_associative():
    rng = np.random.default_rng(11)
    parts = [(rng.standard_normal((4, 3)), rng.standard_normal(4) * 3) for _ in range(3)]
    (oa, la), (ob, lb), (oc, lc) = parts
    ab = orc.lse_merge(oa, la, ob, lb)
    ba = orc.lse_merge(ob, lb, oa, la)
    np.testing.assert_allclose(ab[0], ba[0], rtol=0, atol=1e-14)
    np.testing.assert_allclose(ab[1], ba[1], rtol=0, atol=1e-14)
    left = orc.lse_merge(*ab, oc, lc)
    right = orc.lse_merge(oa, la, *orc.lse_merge(ob, lb, oc, lc))
    np.testing.assert_allclose(left[0], right[0], rtol=0, atol=1e-13)
    np.testing.assert_allclose(left[1], right[1], rtol=0, atol=1e-13)


def _tiny_case(seed, H=3, L=50, d=4, b=8, i0=1, i1=5, keep=3):
    rng = np.random.default_rng(seed)
    Q, K, V = (rng.standard_normal((H, L, d)) for _ in range(3))
    n = orc.num_blocks(L, b)
    scores = rng.standard_normal((H, i1 - i0, n)).astype(np.float32)
    mask, _ = orc.select_topk(scores, keep, i0)
    return Q, K, V, mask, n


def test_part_over_every_block_is_the_whole_row_and_empty_part_is_identity():
    Q, K, V, mask, n = _tiny_case(3)
    b, L, scale = 8, 50, 0.5
    for h, r in itertools.product(range(3), range(4)):
        o, l = orc.attend_part(Q[h], K[h], V[h], mask[h, r], 1 + r, L, b, scale, (0, n))
        o2, l2 = orc.attend_block(Q[h], K[h], V[h], mask[h, r], 1 + r, L, b, scale)
        np.testing.assert_array_equal(o, o2)
        np.testing.assert_array_equal(l, l2)
        kept = np.nonzero(mask[h, r])[0]
        lo = kept.max() + 1  # a range past every kept block
        o, l = orc.attend_part(Q[h], K[h], V[h], mask[h, r], 1 + r, L, b, scale, (lo, n + 1))
        assert (o == 0).all() and np.isneginf(l).all()


def test_part_brute_force_against_library_attention():
    Q, K, V, mask, n = _tiny_case(5)
    b, L, scale = 8, 50, 0.5
    lo, hi = 2, 5
    for h, r in itertools.product(range(3), range(4)):
        i = 1 + r
        o, l = orc.attend_part(Q[h], K[h], V[h], mask[h, r], i, L, b, scale, (lo, hi))
        toks = [t for j in range(lo, hi) if mask[h, r, j] for t in range(j * b, min(L, (j + 1) * b))]
        q_rows = list(range(i * b, min(L, (i + 1) * b)))
        if not toks:
            assert (o == 0).all() and np.isneginf(l).all()
            continue
        o_ref, l_ref = _sdpa(Q[h][q_rows], K[h][toks], V[h][toks], scale)
        np.testing.assert_allclose(o[: len(q_rows)], o_ref, rtol=0, atol=1e-12)
        np.testing.assert_allclose(l[: len(q_rows)], l_ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("ranks,rank,hpc,tail", [(2, 0, 1, 1), (3, 1, 2, 1), (4, 3, 3, 2), (5, 2, 2, 1)])
def test_chunked_attention_equals_the_unchunked_result(ranks, rank, hpc, tail):
    Q, K, V, mask, n = _tiny_case(17 + ranks)
    b, L, scale, i0 = 8, 50, 0.5, 1
    plan = orc.chunk_plan(orc.demand_union(mask), ranks, rank, hpc, tail)
    O, LSE = orc.chunked_attention(Q, K, V, mask, L, b, i0, scale, plan)
    O_ref, LSE_ref = orc.sparse_attention(Q, K, V, mask, L, b, i0, scale)
    np.testing.assert_allclose(O, O_ref, rtol=0, atol=1e-12)
    np.testing.assert_allclose(LSE, LSE_ref, rtol=0, atol=1e-12)


def test_chunk_plan_hand_example():
    # H = 3 heads, n = 6 blocks, R = 3 owners of 2 blocks each, rank 1.
    demand = np.array([[1, 1, 0, 1, 1, 0],
                       [0, 1, 1, 1, 0, 0],
                       [1, 0, 1, 0, 1, 1]], dtype=bool)
    plan = orc.chunk_plan(demand, 3, 1, 2, 1)
    assert plan == [
        # local shard (owner 1, blocks 2..3) whole: 1 + 2 + 1 demanded blocks
        (1, 2, 4, 0, 3, 4),
        # ring distance 1 (owner 2, blocks 4..5), runs of two heads:
        # heads {2} hold 2 blocks, heads {0, 1} hold 1 -> descending
        (2, 4, 6, 2, 3, 2),
        (2, 4, 6, 0, 2, 1),
        # last shard (owner 0, blocks 0..1), runs of one head: 2, 1, 1 blocks
        (0, 0, 2, 0, 1, 2),
        (0, 0, 2, 1, 2, 1),
        (0, 0, 2, 2, 3, 1),
    ]


@pytest.mark.parametrize("seed", range(6))
def test_chunk_plan_invariants_brute_force(seed):
    rng = np.random.default_rng(seed)
    H, n = int(rng.integers(1, 9)), int(rng.integers(2, 40))
    ranks = int(rng.integers(1, min(n, 7) + 1))
    rank = int(rng.integers(0, ranks))
    hpc, tail = int(rng.integers(1, 5)), int(rng.integers(1, 4))
    demand = rng.random((H, n)) < 0.4
    plan = orc.chunk_plan(demand, ranks, rank, hpc, tail)
    owners = [(p * n // ranks, (p + 1) * n // ranks) for p in range(ranks)]
    # every (owner, head) pair exactly once
    seen = {}
    for (p, lo, hi, h0, h1, blocks) in plan:
        assert (lo, hi) == owners[p]
        count = 0
        for h in range(h0, h1):
            assert (p, h) not in seen
            seen[(p, h)] = True
            for j in range(lo, hi):
                count += int(demand[h, j])
        assert blocks == count
    assert len(seen) == ranks * H
    # local shard first and whole; shards in ring order after it
    assert plan[0][:5] == (rank, *owners[rank], 0, H)
    order = [c[0] for c in plan[1:]]
    dist = [(p - rank) % ranks for p in order]
    assert dist == sorted(dist)
    # chunk sizes and order inside each remote shard
    for k in range(1, ranks):
        p = (rank + k) % ranks
        chunks = [c for c in plan[1:] if c[0] == p]
        size = tail if k == ranks - 1 else hpc
        by_head = sorted(chunks, key=lambda c: c[3])
        assert [c[3] for c in by_head] == list(range(0, H, size))
        assert all(c[4] == min(H, c[3] + size) for c in by_head)
        keys = [(-c[5], c[3]) for c in chunks]
        assert keys == sorted(keys)
    if ranks > 1:
        last_shard = [c for c in plan if c[0] == (rank + ranks - 1) % ranks]
        assert plan[-1][5] == min(c[5] for c in last_shard)
