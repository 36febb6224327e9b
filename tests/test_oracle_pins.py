"""Pins for the float64 oracle against things other than itself.

Each check comes from the paper's definitions (Eq. 1, Section 4.1's mask M,
Eq. 2, Eq. 3, Section 5.2's packing order), from closed forms, from library
routines that are special cases (torch's scaled_dot_product_attention on the
CPU in float64), or from brute force in plain Python loops on tiny inputs.
The cases are picked so that a plausible slip in the oracle (a padded token
averaged in, a wrong score scale, a reversed tie-break, the diagonal taken at
the local row instead of the global block, a transposed V block, an
unnormalised softmax, a padded key left in) fails at least one of them.
"""

import itertools
import math

import numpy as np
import pytest

import oracle as orc

pytestmark = pytest.mark.filterwarnings("ignore::DeprecationWarning")


# ---------------------------------------------------------------------------
# number format
# ---------------------------------------------------------------------------

def test_decode_bf16_known_patterns():
    bits = np.array([0x3F80, 0xC000, 0x0000, 0x8000, 0x7F80, 0xFF80, 0x3FC0, 0x0001, 0x4049],
                    dtype=np.uint16)
    got = orc.decode_bf16(bits)
    want = [1.0, -2.0, 0.0, -0.0, math.inf, -math.inf, 1.5, 2.0 ** -133, 3.140625]
    assert got.tolist() == want
    assert math.copysign(1.0, got[3]) == -1.0


# ---------------------------------------------------------------------------
# pooling (Section 4.2)
# ---------------------------------------------------------------------------

def test_pool_constant_blocks_give_the_row():
    rng = np.random.default_rng(1)
    H, b, n, d = 2, 4, 5, 3
    rows = rng.standard_normal((H, n, d))
    X = np.repeat(rows, b, axis=1)  # every token of block j equals rows[:, j]
    np.testing.assert_array_equal(orc.pool_blocks(X, n * b, b), rows)


def test_pool_block_of_one_is_identity():
    X = np.random.default_rng(2).standard_normal((3, 7, 5))
    np.testing.assert_array_equal(orc.pool_blocks(X, 7, 1), X)


def test_pool_ragged_last_block_brute_force():
    rng = np.random.default_rng(3)
    H, L, d, b = 2, 11, 3, 4  # blocks of 4, 4, 3 valid tokens
    X = rng.standard_normal((H, L, d))
    got = orc.pool_blocks(X, L, b)
    for h in range(H):
        for j in range(3):
            toks = [t for t in range(L) if t // b == j]
            for c in range(d):
                want = sum(X[h, t, c] for t in toks) / len(toks)
                assert abs(got[h, j, c] - want) < 1e-15
    assert orc.block_valid_counts(L, b).tolist() == [4, 4, 3]


# ---------------------------------------------------------------------------
# scores (Sections 4.1, 4.2)
# ---------------------------------------------------------------------------

def test_scores_block_one_equal_token_scores():
    rng = np.random.default_rng(4)
    H, L, d = 2, 6, 4
    Q = rng.standard_normal((H, L, d))
    K = rng.standard_normal((H, L, d))
    S = orc.block_scores(orc.pool_blocks(Q, L, 1), orc.pool_blocks(K, L, 1), d)
    assert S.dtype == np.float32
    for h in range(H):
        for i in range(L):
            for j in range(L):
                dot = 0.0
                for c in range(d):
                    dot += Q[h, i, c] * K[h, j, c]
                assert S[h, i, j] == np.float32(dot / math.sqrt(d))


def test_scores_exact_small_integers():
    # d = 4 -> scale exactly 1/2; integer pooled values -> exact products.
    pq = np.array([[[1.0, 2.0, 0.0, -1.0]]])
    pk = np.array([[[3.0, 0.0, 1.0, 1.0], [-2.0, 1.0, 0.0, 4.0]]])
    S = orc.block_scores(pq, pk, 4)
    assert S.tolist() == [[[1.0, -2.0]]]


# ---------------------------------------------------------------------------
# selection (Section 4.1's M by top-k, forced diagonal, lowest-index ties)
# ---------------------------------------------------------------------------

def _brute_select(scores, keep, i0, G):
    H, nq, n = scores.shape
    mask = np.zeros((H, nq, n), dtype=bool)
    for h in range(H):
        for r in range(nq):
            i = i0 + r
            forced = set(G) | {i}
            cands = [j for j in range(n) if j not in forced]
            # Python floats: -0.0 == 0.0, so the index decides that tie.
            cands.sort(key=lambda j: (-float(scores[h, r, j]), j))
            for j in list(forced) + cands[: keep - len(forced)]:
                mask[h, r, j] = True
    return mask


@pytest.mark.parametrize("seed", range(12))
def test_select_matches_brute_force(seed):
    rng = np.random.default_rng(100 + seed)
    n = int(rng.integers(3, 20))
    nq = int(rng.integers(1, n + 1))
    i0 = int(rng.integers(0, n - nq + 1))
    G = sorted(set(rng.integers(0, n, size=int(rng.integers(0, 3))).tolist()))
    keep = int(rng.integers(len(G) + 1, n + 1))
    # Coarse values force many exact ties.
    scores = (rng.integers(-3, 4, size=(2, nq, n)) * 0.5).astype(np.float32)
    mask, sel = orc.select_topk(scores, keep, i0, G)
    np.testing.assert_array_equal(mask, _brute_select(scores, keep, i0, G))
    assert sel.shape == (2, nq, keep)
    for h in range(2):
        for r in range(nq):
            assert sel[h, r].tolist() == np.nonzero(mask[h, r])[0].tolist()


def test_select_invariants_random():
    rng = np.random.default_rng(7)
    H, n, nq, i0, keep, G = 3, 40, 10, 25, 9, [2, 39]
    scores = rng.standard_normal((H, nq, n)).astype(np.float32)
    mask, sel = orc.select_topk(scores, keep, i0, G)
    assert (mask.sum(axis=2) == keep).all()
    for h in range(H):
        for r in range(nq):
            i = i0 + r
            assert mask[h, r, i] and mask[h, r, 2] and mask[h, r, 39]
            cand = [j for j in range(n) if j not in (i, 2, 39)]
            taken = [scores[h, r, j] for j in cand if mask[h, r, j]]
            left = [scores[h, r, j] for j in cand if not mask[h, r, j]]
            assert min(taken) >= max(left)
            assert (np.diff(sel[h, r]) > 0).all()


def test_select_all_equal_row_takes_lowest_indices():
    n, keep = 10, 4
    scores = np.zeros((1, 1, n), dtype=np.float32)
    mask, sel = orc.select_topk(scores, keep, 6, ())
    assert sel[0, 0].tolist() == [0, 1, 2, 6]


def test_select_signed_zero_is_a_tie():
    # Blocks 1 (+0.0) and 3 (-0.0) tie: the lower index wins, whatever the sign.
    scores = np.array([[[-1.0, 0.0, -1.0, -0.0, -2.0]]], dtype=np.float32)
    _, sel = orc.select_topk(scores, 2, 0, ())
    assert sel[0, 0].tolist() == [0, 1]
    scores = np.array([[[-1.0, -0.0, -1.0, 0.0, -2.0]]], dtype=np.float32)
    _, sel = orc.select_topk(scores, 2, 0, ())
    assert sel[0, 0].tolist() == [0, 1]


def test_select_diagonal_is_the_global_block_index():
    # Local row 0 is global block 5: block 5 is forced, block 0 is not.
    scores = np.full((1, 1, 8), -1.0, dtype=np.float32)
    scores[0, 0, 7] = 3.0
    _, sel = orc.select_topk(scores, 2, 5, ())
    assert sel[0, 0].tolist() == [5, 7]


def test_select_extremes_and_diagonal_in_global_set():
    scores = np.random.default_rng(8).standard_normal((1, 3, 6)).astype(np.float32)
    mask, _ = orc.select_topk(scores, 6, 0, ())
    assert mask.all()
    mask, sel = orc.select_topk(scores, 2, 0, [1])
    # Row 1 is global block 1, already global: F = {1}, one more candidate taken.
    assert mask.sum(axis=2).tolist() == [[2, 2, 2]]
    assert sel[0, 0].tolist() == [0, 1] and sel[0, 2].tolist() == [1, 2]
    assert 1 in sel[0, 1]


def test_select_rejects_bad_arguments():
    s = np.zeros((1, 2, 4), dtype=np.float32)
    with pytest.raises(ValueError):
        orc.select_topk(s, 1, 0, [3])  # keep < |F|
    with pytest.raises(ValueError):
        orc.select_topk(s, 5, 0, ())  # keep > n
    bad = s.copy()
    bad[0, 1, 2] = np.nan
    with pytest.raises(ValueError):
        orc.select_topk(bad, 2, 0, ())
    with pytest.raises(TypeError):
        orc.select_topk(s.astype(np.float64), 2, 0, ())


def test_mask_words_bit_layout():
    mask = np.zeros((1, 130), dtype=bool)
    mask[0, [0, 63, 64, 129]] = True
    w = orc.mask_to_words(mask)
    assert w.dtype == np.uint64
    assert w.tolist() == [[1 | (1 << 63), 1, 2]]
    np.testing.assert_array_equal(orc.words_to_mask(w, 130), mask)


# ---------------------------------------------------------------------------
# demand (Eq. 2) and packing (Section 5.2)
# ---------------------------------------------------------------------------

def test_demand_is_or_of_rows_brute_force():
    rng = np.random.default_rng(9)
    H, nq, n = 3, 5, 17
    mask = rng.random((H, nq, n)) < 0.2
    D = orc.demand_union(mask)
    for h in range(H):
        for j in range(n):
            assert D[h, j] == any(mask[h, i, j] for i in range(nq))


def test_demand_invariants_after_selection():
    rng = np.random.default_rng(10)
    H, n, nq, i0, keep = 4, 30, 6, 12, 5
    scores = rng.standard_normal((H, nq, n)).astype(np.float32)
    mask, _ = orc.select_topk(scores, keep, i0, ())
    D = orc.demand_union(mask)
    assert D[:, i0:i0 + nq].all()  # every local diagonal
    assert (D.sum(axis=1) <= min(n, nq * keep)).all()


def test_packing_plan_hand_example():
    D = np.array([[1, 0, 1, 0], [0, 1, 1, 1]], dtype=bool)
    head_off, gather_blk, slot_of = orc.packing_plan(D)
    assert head_off.tolist() == [0, 2, 5]
    assert gather_blk.tolist() == [0, 2, 1, 2, 3]
    assert slot_of.tolist() == [[0, -1, 1, -1], [-1, 2, 3, 4]]


def test_packing_plan_inverse_maps():
    rng = np.random.default_rng(11)
    D = rng.random((5, 23)) < 0.4
    head_off, gather_blk, slot_of = orc.packing_plan(D)
    assert head_off[0] == 0 and (np.diff(head_off) == D.sum(axis=1)).all()
    for h in range(5):
        for s in range(head_off[h], head_off[h + 1]):
            assert slot_of[h, gather_blk[s]] == s
        seg = gather_blk[head_off[h]:head_off[h + 1]]
        assert (np.diff(seg) > 0).all()
        assert (slot_of[h][~D[h]] == -1).all()


def test_pack_kv_bitwise_transposed_v_and_zero_tail():
    rng = np.random.default_rng(12)
    H, L, d, b = 2, 10, 3, 4  # last block holds 2 valid tokens
    K = rng.integers(1, 60000, size=(H, L, d)).astype(np.uint16)
    V = rng.integers(1, 60000, size=(H, L, d)).astype(np.uint16)
    D = np.array([[1, 0, 1], [0, 1, 0]], dtype=bool)
    head_off, gather_blk, _ = orc.packing_plan(D)
    Kp, Vp = orc.pack_kv(K, V, head_off, gather_blk, L, b)
    assert Kp.shape == (3, b, d) and Vp.shape == (3, d, b)
    # slot 0: head 0 block 0; slot 1: head 0 block 2 (ragged); slot 2: head 1 block 1
    for s, (h, j) in enumerate([(0, 0), (0, 2), (1, 1)]):
        for t in range(b):
            tok = j * b + t
            for c in range(d):
                kv = K[h, tok, c] if tok < L else 0
                vv = V[h, tok, c] if tok < L else 0
                assert Kp[s, t, c] == kv
                assert Vp[s, c, t] == vv


# ---------------------------------------------------------------------------
# attention (Eq. 1 restricted to the kept blocks)
# ---------------------------------------------------------------------------

def _token_mask(mask_rows, L, b, i0):
    """Boolean [nq*b valid queries, L] mask expanded from block rows (valid tokens only)."""
    H, nq, n = mask_rows.shape
    out = np.zeros((H, nq * b, L), dtype=bool)
    for h in range(H):
        for r in range(nq):
            for j in range(n):
                if mask_rows[h, r, j]:
                    out[h, r * b:(r + 1) * b, j * b:min((j + 1) * b, L)] = True
    return out


def _case(seed, H=2, L=37, d=8, b=8, nq=None, i0=0, keep=3, G=()):
    rng = np.random.default_rng(seed)
    n = -(-L // b)
    nq = n - i0 if nq is None else nq
    Q = rng.standard_normal((H, L, d))
    K = rng.standard_normal((H, L, d))
    V = rng.standard_normal((H, L, d))
    scores = rng.standard_normal((H, nq, n)).astype(np.float32)
    mask, _ = orc.select_topk(scores, keep, i0, G)
    return Q, K, V, mask, n


@pytest.mark.parametrize("seed,i0", [(20, 0), (21, 2), (22, 4)])
def test_attention_matches_torch_sdpa(seed, i0):
    torch = pytest.importorskip("torch")
    L, b, d = 37, 8, 8  # 5 blocks, the last with 5 valid tokens
    Q, K, V, mask, n = _case(seed, L=L, d=d, b=b, i0=i0)
    nq = n - i0
    scale = 1.0 / math.sqrt(d)
    O, lse = orc.sparse_attention(Q, K, V, mask, L, b, i0, scale)
    tm = _token_mask(mask, L, b, i0)
    for h in range(2):
        for r in range(nq):
            q_lo, q_hi = (i0 + r) * b, min((i0 + r + 1) * b, L)
            nv = q_hi - q_lo
            qt = torch.from_numpy(Q[h, q_lo:q_hi])[None]
            km = torch.from_numpy(tm[h, r * b:r * b + nv])[None]
            ref = torch.nn.functional.scaled_dot_product_attention(
                qt, torch.from_numpy(K[h])[None], torch.from_numpy(V[h])[None],
                attn_mask=km, scale=scale)[0].numpy()
            np.testing.assert_allclose(O[h, r * b:r * b + nv], ref, rtol=1e-12, atol=1e-13)
            assert (O[h, r * b + nv:(r + 1) * b] == 0).all()
            assert np.isneginf(lse[h, r * b + nv:(r + 1) * b]).all()


def test_attention_all_ones_is_dense_eq1_brute_force():
    rng = np.random.default_rng(30)
    H, L, d, b = 1, 6, 3, 2
    Q, K, V = (rng.standard_normal((H, L, d)) for _ in range(3))
    n = 3
    mask = np.ones((H, n, n), dtype=bool)
    scale = 1.0 / math.sqrt(d)
    O, lse = orc.sparse_attention(Q, K, V, mask, L, b, 0, scale)
    for q in range(L):
        s = [sum(Q[0, q, c] * K[0, t, c] for c in range(d)) * scale for t in range(L)]
        z = sum(math.exp(x) for x in s)
        for c in range(d):
            want = sum(math.exp(s[t]) / z * V[0, t, c] for t in range(L))
            assert abs(O[0, q, c] - want) < 1e-13
        assert abs(lse[0, q] - math.log(z)) < 1e-13
    np.testing.assert_allclose(O, orc.dense_attention(Q, K, V, scale), rtol=1e-13, atol=1e-14)


def test_attention_diagonal_only_is_per_block_local_attention():
    torch = pytest.importorskip("torch")
    L, b, d = 29, 8, 4
    rng = np.random.default_rng(31)
    Q, K, V = (rng.standard_normal((2, L, d)) for _ in range(3))
    n = 4
    scores = rng.standard_normal((2, n, n)).astype(np.float32)
    mask, sel = orc.select_topk(scores, 1, 0, ())
    assert (sel[..., 0] == np.arange(n)).all()
    O, _ = orc.sparse_attention(Q, K, V, mask, L, b, 0, 0.5)
    for h in range(2):
        for i in range(n):
            lo, hi = i * b, min((i + 1) * b, L)
            blk = [torch.from_numpy(x[h, lo:hi])[None] for x in (Q, K, V)]
            ref = torch.nn.functional.scaled_dot_product_attention(*blk, scale=0.5)[0].numpy()
            np.testing.assert_allclose(O[h, i * b:i * b + hi - lo], ref, rtol=1e-12, atol=1e-13)


def test_attention_probability_rows_sum_to_one_and_follow_the_mask():
    Q, K, V, mask, n = _case(32, L=37, b=8, keep=2)
    _, _, p, toks = orc.attend_block(Q[0], K[0], V[0], mask[0, 3], 3, 37, 8, 0.3,
                                     return_probs=True)
    np.testing.assert_allclose(p.sum(axis=1), 1.0, rtol=0, atol=1e-14)
    assert set(t // 8 for t in toks) == set(np.nonzero(mask[0, 3])[0].tolist())
    assert (toks < 37).all()


def test_attention_constant_v_gives_constant_output():
    Q, K, V, mask, n = _case(33)
    V[:] = np.array([1.5, -2.0, 0.25, 0.0, 3.0, 1.0, -1.0, 2.0])
    O, _ = orc.sparse_attention(Q, K, V, mask, 37, 8, 0, 0.35)
    valid = np.arange(n * 8) < 37
    np.testing.assert_allclose(O[:, valid], np.broadcast_to(V[0, 0], O[:, valid].shape),
                               rtol=0, atol=1e-14)


def test_attention_zero_query_is_mean_of_kept_valid_values():
    Q, K, V, mask, n = _case(34)
    Q[:] = 0.0
    O, _ = orc.sparse_attention(Q, K, V, mask, 37, 8, 0, 0.35)
    for h in range(2):
        for r in range(n):
            toks = [t for t in range(37) if mask[h, r, t // 8]]
            want = V[h, toks].mean(axis=0)
            nv = min(8, 37 - r * 8)
            np.testing.assert_allclose(O[h, r * 8:r * 8 + nv], np.broadcast_to(want, (nv, 8)),
                                       rtol=0, atol=1e-14)


def test_attention_invariant_to_kv_block_permutation():
    L, b, d = 32, 8, 4  # whole blocks, so permuting blocks keeps every block full
    Q, K, V, mask, n = _case(35, L=L, b=b, d=d)
    perm = np.array([2, 0, 3, 1])
    tok = np.concatenate([np.arange(p * b, (p + 1) * b) for p in perm])
    # New block k holds old block perm[k]; mask column k must name old column perm[k].
    O1, _ = orc.sparse_attention(Q, K, V, mask, L, b, 0, 0.4)
    O2, _ = orc.sparse_attention(Q, K[:, tok], V[:, tok], mask[:, :, perm], L, b, 0, 0.4)
    np.testing.assert_allclose(O1, O2, rtol=1e-12, atol=1e-13)


def test_attention_is_linear_in_v():
    Q, K, V, mask, n = _case(36)
    V2 = np.random.default_rng(37).standard_normal(V.shape)
    f = lambda vv: orc.sparse_attention(Q, K, vv, mask, 37, 8, 0, 0.35)[0]
    np.testing.assert_allclose(f(2.0 * V - 3.0 * V2), 2.0 * f(V) - 3.0 * f(V2),
                               rtol=1e-12, atol=1e-12)


def test_attention_flops_hand_count():
    # L=10, b=4: blocks of 4, 4, 2 tokens. Local rows 1 and 2.
    mask = np.array([[[1, 1, 0], [0, 1, 1]]], dtype=bool)
    # row block 1 (4 queries): keys 4 + 4; row block 2 (2 queries): keys 4 + 2
    want = 4 * 5 * (4 * 8 + 2 * 6)
    assert orc.attention_flops(mask, 10, 4, 1, 5) == want


# ---------------------------------------------------------------------------
# Eq. 3
# ---------------------------------------------------------------------------

def test_exchange_volume_hand_example():
    # n = 8 blocks over R = 4 ranks: owners 0 0 1 1 2 2 3 3. Rank 1 owns {2, 3}.
    D = np.zeros((2, 8), dtype=bool)
    D[0, [1, 2, 3, 6]] = True  # remote: 1, 6
    D[1, [3, 7]] = True  # remote: 7
    b, d, w = 128, 64, 2
    assert orc.exchange_volume(D, 4, 1, b, d, w) == 2 * b * d * w * 3
    assert orc.local_range(8, 4, 1) == (2, 4)
    assert [orc.local_range(591, 4, r) for r in range(4)] == [(0, 147), (147, 295), (295, 443),
                                                             (443, 591)]
