"""Pins for the oracle's dependency-aware placement (Section 4.3, Eq. 4).

Checked against hand-worked layouts, Eq. 4 written out with the frame and
in-frame block index, the halo bound the paper derives for a multi-diagonal
mask (at most 2 delta T remote blocks per head), brute-force demand sets from
plain loops, and the contiguous counter already pinned for Eq. 3. A slip such
as a rank computed from the block index instead of its frame position, a
ragged block moved off the end, a permutation applied backwards or a demand
union taken over the wrong rows fails here.
"""

import numpy as np
import pytest

import oracle as orc


def test_eq4_hand_example_whole_blocks_per_frame():
    # 3 frames of 64 tokens, blocks of 8: B = 8 blocks per frame, G = 4 ranks.
    owner = orc.periodic_owner(L=3 * 64, block=8, frame_tokens=64, ranks=4)
    assert owner.tolist() == [0, 0, 1, 1, 2, 2, 3, 3] * 3


def test_eq4_hand_example_blocks_straddle_frames():
    # 12-token frames, 8-token blocks, 36 tokens: blocks start at 0, 8, 16, 24, 32,
    # in-frame offsets 0, 8, 4, 0, 8 -> ranks 0, 1, 0, 0; the ragged block 4 -> last rank.
    owner = orc.periodic_owner(L=36, block=8, frame_tokens=12, ranks=2)
    assert owner.tolist() == [0, 1, 0, 0, 1]
    perm, begin = orc.placement_permutation(owner, 2)
    assert perm.tolist() == [0, 2, 3, 1, 4]
    assert begin.tolist() == [0, 3, 5]


@pytest.mark.parametrize("seed", range(5))
def test_eq4_written_out_when_frames_hold_whole_blocks(seed):
    rng = np.random.default_rng(seed)
    B, b, T = int(rng.integers(2, 40)), int(rng.integers(1, 9)), int(rng.integers(1, 7))
    G = int(rng.integers(1, B + 1))
    owner = orc.periodic_owner(L=T * B * b, block=b, frame_tokens=B * b, ranks=G)
    for j in range(T * B):
        t, s = divmod(j, B)  # frame and block index inside the frame
        assert owner[j] == (G * s) // B


@pytest.mark.parametrize("seed", range(5))
def test_permutation_round_trip_and_block_contents(seed):
    rng = np.random.default_rng(10 + seed)
    b, F = int(rng.integers(2, 9)), int(rng.integers(5, 60))
    L = int(rng.integers(b + 1, 300))
    G = int(rng.integers(1, 5))
    owner = orc.periodic_owner(L, b, F, G)
    perm, begin = orc.placement_permutation(owner, G)
    inv = orc.inverse_permutation(perm)
    n = orc.num_blocks(L, b)
    assert sorted(perm.tolist()) == list(range(n))
    assert (perm[inv] == np.arange(n)).all() and (inv[perm] == np.arange(n)).all()
    assert perm[-1] == n - 1  # a ragged last block stays last
    for p in range(G):  # contiguous rank ranges in the placed order, logical order inside
        block_ids = perm[begin[p]:begin[p + 1]]
        assert (owner[block_ids] == p).all() and (np.diff(block_ids) > 0).all()
    X = rng.standard_normal((2, L, 3))
    Y = orc.permute_blocks(X, perm, L, b)
    for k in range(n):
        j = perm[k]
        c = min(b, L - j * b)
        np.testing.assert_array_equal(Y[:, k * b:k * b + c], X[:, j * b:j * b + c])
    np.testing.assert_array_equal(orc.permute_blocks(Y, inv, L, b), X)


def multi_diagonal_mask(T, B, delta, H=1):
    """Every query at in-frame position s keeps the positions [s - delta, s + delta] of every frame."""
    n = T * B
    s = np.arange(n) % B
    M = np.abs(s[:, None] - s[None, :]) <= delta
    return np.broadcast_to(M, (H, n, n)).copy()


@pytest.mark.parametrize("T,B,G,delta", [(6, 8, 4, 1), (5, 12, 3, 2), (4, 16, 4, 3), (3, 20, 5, 1)])
def test_halo_bound_on_a_multi_diagonal_mask(T, B, G, delta):
    b = 4
    M = multi_diagonal_mask(T, B, delta)
    owner = orc.periodic_owner(T * B * b, b, B * b, G)
    width = B // G
    for r in range(G):
        D = orc.rank_demand(M, owner, r)
        remote = orc.remote_blocks(D, owner, r)
        # closed form: the halo positions of [r w, (r+1) w) inside [0, B), in each of T frames
        halo = len([x for x in range(r * width - delta, (r + 1) * width + delta)
                    if 0 <= x < B and not r * width <= x < (r + 1) * width])
        assert remote == halo * T
        assert remote <= 2 * delta * T
        contiguous = orc.contiguous_owner(T * B, G)
        Dc = orc.rank_demand(M, contiguous, r)
        assert remote <= orc.remote_blocks(Dc, contiguous, r)


@pytest.mark.parametrize("seed", range(4))
def test_rank_demand_brute_force_and_contiguous_counter(seed):
    rng = np.random.default_rng(40 + seed)
    H, n, G = 2, int(rng.integers(4, 30)), int(rng.integers(1, 5))
    G = min(G, n)
    M = rng.random((H, n, n)) < 0.2
    owner = rng.integers(0, G, n)
    for r in range(G):
        D = orc.rank_demand(M, owner, r)
        for h in range(H):
            for j in range(n):
                want = any(M[h, i, j] for i in range(n) if owner[i] == r)
                assert D[h, j] == want
        want_remote = sum(1 for h in range(H) for j in range(n) if D[h, j] and owner[j] != r)
        assert orc.remote_blocks(D, owner, r) == want_remote
    contiguous = orc.contiguous_owner(n, G)
    for r in range(G):
        D = orc.rank_demand(M, contiguous, r)
        assert orc.exchange_volume(D, G, r, 8, 4, 2) == 2 * 8 * 4 * 2 * orc.remote_blocks(D, contiguous, r)
