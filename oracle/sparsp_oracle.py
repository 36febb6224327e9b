"""Plain float64 reference for one rank's share of SparSP sparse attention.

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product path. Nothing here is
shared with the HIP library.

The computation follows the paper (arXiv 2609.32197):

* Eq. 1 (Section 2.2): attention O = softmax(Q K^T / sqrt(d)) V.
* Section 2.2: sparse attention keeps part of the scores and aggregates V
  with the kept ones; block-sparse kernels renormalise the softmax over the
  kept keys, which is what this oracle computes.
* Section 4.1: M[h, i, j] says whether query block i of head h consumes KV
  block j; Eq. 2 defines a rank's demand as the union of its local rows;
  Eq. 3 gives the bytes a rank receives.
* Section 4.2: the mask is built from pooled query and key tiles.
* Section 5.2: demand is kept per head (not unioned across heads) and blocks
  are packed row-major, each head a contiguous range, so that offsets can be
  derived locally on both ends.
* Section 5.1: a producer sends each consumer only the blocks of its shard
  that consumer demands (directly, not relayed around the ring); Section 5.2:
  per head, packed row-major, offsets derived from the shared mask on both
  ends;
* Section 8.1: the evaluation's selection rule (CDF mode) keeps, for each
  query, the highest-scoring key blocks until their cumulative attention mass
  reaches a threshold tau;
* Section 4.3, Eq. 4: the interval-periodic layout gives spatial interval
  floor(G s / B) of every frame to the same rank, realised as a block
  permutation of the sequence and its inverse;
* Section 2.3 and Section 7: a rank attends to the KV shards of the owners
  one at a time and combines the partial results with the online softmax;
  Section 7.1 keeps the local shard whole and cuts the last remote shard into
  finer chunks; Section 7.2 cuts shards into chunks of heads and runs the
  sparsest chunk last.

Readings taken where the paper is silent:

* pooling is the arithmetic mean over the valid tokens of a block;
* the block score is the pooled dot product scaled by d**-0.5, rounded to
  float32, with no softmax (softmax is monotone so top-k is unchanged);
* selection keeps, per row, the diagonal block (global index), the global
  blocks, and the best remaining blocks by (score descending, index
  ascending), keep counting every kept block; +0.0 and -0.0 tie; NaN scores
  are rejected;
* demand packs every demanded block, local and remote; the remote part is
  what Eq. 3 counts;
* the packed K buffer keeps each block as [block, d]; the packed V buffer
  stores each block transposed, [d, block]; token rows past L are zero;
* placement: a block's frame position is that of its first token, so block j
  goes to rank floor(G (j b mod F) / F) for F tokens per frame (Eq. 4 exactly
  when F is a multiple of b); a ragged last block stays last and belongs to
  the last rank; the placed order lists each rank's blocks in logical order,
  rank after rank;
* CDF mode per query block: the softmax of the row's float32 block scores over
  all n blocks; blocks ordered by (score descending, index ascending); the
  shortest prefix of that order whose mass reaches tau is kept, then the
  diagonal and global blocks are added; tau in (0, 1]. "Reaches tau" is
  decided on the mass the prefix leaves out (at most (1 - tau) of the total),
  summed from the smallest block upward, and tau = 1 keeps every block, since
  every block's softmax mass is positive; the scores must be finite;
* a chunk is (owner shard, run of consecutive heads); shards are taken in
  ring order from the local one (r, r+1, ..., r+R-1 mod R); remote shards are
  cut into chunks of a given number of heads, the last remote shard into
  chunks of a second, smaller number; inside each remote shard, chunks run
  in order of selected blocks descending (the heads' demanded blocks in that
  shard), ties by head, so that the sparsest chunk of the last shard ends the
  pipeline.

Precision: every arithmetic step is float64; the float32 block scores are the
hand-off value for selection. Attention is evaluated directly from Q, K, V
through the mask (not through the packed buffers) so that it also checks the
packing and slot map of the GPU path.
"""

from __future__ import annotations

import math
from typing import Iterable, Optional, Sequence

import numpy as np

__all__ = [
    "decode_bf16",
    "decode_input",
    "num_blocks",
    "block_valid_counts",
    "local_range",
    "pool_blocks",
    "block_scores",
    "forced_blocks",
    "select_topk",
    "mask_to_words",
    "words_to_mask",
    "demand_union",
    "packing_plan",
    "pack_kv",
    "attend_block",
    "sparse_attention",
    "dense_attention",
    "attention_flops",
    "exchange_volume",
    "owner_ranges",
    "attend_part",
    "lse_merge",
    "chunk_plan",
    "chunked_attention",
    "periodic_owner",
    "contiguous_owner",
    "placement_permutation",
    "inverse_permutation",
    "permute_blocks",
    "rank_demand",
    "remote_blocks",
    "cdf_order_and_mass",
    "cdf_cut",
    "select_cdf",
    "provide_masks",
    "pack_by_consumer",
    "route_volume",
]


# ---------------------------------------------------------------------------
# number formats
# ---------------------------------------------------------------------------

def decode_bf16(bits: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) -> float64, exactly.

    A bfloat16 is the upper half of a float32: shift the 16 bits up and
    reinterpret.
    """
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def decode_input(x: np.ndarray, dtype: str) -> np.ndarray:
    """Decode a generator tensor ('bf16' bits or 'f32' values) to float64."""
    if dtype == "bf16":
        return decode_bf16(x)
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")


# ---------------------------------------------------------------------------
# geometry
# ---------------------------------------------------------------------------

def num_blocks(L: int, block: int) -> int:
    """n = ceil(L / b): blocks of b tokens, the last one possibly partial."""
    return -(-L // block)


def block_valid_counts(L: int, block: int) -> np.ndarray:
    """c_j = min(b, L - j*b): the number of real tokens in block j."""
    n = num_blocks(L, block)
    return np.minimum(block, L - block * np.arange(n))


def local_range(n: int, ranks: int, rank: int) -> tuple:
    """Contiguous block ownership: rank r owns [floor(r n / R), floor((r+1) n / R))."""
    return rank * n // ranks, (rank + 1) * n // ranks


# ---------------------------------------------------------------------------
# Section 4.2: pooled tiles and block scores
# ---------------------------------------------------------------------------

def pool_blocks(X: np.ndarray, L: int, block: int,
                blocks: Optional[Iterable[int]] = None) -> np.ndarray:
    """Mean of each token block over its valid tokens.

    X: float64 [H, L, d]. Returns float64 [H, len(blocks), d] (all n blocks by
    default). Tokens past L do not exist and are not averaged in.
    """
    n = num_blocks(L, block)
    if blocks is None:
        blocks = range(n)
    out = []
    for j in blocks:
        lo, hi = j * block, min((j + 1) * block, L)
        out.append(X[:, lo:hi, :].mean(axis=1))
    return np.stack(out, axis=1)


def block_scores(pooled_q: np.ndarray, pooled_k: np.ndarray, d: int) -> np.ndarray:
    """S[h, i, j] = <q_bar[h, i], k_bar[h, j]> * d**-0.5, in float64, then rounded to float32."""
    s = np.matmul(pooled_q, np.swapaxes(pooled_k, 1, 2)) * (1.0 / math.sqrt(d))
    return s.astype(np.float32)


# ---------------------------------------------------------------------------
# Section 4.1: the block mask M[h, i, j] by top-k selection
# ---------------------------------------------------------------------------

def forced_blocks(i: int, global_blocks: Sequence[int]) -> set:
    """F_i = {i} U G: the diagonal block (global index i) and every global block."""
    return {int(i)} | {int(g) for g in global_blocks}


def select_topk(scores: np.ndarray, keep: int, i0: int,
                global_blocks: Sequence[int] = ()) -> tuple:
    """Top-k block selection with a forced diagonal and lowest-index tie-break.

    scores: float32 [H, nq, n]; row r is global query block i = i0 + r.
    Each row keeps F_i plus the first keep - |F_i| candidates (blocks not in
    F_i) ordered by score descending, then block index ascending; scores are
    compared as float32 values, so +0.0 and -0.0 are equal.

    Returns (mask bool [H, nq, n], sel int32 [H, nq, keep] ascending).
    """
    s = np.asarray(scores)
    if s.dtype != np.float32:
        raise TypeError("scores must be float32")
    if np.isnan(s).any():
        raise ValueError("NaN block score")
    H, nq, n = s.shape
    G = sorted({int(g) for g in global_blocks})
    if any(g < 0 or g >= n for g in G):
        raise ValueError("global block out of range")
    if keep > n:
        raise ValueError("keep > n")
    if i0 < 0 or i0 + nq > n:
        raise ValueError("local query blocks out of range")

    forced = np.zeros((nq, n), dtype=bool)
    for r in range(nq):
        for j in forced_blocks(i0 + r, G):
            forced[r, j] = True
    n_forced = forced.sum(axis=1)
    if (keep < n_forced).any():
        raise ValueError("keep smaller than the forced set of some row")
    take = keep - n_forced  # candidates to take per row

    forced3 = np.broadcast_to(forced, (H, nq, n))
    index = np.broadcast_to(np.arange(n), (H, nq, n))
    neg_score = -s.astype(np.float64)
    # lexsort: last key is primary. Candidates first, then score descending,
    # then index ascending.
    order = np.lexsort((index, neg_score, forced3), axis=-1)
    rank = np.empty_like(order)
    np.put_along_axis(rank, order, np.broadcast_to(np.arange(n), (H, nq, n)), axis=-1)
    taken = (~forced3) & (rank < take[None, :, None])
    mask = forced3 | taken
    sel = np.nonzero(mask)[2].reshape(H, nq, keep).astype(np.int32)
    return mask, sel


def mask_to_words(mask: np.ndarray) -> np.ndarray:
    """Bit j % 64 of word j // 64 stands for block j. bool [..., n] -> uint64 [..., ceil(n/64)]."""
    n = mask.shape[-1]
    W = -(-n // 64)
    words = np.zeros(mask.shape[:-1] + (W,), dtype=np.uint64)
    for j in range(n):
        bit = np.uint64(1) << np.uint64(j % 64)
        words[..., j // 64] |= np.where(mask[..., j], bit, np.uint64(0))
    return words


def words_to_mask(words: np.ndarray, n: int) -> np.ndarray:
    """Inverse of mask_to_words."""
    w = np.asarray(words, dtype=np.uint64)
    out = np.zeros(w.shape[:-1] + (n,), dtype=bool)
    for j in range(n):
        out[..., j] = ((w[..., j // 64] >> np.uint64(j % 64)) & np.uint64(1)) == 1
    return out


# ---------------------------------------------------------------------------
# Eq. 2 and Section 5.2: per-head demand and the packing plan
# ---------------------------------------------------------------------------

def demand_union(mask: np.ndarray) -> np.ndarray:
    """D_h = union over local rows i of {j : M[h, i, j] = 1}, over all owners.

    Demand is kept per head (Section 5.2). mask bool [H, nq, n] -> bool [H, n].
    """
    return np.any(mask, axis=1)


def packing_plan(demand: np.ndarray) -> tuple:
    """Row-major packing order: head-major, block index ascending.

    Returns head_off int32 [H+1] (exclusive scan of U_h = |D_h|),
    gather_blk int32 [sum U_h] (each head's demanded blocks, ascending,
    heads concatenated) and slot_of int32 [H, n] (slot of block j of head h
    in the packed buffer, -1 when not demanded).
    """
    H, n = demand.shape
    U = demand.sum(axis=1)
    head_off = np.zeros(H + 1, dtype=np.int64)
    head_off[1:] = np.cumsum(U)
    gather_blk = []
    slot_of = np.full((H, n), -1, dtype=np.int64)
    for h in range(H):
        blocks = np.nonzero(demand[h])[0]
        gather_blk.extend(blocks.tolist())
        slot_of[h, blocks] = head_off[h] + np.arange(len(blocks))
    return (head_off.astype(np.int32), np.asarray(gather_blk, dtype=np.int32),
            slot_of.astype(np.int32))


def pack_kv(K: np.ndarray, V: np.ndarray, head_off: np.ndarray, gather_blk: np.ndarray,
            L: int, block: int) -> tuple:
    """Copy the demanded blocks into the packed buffers, bit for bit.

    K, V: raw element arrays [H, L, d] (bf16 bit patterns or float32).
    Returns K_packed [S, block, d] and V_packed [S, d, block]: slot s holds
    block gather_blk[s] of its head; the V block is stored transposed; token
    rows past L are zero.
    """
    H, _, d = K.shape
    S = int(head_off[-1])
    Kp = np.zeros((S, block, d), dtype=K.dtype)
    Vp = np.zeros((S, d, block), dtype=V.dtype)
    for h in range(H):
        for s in range(int(head_off[h]), int(head_off[h + 1])):
            j = int(gather_blk[s])
            lo, hi = j * block, min((j + 1) * block, L)
            Kp[s, : hi - lo, :] = K[h, lo:hi, :]
            Vp[s, :, : hi - lo] = V[h, lo:hi, :].T
    return Kp, Vp


# ---------------------------------------------------------------------------
# Eq. 1 restricted to the kept blocks: block-sparse attention
# ---------------------------------------------------------------------------

def _softmax_attend(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float):
    """Rows of softmax(q k^T * scale) v, with the log-sum-exp of each row."""
    s = (q @ k.T) * scale
    m = s.max(axis=1, keepdims=True)
    e = np.exp(s - m)
    l = e.sum(axis=1, keepdims=True)
    return (e @ v) / l, (m + np.log(l))[:, 0], e / l


def attend_block(Qh: np.ndarray, Kh: np.ndarray, Vh: np.ndarray, mask_row: np.ndarray,
                 i: int, L: int, block: int, scale: float, return_probs: bool = False):
    """Attention of query block i of one head over the valid tokens of its kept blocks.

    Qh, Kh, Vh: float64 [L, d]; mask_row: bool [n]. Returns O [block, d] and
    lse [block] (natural log); query rows past L get O = 0 and lse = -inf.
    With return_probs, also the [valid queries, kept tokens] probabilities and
    the kept token indices.
    """
    n = mask_row.shape[0]
    d = Qh.shape[1]
    tokens = np.concatenate([np.arange(j * block, min((j + 1) * block, L))
                             for j in range(n) if mask_row[j]])
    q_lo, q_hi = i * block, min((i + 1) * block, L)
    o, lse, p = _softmax_attend(Qh[q_lo:q_hi], Kh[tokens], Vh[tokens], scale)
    O = np.zeros((block, d))
    LSE = np.full(block, -np.inf)
    O[: q_hi - q_lo] = o
    LSE[: q_hi - q_lo] = lse
    if return_probs:
        return O, LSE, p, tokens
    return O, LSE


def sparse_attention(Q: np.ndarray, K: np.ndarray, V: np.ndarray, mask: np.ndarray,
                     L: int, block: int, i0: int, scale: float,
                     pairs: Optional[Iterable[tuple]] = None):
    """Block-sparse attention of the local query blocks.

    Q, K, V: float64 [H, L, d] (Q may also be given for all tokens; only the
    local blocks are read). mask: bool [H, nq, n] for rows i0 .. i0+nq-1.
    Returns O [H, nq*block, d] and lse [H, nq*block]. With ``pairs`` (an
    iterable of (h, local row) pairs) only those query blocks are evaluated;
    the rest of O and lse are NaN.
    """
    H, nq, n = mask.shape
    d = Q.shape[2]
    O = np.full((H, nq * block, d), np.nan)
    LSE = np.full((H, nq * block), np.nan)
    if pairs is None:
        pairs = [(h, r) for h in range(H) for r in range(nq)]
    for h, r in pairs:
        o, lse = attend_block(Q[h], K[h], V[h], mask[h, r], i0 + r, L, block, scale)
        O[h, r * block:(r + 1) * block] = o
        LSE[h, r * block:(r + 1) * block] = lse
    return O, LSE


def dense_attention(Q: np.ndarray, K: np.ndarray, V: np.ndarray, scale: float) -> np.ndarray:
    """Eq. 1 over all tokens of every head: softmax(Q K^T * scale) V."""
    return np.stack([_softmax_attend(Q[h], K[h], V[h], scale)[0] for h in range(Q.shape[0])])


def attention_flops(mask: np.ndarray, L: int, block: int, i0: int, d: int) -> int:
    """Algorithmic FLOPs of the kept tiles: 4 d c_i c_j per kept (i, j) (QK^T and PV)."""
    c = block_valid_counts(L, block).astype(np.int64)
    H, nq, n = mask.shape
    ci = c[i0:i0 + nq]
    per_row = mask.astype(np.int64) @ c  # [H, nq]: valid keys per row
    return int(4 * d * (per_row * ci[None, :]).sum())


# ---------------------------------------------------------------------------
# Eq. 3: bytes received by rank r
# ---------------------------------------------------------------------------

def exchange_volume(demand: np.ndarray, ranks: int, rank: int, block: int, d: int,
                    w: int) -> int:
    """V_r = 2 b d w sum_h sum_{p != r} |D_{r,h,p}| under contiguous ownership.

    Block j is owned by the rank p with floor(p n / R) <= j < floor((p+1) n / R).
    """
    H, n = demand.shape
    owner = np.empty(n, dtype=np.int64)
    for p in range(ranks):
        lo, hi = local_range(n, ranks, p)
        owner[lo:hi] = p
    remote = demand & (owner[None, :] != rank)
    return int(2 * block * d * w * remote.sum())


# ---------------------------------------------------------------------------
# Section 2.3 and Section 7: attention shard by shard, chunks of heads, and the
# online-softmax merge of the partial results
# ---------------------------------------------------------------------------

def owner_ranges(n: int, ranks: int) -> list:
    """[(lo, hi)] per owner p: the contiguous blocks [floor(p n / R), floor((p+1) n / R))."""
    return [local_range(n, ranks, p) for p in range(ranks)]


def attend_part(Qh: np.ndarray, Kh: np.ndarray, Vh: np.ndarray, mask_row: np.ndarray, i: int,
                L: int, block: int, scale: float, kv_range: tuple):
    """Attention of query block i over the kept blocks that lie in [lo, hi) only.

    The softmax and its log-sum-exp run over that part of the kept keys alone.
    Rows with no kept key in the range get O = 0 and lse = -inf, the identity
    of the merge below.
    """
    lo, hi = kv_range
    part = mask_row.copy()
    part[:lo] = False
    part[hi:] = False
    d = Qh.shape[1]
    if not part.any():
        return np.zeros((block, d)), np.full(block, -np.inf)
    return attend_block(Qh, Kh, Vh, part, i, L, block, scale)


def lse_merge(O_a: np.ndarray, lse_a: np.ndarray, O_b: np.ndarray, lse_b: np.ndarray) -> tuple:
    """Softmax results over two disjoint key sets A and B -> the result over A u B.

    With Z_X = exp(lse_X) the softmax denominator over X and O_X its weighted
    mean of V: O = (Z_A O_A + Z_B O_B) / (Z_A + Z_B), lse = log(Z_A + Z_B),
    evaluated relative to m = max(lse_A, lse_B). A row with lse = -inf on one
    side takes the other side unchanged; on both sides it stays O = 0, -inf.
    Shapes: O [..., d], lse [...].
    """
    m = np.maximum(lse_a, lse_b)
    finite = np.isfinite(m)
    m_safe = np.where(finite, m, 0.0)
    w_a = np.where(np.isfinite(lse_a), np.exp(lse_a - m_safe), 0.0)
    w_b = np.where(np.isfinite(lse_b), np.exp(lse_b - m_safe), 0.0)
    tot = w_a + w_b
    safe = np.where(finite, tot, 1.0)
    O = np.where(finite[..., None], (w_a[..., None] * O_a + w_b[..., None] * O_b) / safe[..., None],
                 0.0)
    lse = np.where(finite, m_safe + np.log(safe), -np.inf)
    return O, lse


def chunk_plan(demand: np.ndarray, ranks: int, rank: int, heads_per_chunk: int,
               tail_heads_per_chunk: int) -> list:
    """Chunk schedule of rank r's attention (Section 7.1, Section 7.2).

    demand: bool [H, n]. Returns [(owner, lo, hi, h_begin, h_end, blocks)] in
    execution order: the local shard (owner r, all heads) first, then the
    remote shards in ring order r+1, ..., r+R-1 (mod R). A remote shard is cut
    into runs of heads_per_chunk heads (the last one of the pipeline into runs
    of tail_heads_per_chunk), and its chunks run by selected blocks
    descending, then head ascending. `blocks` counts the demanded blocks of
    the chunk's heads inside the shard.
    """
    H, n = demand.shape
    if heads_per_chunk < 1 or tail_heads_per_chunk < 1:
        raise ValueError("chunk sizes must be positive")
    if not 0 <= rank < ranks:
        raise ValueError("rank out of range")
    rng = owner_ranges(n, ranks)
    plan = []
    lo, hi = rng[rank]
    plan.append((rank, lo, hi, 0, H, int(demand[:, lo:hi].sum())))
    for k in range(1, ranks):
        p = (rank + k) % ranks
        lo, hi = rng[p]
        size = tail_heads_per_chunk if k == ranks - 1 else heads_per_chunk
        chunks = []
        for h0 in range(0, H, size):
            h1 = min(H, h0 + size)
            chunks.append((p, lo, hi, h0, h1, int(demand[h0:h1, lo:hi].sum())))
        chunks.sort(key=lambda c: (-c[5], c[3]))
        plan.extend(chunks)
    return plan


def chunked_attention(Q: np.ndarray, K: np.ndarray, V: np.ndarray, mask: np.ndarray, L: int,
                      block: int, i0: int, scale: float, plan: Sequence[tuple],
                      pairs: Optional[Iterable[tuple]] = None) -> tuple:
    """Block-sparse attention evaluated chunk by chunk in `plan` order and merged.

    Every chunk attends the query blocks of its heads to the kept blocks inside
    its shard (attend_part) and is folded into the running result with
    lse_merge. With ``pairs`` only those (h, local row) query blocks are
    evaluated; the rest of O and lse are NaN.
    """
    H, nq, n = mask.shape
    d = Q.shape[2]
    want = set(pairs) if pairs is not None else None
    O = np.zeros((H, nq * block, d))
    LSE = np.full((H, nq * block), -np.inf)
    for (_, lo, hi, h0, h1, _) in plan:
        for h in range(h0, h1):
            for r in range(nq):
                if want is not None and (h, r) not in want:
                    continue
                rows = slice(r * block, (r + 1) * block)
                o, l = attend_part(Q[h], K[h], V[h], mask[h, r], i0 + r, L, block, scale, (lo, hi))
                O[h, rows], LSE[h, rows] = lse_merge(O[h, rows], LSE[h, rows], o, l)
    if want is not None:
        keep_rows = np.zeros((H, nq * block), dtype=bool)
        for h, r in want:
            keep_rows[h, r * block:(r + 1) * block] = True
        O[~keep_rows] = np.nan
        LSE[~keep_rows] = np.nan
    return O, LSE


# ---------------------------------------------------------------------------
# Section 4.3, Eq. 4: dependency-aware (interval-periodic) placement
# ---------------------------------------------------------------------------

def periodic_owner(L: int, block: int, frame_tokens: int, ranks: int) -> np.ndarray:
    """Owner of every logical block under Eq. 4: floor(G s / B).

    With F = frame_tokens and s / B read as the spatial offset of the block's
    first token inside its frame over the frame size, block j goes to
    floor(G ((j b) mod F) / F). A ragged last block belongs to the last rank.
    """
    n = num_blocks(L, block)
    j = np.arange(n, dtype=np.int64)
    owner = (ranks * ((j * block) % frame_tokens)) // frame_tokens
    if L % block:
        owner[n - 1] = ranks - 1
    return owner.astype(np.int64)


def contiguous_owner(n: int, ranks: int) -> np.ndarray:
    """Owner of every block when rank p holds [floor(p n / R), floor((p+1) n / R))."""
    owner = np.empty(n, dtype=np.int64)
    for p in range(ranks):
        lo, hi = local_range(n, ranks, p)
        owner[lo:hi] = p
    return owner


def placement_permutation(owner: np.ndarray, ranks: int) -> tuple:
    """The placed order: rank 0's blocks in logical order, then rank 1's, ...

    Returns (perm, rank_begin): perm[k] is the logical block at placed
    position k, and rank p holds the placed positions [rank_begin[p],
    rank_begin[p+1]).
    """
    perm = np.concatenate([np.nonzero(owner == p)[0] for p in range(ranks)]).astype(np.int64)
    counts = np.array([(owner == p).sum() for p in range(ranks)], dtype=np.int64)
    rank_begin = np.concatenate([[0], np.cumsum(counts)])
    return perm, rank_begin


def inverse_permutation(perm: np.ndarray) -> np.ndarray:
    """inv[perm[k]] = k."""
    inv = np.empty_like(perm)
    inv[perm] = np.arange(perm.shape[0], dtype=perm.dtype)
    return inv


def permute_blocks(X: np.ndarray, perm: np.ndarray, L: int, block: int) -> np.ndarray:
    """Token tensor [H, L, d] in placed order: placed block k holds logical block perm[k].

    Block membership is unchanged (whole blocks move); the ragged last block,
    if any, is the last logical block and stays last.
    """
    Y = np.empty_like(X)
    for k, j in enumerate(perm):
        c = min(block, L - int(j) * block)
        assert c == min(block, L - k * block), "only the last block may be ragged"
        Y[:, k * block:k * block + c] = X[:, int(j) * block:int(j) * block + c]
    return Y


def rank_demand(mask_all: np.ndarray, owner: np.ndarray, rank: int) -> np.ndarray:
    """Eq. 2 over every owner: D_r[h, j] = exists i with owner(i) = r and M[h, i, j].

    mask_all: bool [H, n, n] over every query block (logical indices).
    Returns bool [H, n]; D_{r,h,p} is its restriction to owner(j) = p.
    """
    rows = owner == rank
    return mask_all[:, rows, :].any(axis=1)


def remote_blocks(demand: np.ndarray, owner: np.ndarray, rank: int) -> int:
    """sum over h and p != r of |D_{r,h,p}|: Eq. 3's block count (times 2 b d w for bytes)."""
    return int((demand & (owner[None, :] != rank)).sum())


# ---------------------------------------------------------------------------
# Section 8.1: CDF-mode selection (cumulative attention mass up to tau)
# ---------------------------------------------------------------------------

def cdf_order_and_mass(score_row: np.ndarray) -> tuple:
    """The CDF order of one row and the softmax mass each prefix leaves out.

    score_row: float32 [n]. Returns (order, left, Z): order int64 [n] lists the
    blocks by score descending, then index ascending; p_j = exp(S_j - max S)
    (unnormalised softmax weights) and Z = sum_j p_j; left float64 [n + 1] is
    the mass left out by the first k blocks of the order, left[k] = sum of
    p over order[k:], summed from the smallest weight upward (so a prefix's
    left-out mass is resolved down to the smallest weight, not to the rounding
    of a running total near Z); left[0] = Z and left[n] = 0.
    """
    s = np.asarray(score_row)
    if s.dtype != np.float32:
        raise TypeError("scores must be float32")
    if not np.isfinite(s).all():
        raise ValueError("non-finite block score")
    s64 = s.astype(np.float64)
    order = np.lexsort((np.arange(s.shape[0]), -s64))
    p = np.exp(s64 - s64.max())[order]
    left = np.zeros(s.shape[0] + 1, dtype=np.float64)
    left[:-1] = np.cumsum(p[::-1])[::-1]
    return order.astype(np.int64), left, float(left[0])


def cdf_cut(left: np.ndarray, Z: float, tau: float) -> int:
    """Length of the shortest prefix of the CDF order whose mass reaches tau Z.

    A prefix's mass reaches tau Z exactly when the mass it leaves out is at
    most (1 - tau) Z. Every block carries strictly positive mass, so tau = 1
    keeps all n blocks (float64 exp can underflow to 0 for very low scores;
    the definition, not the rounding, decides that case).
    """
    n = left.shape[0] - 1
    if tau >= 1.0:
        return n
    budget = (1.0 - tau) * Z
    return int(np.argmax(left[1:] <= budget)) + 1  # left[n] = 0, so some k qualifies


def select_cdf(scores: np.ndarray, tau: float, i0: int, global_blocks: Sequence[int] = ()) -> tuple:
    """CDF-mode block mask: the shortest prefix of the CDF order with mass >= tau, plus F_i.

    scores: float32 [H, nq, n]; row r is global query block i0 + r. Returns
    (mask bool [H, nq, n], sel int32 [H, nq, n]: each row's kept blocks
    ascending then -1, counts int32 [H, nq]).
    """
    if not 0.0 < tau <= 1.0:
        raise ValueError("tau must be in (0, 1]")
    s = np.asarray(scores)
    H, nq, n = s.shape
    G = sorted({int(g) for g in global_blocks})
    if any(g < 0 or g >= n for g in G):
        raise ValueError("global block out of range")
    mask = np.zeros((H, nq, n), dtype=bool)
    for h in range(H):
        for r in range(nq):
            order, left, Z = cdf_order_and_mass(s[h, r])
            k = cdf_cut(left, Z, tau)
            mask[h, r, order[:k]] = True
            for j in forced_blocks(i0 + r, G):
                mask[h, r, j] = True
    counts = mask.sum(axis=2).astype(np.int32)
    sel = np.full((H, nq, n), -1, dtype=np.int32)
    for h in range(H):
        for r in range(nq):
            idx = np.nonzero(mask[h, r])[0]
            sel[h, r, :idx.size] = idx
    return mask, sel, counts


# ---------------------------------------------------------------------------
# Section 5: demand-directed KV routing, producer side
# ---------------------------------------------------------------------------

def provide_masks(demands: Sequence[np.ndarray], ranks: int, producer: int) -> list:
    """What producer p sends to each consumer (Eq. 2's D_{c,h,p}), in ring order.

    demands: one bool [H, n] per rank c, the union of c's kept blocks over its
    query blocks. Returns [(c, bool [H, n])] for c = p+1, ..., p+R-1 (mod R):
    c's demand restricted to p's shard [floor(p n / R), floor((p+1) n / R)).
    """
    H, n = demands[producer].shape
    lo, hi = local_range(n, ranks, producer)
    out = []
    for k in range(1, ranks):
        c = (producer + k) % ranks
        m = np.zeros((H, n), dtype=bool)
        m[:, lo:hi] = demands[c][:, lo:hi]
        out.append((c, m))
    return out


def pack_by_consumer(provides: Sequence[tuple], K: np.ndarray, V: np.ndarray, L: int,
                     block: int) -> dict:
    """Producer-side packing for every consumer, consumers in the given order.

    Each consumer's blocks are packed per head, head-major, block ascending
    (Section 5.2), consumer after consumer: virtual head v = (consumer index)
    * H + h. Returns head_off [C*H + 1] (slot offsets of each (consumer, head)
    run), gather_blk (block per slot), cons_off [C + 1] (first slot of each
    consumer) and the packed K [slots, block, d] and V (transposed blocks).
    """
    H = K.shape[0]
    C = len(provides)
    stacked = np.concatenate([m for _, m in provides], axis=0) if C else np.zeros((0, K.shape[1]))
    head_off, gather_blk, _ = packing_plan(stacked)
    Kr = np.concatenate([K] * C, axis=0) if C else K[:0]
    Vr = np.concatenate([V] * C, axis=0) if C else V[:0]
    Kp, Vp = pack_kv(Kr, Vr, head_off, gather_blk, L, block)
    cons_off = head_off[::H] if C else np.zeros(1, dtype=head_off.dtype)
    return {"head_off": head_off, "gather_blk": gather_blk, "cons_off": cons_off,
            "K_packed": Kp, "V_packed": Vp}


def route_volume(provides: Sequence[tuple], shard_blocks: int) -> dict:
    """Block transfers of one producer's shard under three routings (Section 5.1).

    provides: [(c, bool [H, n])] in ring order (distance 1, 2, ...). Counts, in
    block-hops summed over heads:
      dense: the whole shard crosses every one of the R-1 hops;
      relay: hop k carries the blocks still needed by consumers at distance
             >= k (the union of their demands);
      direct: each consumer receives exactly its own blocks once.
    """
    C = len(provides)
    if C == 0:
        return {"dense": 0, "relay": 0, "direct": 0}
    H = provides[0][1].shape[0]
    relay = 0
    for k in range(C):
        downstream = np.zeros_like(provides[0][1])
        for _, m in provides[k:]:
            downstream |= m
        relay += int(downstream.sum())
    direct = int(sum(int(m.sum()) for _, m in provides))
    return {"dense": C * H * shard_blocks, "relay": relay, "direct": direct}
