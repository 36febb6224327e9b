"""Attention with long rows split over several workgroups
(sparsp_block_sparse_attn_split).

Splitting changes the schedule and adds one float32 merge through the
log-sum-exp, so:

* the result meets the same bar against the oracle's attention as the unsplit
  kernels (bf16 and float32 outputs, lse), for selections whose rows differ
  greatly in length, with pieces short enough that most rows split;
* with max_pieces = 0 nothing splits and the outputs equal
  sparsp_block_sparse_attn's bit for bit;
* the plan the call leaves in its workspace follows the documented rule,
  recomputed here: which rows split (the count threshold under the piece
  budget), their workspace slots (row order), the block ranges of the pieces
  (a partition of [0, n) at every T-th kept block) and the launch layout (the
  row order's eight queues, each longest item first). Items of equal length
  may come in any order, so that order is checked for validity only.
"""

import numpy as np
import pytest

import oracle as orc
import paper_2609_32197_amd as sp
from tests import _parity as P
from tests.test_gpu_kernels import _rand_inputs, ctypes_scale
from tests.test_gpu_row_order import _queues

pytestmark = pytest.mark.gpu


def _skewed_selection(seed, H, nq, n, i0):
    """Rows of very unequal length: most keep a few blocks, some nearly all.
    Every row keeps its diagonal block. Returns the boolean mask [H, nq, n],
    sel [H, nq, n] (ascending, padded with -1) and the counts [H, nq]."""
    rng = np.random.default_rng(seed)
    mask = np.zeros((H, nq, n), dtype=bool)
    for h in range(H):
        for r in range(nq):
            c = int(np.clip(round(n * rng.random() ** 4), 1, n))
            mask[h, r, rng.choice(n, c, replace=False)] = True
            mask[h, r, i0 + r] = True
    counts = mask.sum(axis=2).astype(np.int32)
    sel = np.full((H, nq, n), -1, dtype=np.int32)
    for h in range(H):
        for r in range(nq):
            idx = np.flatnonzero(mask[h, r])
            sel[h, r, :idx.size] = idx
    return mask, sel, counts


def _setup(geo, seed=7):
    H, L, d, b, i0, i1, dt = geo
    n = -(-L // b)
    q, k, v = _rand_inputs(seed, H, L, d, dt)
    g = P.geometry(H, L, d, b, i0, i1, dt)
    mask, sel, counts = _skewed_selection(seed, H, i1 - i0, n, i0)
    torch = P.torch()
    out = sp.sparsp_demand_union_gather(g, torch.from_numpy(P.words_as_int64(mask)).cuda(),
                                        P.to_device(k, dt), P.to_device(v, dt))
    dev = dict(Q=P.to_device(q, dt), sel=torch.from_numpy(sel).cuda(),
               counts=torch.from_numpy(counts).cuda(), out=out)
    return q, k, v, g, mask, sel, counts, dev


def _split(g, dev, T, Pmax, odt, ws=None):
    o = dev["out"]
    return sp.sparsp_block_sparse_attn_split(g, dev["Q"], dev["sel"], o["slot_of"], o["K_packed"],
                                             o["V_packed"], dev["counts"], T, Pmax, workspace=ws,
                                             softmax_scale=ctypes_scale(g.d), out_dtype=odt)


def _reference_plan(counts, sel, n, T, Pmax):
    """The documented plan: threshold, slots and the set of work items."""
    c = np.clip(counts.reshape(-1), 0, n).astype(np.int64)
    R, keep = c.size, sel.shape[-1]
    srows = sel.reshape(R, keep)
    T = min(T, n)
    cstar = n + 1
    for v in range(n, T, -1):  # the need only grows as the threshold falls
        if np.sum(-(-c[c >= v] // T)) <= Pmax:
            cstar = v
        else:
            break
    split = (c > T) & (c >= cstar)
    npieces = np.where(split, -(-c // T), 1)
    base = np.full(R, -1, dtype=np.int64)
    run = 0
    for r in range(R):
        if split[r]:
            base[r] = run
            run += npieces[r]
    items = {}
    for r in range(R):
        if not split[r]:
            items[(r, 0, n, -1)] = int(c[r])
            continue
        lo = 0
        for p in range(npieces[r]):
            if p + 1 < npieces[r]:
                e = (p + 1) * T
                hi = int(min(max(srows[r, e] if e < keep else n, lo), n))
            else:
                hi = n
            items[(r, lo, hi, int(base[r] + p))] = int(min(T, c[r] - p * T))
            lo = hi
    return cstar, base, items


GEOMS = [
    (3, 9000, 128, 128, 20, 71, "bf16"),   # 128-token kernel, ragged last block
    (2, 4400, 64, 128, 3, 35, "bf16"),     # 128-token kernel, d = 64
    (2, 4500, 64, 64, 30, 71, "bf16"),     # 64-token kernel
    (2, 4100, 128, 64, 0, 40, "bf16"),     # 64-token kernel, d = 128
    (3, 1000, 64, 64, 5, 16, "f32"),       # float32 kernel
    (2, 1000, 20, 32, 3, 30, "f32"),       # float32 kernel, odd shape
]
IDS = ["H{}L{}d{}b{}_{}-{}_{}".format(*g) for g in GEOMS]


@pytest.mark.parametrize("geo", GEOMS, ids=IDS)
@pytest.mark.parametrize("T", [1, 3])
def test_split_attention_parity(gpu, geo, T):
    q, k, v, g, mask, sel, counts, dev = _setup(geo)
    dt = geo[-1]
    c = counts.reshape(-1).astype(np.int64)
    need = int(np.sum(np.where(c > T, -(-c // T), 0)))
    Qf, Kf, Vf = (orc.decode_input(x, dt) for x in (q, k, v))
    O_ref, lse_ref = orc.sparse_attention(Qf, Kf, Vf, mask, g.L, g.block, g.i0, ctypes_scale(g.d))
    fin = np.isfinite(lse_ref)
    for odt in ([sp.F32, sp.BF16] if dt == "bf16" else [sp.F32]):
        O, lse = _split(g, dev, T, need + 5, odt)
        P.check_attention(O.float().cpu().numpy(), O_ref, dt == "bf16",
                          f"split T={T} {geo} out={odt}")
        ln = lse.cpu().numpy()
        assert (np.isneginf(ln) == ~fin).all()
        assert np.abs(ln[fin] - lse_ref[fin]).max() <= (1e-4 if dt == "bf16" else 1e-5)


@pytest.mark.parametrize("geo", GEOMS, ids=IDS)
def test_no_pieces_is_bit_identical(gpu, geo):
    torch = P.torch()
    q, k, v, g, mask, sel, counts, dev = _setup(geo, seed=3)
    o = dev["out"]
    for odt in ([sp.F32, sp.BF16] if geo[-1] == "bf16" else [sp.F32]):
        O0, l0 = sp.sparsp_block_sparse_attn(g, dev["Q"], dev["sel"], o["slot_of"], o["K_packed"],
                                             o["V_packed"], ctypes_scale(g.d), out_dtype=odt)
        O1, l1 = _split(g, dev, 2, 0, odt)
        bits = torch.int16 if odt == sp.BF16 else torch.int32
        assert torch.equal(O0.view(bits), O1.view(bits))
        assert torch.equal(l0.view(torch.int32), l1.view(torch.int32))


@pytest.mark.parametrize("geo", GEOMS[:1] + GEOMS[2:3] + GEOMS[4:5], ids=[IDS[0], IDS[2], IDS[4]])
@pytest.mark.parametrize("T,budget", [(2, 1.0), (3, 0.5), (4, 0.1), (1000, 1.0)])
def test_split_plan_follows_the_rule(gpu, geo, T, budget):
    torch = P.torch()
    q, k, v, g, mask, sel, counts, dev = _setup(geo, seed=11)
    n = g.n
    R = g.H * g.nq
    c = np.clip(counts.reshape(-1), 0, n).astype(np.int64)
    Tn = min(T, n)
    full = int(np.sum(np.where(c > Tn, -(-c // Tn), 0)))
    Pmax = int(budget * full)
    nbytes = sp.sparsp_split_workspace_bytes(g, Pmax)
    ws = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
    _split(g, dev, T, Pmax, sp.F32, ws=ws)
    torch.cuda.synchronize()
    up = lambda x: (x + 255) // 256 * 256
    raw = ws.cpu().numpy()
    items = raw[:(R + Pmax) * 16].view(np.int32).reshape(-1, 4)
    off = up((R + Pmax) * 16)
    base = raw[off:off + R * 4].view(np.int32)

    cstar, base_ref, items_ref = _reference_plan(counts, sel, n, T, Pmax)
    np.testing.assert_array_equal(base, base_ref)
    valid = items[:, 0] >= 0
    n_items = int(valid.sum())
    assert valid[:n_items].all() and not valid[n_items:].any()   # padding at the end
    got = [tuple(int(x) for x in it) for it in items[:n_items]]
    assert len(got) == len(set(got)) and set(got) == set(items_ref)
    # launch layout: the row order's queues, each longest item first
    q_of, _ = _queues(counts, n)
    qlen = [0] * 8
    for it in got:
        qlen[q_of[it[0] // g.nq]] += 1
    queues, pos = [[] for _ in range(8)], 0
    for kk in range(max(qlen)):
        for x in range(8):
            if kk < qlen[x]:
                queues[x].append(got[pos])
                pos += 1
    for x in range(8):
        assert all(q_of[it[0] // g.nq] == x for it in queues[x])
        lens = [items_ref[it] for it in queues[x]]
        assert lens == sorted(lens, reverse=True)


def test_split_full_size_wan_share_cdf(gpu):
    """The wan-share layer under CDF selection (tau 0.9, rows of 1 to ~280
    blocks), split at 32 blocks: the longest rows against the oracle, and every
    row against the unsplit kernel."""
    torch = P.torch()
    from workloads import get_workload, make_qkv
    wl = get_workload("wan-share")
    q, k, v = make_qkv(wl)
    g = P.geometry(wl.H, wl.L, wl.d, wl.block, wl.i0, wl.i1, wl.dtype)
    Qd, Kd, Vd = (P.to_device(x, wl.dtype) for x in (q, k, v))
    _, _, sc = sp.sparsp_block_scores(g, Qd, Kd)
    m, sel, cnt = sp.sparsp_cdf_mask(g, sc, 0.9)
    out = sp.sparsp_demand_union_gather(g, m, Kd, Vd)
    args = (g, Qd, sel, out["slot_of"], out["K_packed"], out["V_packed"])
    O0, l0 = sp.sparsp_block_sparse_attn(*args, wl.softmax_scale)
    O1, l1 = sp.sparsp_block_sparse_attn_split(*args, cnt, 32, 2048,
                                               softmax_scale=wl.softmax_scale)
    d = (O1.float() - O0.float()).abs()
    assert float(d.max()) <= 2e-2 and float(d.mean()) <= 1e-3
    fin = torch.isfinite(l0)
    assert torch.equal(fin, torch.isfinite(l1))
    assert float((l1[fin] - l0[fin]).abs().max()) <= 1e-4
    counts = cnt.cpu().numpy()
    mask = orc.words_to_mask(m.cpu().numpy().view(np.uint64), g.n)
    On = O1.float().cpu().numpy()
    longest = np.argsort(counts.reshape(-1))[::-1][:4]
    for row in longest:
        h, r = divmod(int(row), g.nq)
        qf, kf, vf = (orc.decode_input(x[h], wl.dtype) for x in (q, k, v))
        o_ref, _ = orc.attend_block(qf, kf, vf, mask[h, r], g.i0 + r, wl.L, wl.block,
                                    wl.softmax_scale)
        P.check_attention(On[h, r * wl.block:(r + 1) * wl.block], o_ref, True,
                          f"split wan-share h={h} r={r} count={counts[h, r]}")
