"""GPU parity of shard-by-shard attention (Section 2.3, Section 7) against the oracle.

* sparsp_block_sparse_attn_part against oracle.attend_part, for shards that
  hold some, none and all of the kept blocks, and runs of heads;
* sparsp_lse_merge against oracle.lse_merge, empty rows on either side
  included;
* the part call's accumulate mode (the merge done inside the attention
  kernel) against the oracle's part over the union of the shards;
* sparsp_chunked_attn over a whole schedule against the unchunked float64
  result (the merged result must equal the unchunked one to 1e-5 on the fp32
  path), and on the bf16 path against the oracle and against the GPU's own
  unchunked call, at the small geometries and on the full wan-share share.
"""

import math

import numpy as np
import pytest

import oracle as orc
import paper_2609_32197_amd as sp
from tests import _parity as P
from tests.test_gpu_kernels import _rand_inputs

pytestmark = pytest.mark.gpu

F32_TOL = 1e-5

# (H, L, d, block, i0, i1, dtype)
GEOMS = [
    (3, 1000, 64, 64, 5, 16, "f32"),
    (2, 1024, 128, 64, 0, 16, "f32"),
    (3, 9000, 128, 128, 20, 71, "bf16"),
    (2, 4500, 64, 64, 30, 71, "bf16"),
]
IDS = ["H{}L{}d{}b{}_{}-{}_{}".format(*g) for g in GEOMS]


def _setup(geo, seed, keep_frac=0.3):
    H, L, d, b, i0, i1, dt = geo
    q, k, v = _rand_inputs(seed, H, L, d, dt)
    g = P.geometry(H, L, d, b, i0, i1, dt)
    n = g.n
    keep = max(1, int(round(keep_frac * n)))
    scores = np.random.default_rng(seed + 99).standard_normal((H, i1 - i0, n)).astype(np.float32)
    mask, _ = orc.select_topk(scores, keep, i0)
    m, sel = sp.sparsp_topk_mask(g, P.to_device(scores, "f32"), keep)
    Qd, Kd, Vd = (P.to_device(x, dt) for x in (q, k, v))
    out = sp.sparsp_demand_union_gather(g, m, Kd, Vd)
    Qf, Kf, Vf = (orc.decode_input(x, dt) for x in (q, k, v))
    scale = float(np.float32(1.0 / math.sqrt(d)))
    return g, mask, sel, out, Qd, (Qf, Kf, Vf), scale


def _check(got, ref, bf16, what):
    got = np.asarray(got, dtype=np.float64)
    if bf16:
        P.check_attention(got, ref, True, what)
    else:
        err = np.abs(got - ref)
        assert err.max() <= F32_TOL, f"{what}: max {err.max():.3g}"


@pytest.mark.parametrize("geo", GEOMS, ids=IDS)
def test_part_matches_oracle(gpu, geo):
    g, mask, sel, out, Qd, (Qf, Kf, Vf), scale = _setup(geo, 3)
    bf16 = g.dtype == sp.BF16
    n, b, i0 = g.n, g.block, g.i0
    for (lo, hi), (h0, h1) in [((0, n), (0, g.H)), ((n // 3, 2 * n // 3), (1, g.H)),
                               ((0, 1), (0, 1)), ((n - 1, n), (g.H - 1, g.H)),
                               ((5, 5), (0, g.H))]:
        O, lse = sp.sparsp_block_sparse_attn_part(g, Qd, sel, out["slot_of"], out["K_packed"],
                                                  out["V_packed"], (lo, hi), (h0, h1), scale)
        O, lse = O.cpu().numpy(), lse.cpu().numpy()
        for h in range(h0, h1):
            for r in range(g.nq):
                o_ref, l_ref = orc.attend_part(Qf[h], Kf[h], Vf[h], mask[h, r], i0 + r, g.L, b,
                                               scale, (lo, hi))
                rows = slice(r * b, (r + 1) * b)
                _check(O[h, rows], o_ref, bf16, f"part [{lo},{hi}) h={h} r={r}")
                empty = np.isneginf(l_ref)
                assert (np.isneginf(lse[h, rows]) == empty).all()
                tol = 1e-4 if bf16 else 1e-5
                assert np.abs(lse[h, rows][~empty] - l_ref[~empty]).max(initial=0) <= tol


@pytest.mark.parametrize("geo", GEOMS, ids=IDS)
def test_part_accumulate_folds_like_the_merge(gpu, geo):
    import torch
    g, mask, sel, out, Qd, (Qf, Kf, Vf), scale = _setup(geo, 4)
    bf16 = g.dtype == sp.BF16
    n, b, i0 = g.n, g.block, g.i0
    cut1, cut2 = n // 4, (3 * n) // 5
    args = (g, Qd, sel, out["slot_of"], out["K_packed"], out["V_packed"])
    # (a) write [cut1, cut2) for all heads, fold in [0, cut1) then [cut2, n) for heads 1..H-1
    O, lse = sp.sparsp_block_sparse_attn_part(*args, (cut1, cut2), (0, g.H), scale)
    sp.sparsp_block_sparse_attn_part(*args, (0, cut1), (1, g.H), scale, O=O, lse=lse,
                                     accumulate=True)
    sp.sparsp_block_sparse_attn_part(*args, (cut2, n), (1, g.H), scale, O=O, lse=lse,
                                     accumulate=True)
    # (b) fold one shard into the empty result
    O2 = torch.zeros_like(O)
    lse2 = torch.full_like(lse, -math.inf)
    sp.sparsp_block_sparse_attn_part(*args, (cut1, n), (0, g.H), scale, O=O2, lse=lse2,
                                     accumulate=True)
    O, lse, O2, lse2 = (x.cpu().numpy() for x in (O, lse, O2, lse2))
    for h in range(g.H):
        rng_a = (0, n) if h >= 1 else (cut1, cut2)
        for r in range(g.nq):
            rows = slice(r * b, (r + 1) * b)
            for got_o, got_l, kv in ((O, lse, rng_a), (O2, lse2, (cut1, n))):
                o_ref, l_ref = orc.attend_part(Qf[h], Kf[h], Vf[h], mask[h, r], i0 + r, g.L, b,
                                               scale, kv)
                _check(got_o[h, rows], o_ref, bf16, f"accumulate h={h} r={r} {kv}")
                empty = np.isneginf(l_ref)
                assert (np.isneginf(got_l[h, rows]) == empty).all()
                tol = 1e-4 if bf16 else 1e-5
                assert np.abs(got_l[h, rows][~empty] - l_ref[~empty]).max(initial=0) <= tol


def test_merge_matches_oracle(gpu):
    import torch
    rng = np.random.default_rng(5)
    H, nq, b, d = 3, 4, 64, 128
    g = sp.Geometry(H, 4 * 64 * 4, d, b, 0, nq, sp.F32)
    shape_o, shape_l = (H, nq * b, d), (H, nq * b)
    Oa, Ob = rng.standard_normal(shape_o), rng.standard_normal(shape_o)
    la, lb = rng.standard_normal(shape_l) * 4, rng.standard_normal(shape_l) * 4
    la[:, ::7] = -np.inf                      # empty on the accumulator side
    lb[:, ::5] = -np.inf                      # empty on the part side (both every 35th row)
    Oa[np.isneginf(la)] = 0.0
    Ob[np.isneginf(lb)] = 0.0
    dev = lambda x: torch.from_numpy(x.astype(np.float32)).cuda()
    O_acc, l_acc, O_p, l_p = dev(Oa), dev(la), dev(Ob), dev(lb)
    sp.sparsp_lse_merge(g, (1, 3), O_acc, l_acc, O_p, l_p)
    ref_o, ref_l = orc.lse_merge(Oa.astype(np.float32).astype(np.float64),
                                 la.astype(np.float32).astype(np.float64),
                                 Ob.astype(np.float32).astype(np.float64),
                                 lb.astype(np.float32).astype(np.float64))
    got_o, got_l = O_acc.cpu().numpy(), l_acc.cpu().numpy()
    np.testing.assert_array_equal(got_o[0], Oa[0].astype(np.float32))   # head 0 untouched
    np.testing.assert_allclose(got_o[1:], ref_o[1:], rtol=0, atol=2e-6)
    fin = np.isfinite(ref_l[1:])
    assert (np.isneginf(got_l[1:]) == ~fin).all()
    # lse reaches |16|, where one float32 ulp is 1.9e-6
    np.testing.assert_allclose(got_l[1:][fin], ref_l[1:][fin], rtol=2e-7, atol=2e-6)


@pytest.mark.parametrize("geo", GEOMS, ids=IDS)
@pytest.mark.parametrize("ranks,rank,hpc,tail", [(4, 0, 2, 1), (3, 2, 1, 1)])
def test_chunked_equals_unchunked(gpu, geo, ranks, rank, hpc, tail):
    g, mask, sel, out, Qd, (Qf, Kf, Vf), scale = _setup(geo, 8)
    bf16 = g.dtype == sp.BF16
    plan = sp.sparsp_chunk_plan(g, out["demand"], ranks, rank, hpc, tail)
    assert [c.astuple() for c in plan] == orc.chunk_plan(orc.demand_union(mask), ranks, rank,
                                                         hpc, tail)
    O, lse = sp.sparsp_chunked_attn(g, Qd, sel, out["slot_of"], out["K_packed"], out["V_packed"],
                                    plan, scale)
    O_ref, lse_ref = orc.sparse_attention(Qf, Kf, Vf, mask, g.L, g.block, g.i0, scale)
    O, lse = O.cpu().numpy(), lse.cpu().numpy()
    _check(O, O_ref, bf16, "chunked vs unchunked oracle")
    fin = np.isfinite(lse_ref)
    assert (np.isneginf(lse) == ~fin).all()
    assert np.abs(lse[fin] - lse_ref[fin]).max() <= (1e-4 if bf16 else 1e-5)
    # against the GPU's own unchunked call, in float32
    O1, lse1 = sp.sparsp_block_sparse_attn(g, Qd, sel, out["slot_of"], out["K_packed"],
                                           out["V_packed"], scale, out_dtype=sp.F32)
    assert np.abs(O - O1.cpu().numpy()).max() <= (2e-3 if bf16 else F32_TOL)


def test_chunked_full_size_wan_share(gpu):
    """The wan-share share (rank 0 of 4): chunked vs unchunked on the GPU, every row vs oracle."""
    import torch
    from workloads import get_workload, make_qkv
    wl = get_workload("wan-share")
    q, k, v = make_qkv(wl)
    g = P.geometry(wl.H, wl.L, wl.d, wl.block, wl.i0, wl.i1, wl.dtype)
    Qd, Kd, Vd = (P.to_device(x, wl.dtype) for x in (q, k, v))
    _, _, sc = sp.sparsp_block_scores(g, Qd, Kd)
    m, sel = sp.sparsp_topk_mask(g, sc, wl.keep, wl.global_blocks)
    out = sp.sparsp_demand_union_gather(g, m, Kd, Vd)
    plan = sp.sparsp_chunk_plan(g, out["demand"], wl.ranks, wl.rank, 8, 2)
    O, lse = sp.sparsp_chunked_attn(g, Qd, sel, out["slot_of"], out["K_packed"], out["V_packed"],
                                    plan, wl.softmax_scale)
    O1, lse1 = sp.sparsp_block_sparse_attn(g, Qd, sel, out["slot_of"], out["K_packed"],
                                           out["V_packed"], wl.softmax_scale, out_dtype=sp.F32)
    # Each shard's probabilities are rounded to bf16 against that shard's own
    # running max, so the two GPU results differ by bf16 rounding of P: held
    # to the bf16 parity bar. The log-sum-exp (total softmax mass) must agree
    # closely: a block lost or counted twice would move it.
    diff = (O - O1).abs()
    d_max, d_mean = diff.max().item(), diff.mean().item()
    d_l = (lse - lse1).abs().max().item()
    assert d_max <= P.BF16_MAX_ABS and d_mean <= P.BF16_MEAN_ABS and d_l <= 1e-4, (d_max, d_mean, d_l)
    # every row against the oracle, through the GPU's own mask
    mask = orc.words_to_mask(m.cpu().numpy().view(np.uint64), g.n)
    worst = P.check_every_row(q, k, v, mask, O.cpu().numpy(), lse.cpu().numpy(), wl, g.i0, g.nq,
                              True, "wan-share chunked", 1e-4)
    print(f"\n[chunked attention] {len(plan)} chunks, {wl.H * g.nq} rows, max-abs {worst:.3g}")
