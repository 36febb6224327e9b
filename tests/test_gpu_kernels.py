"""GPU parity on small geometries: every ABI call against the float64 oracle.

Sizes span several tiles and ragged tails: partial last blocks, block counts
that are not multiples of 64 (several mask words), local slices that start
past block 0 or end at the padded last block, global blocks, ties.
Masks, selections, demand, offsets, slot maps and packed buffers must match
bit for bit when both sides get the same float32 scores; scores and
attention within the tolerances stated in tests/_parity.py.
"""

import math

import numpy as np
import pytest

import oracle as orc
import paper_2609_32197_amd as sp
from tests import _parity as P

pytestmark = pytest.mark.gpu


def _rand_inputs(seed, H, L, d, dtype):
    rng = np.random.default_rng(seed)
    x = [rng.standard_normal((H, L, d)).astype(np.float32) for _ in range(3)]
    if dtype == "bf16":
        from workloads import bf16_round_bits
        x = [bf16_round_bits(a) for a in x]
    return x


# (H, L, d, block, i0, i1, dtype)
GEOMS = [
    (2, 1024, 64, 64, 0, 16, "f32"),
    (3, 1000, 64, 64, 5, 16, "f32"),          # ragged, slice ends at the padded block
    (2, 1500, 128, 128, 0, 12, "bf16"),      # ragged last block (92 tokens)
    (3, 9000, 128, 128, 20, 71, "bf16"),     # n = 71: two mask words
    (2, 4500, 64, 64, 30, 71, "bf16"),       # d = block = 64
    (2, 4400, 128, 64, 0, 69, "bf16"),       # d = 128, block = 64
    (2, 4400, 64, 128, 3, 35, "bf16"),       # d = 64, block = 128
]


@pytest.mark.parametrize("geo", GEOMS, ids=lambda g: "H{}L{}d{}b{}_{}-{}_{}".format(*g))
def test_block_scores_within_bound(gpu, geo):
    H, L, d, b, i0, i1, dt = geo
    q, k, _ = _rand_inputs(1, H, L, d, dt)
    g = P.geometry(H, L, d, b, i0, i1, dt)
    pq, pk, sc = sp.sparsp_block_scores(g, P.to_device(q, dt), P.to_device(k, dt))
    opq, opk, osc, aq, ak = P.oracle_pooled_scores(q, k, dt, L, b, i0, i1, d, with_abs=True)
    # Pooled means: each within its own bound.
    u = 2.0 ** -24
    groups = 256 // (d // (8 if dt == "bf16" else 4))
    e_p = -(-b // groups) + groups + 1
    assert (np.abs(pq.cpu().numpy() - opq) <= 2 * e_p * u * aq + 1e-30).all()
    assert (np.abs(pk.cpu().numpy() - opk) <= 2 * e_p * u * ak + 1e-30).all()
    err = np.abs(sc.cpu().numpy().astype(np.float64) - osc.astype(np.float64))
    tol = P.score_tolerance(opq, opk, aq, ak, osc, d, b, dt)
    assert (err <= tol).all(), f"max excess {(err - tol).max():.3g}"


def _topk_case(seed, H, n, nq, i0, keep, G, coarse):
    rng = np.random.default_rng(seed)
    if coarse:  # many exact ties, and signed zeros
        s = (rng.integers(-2, 3, size=(H, nq, n)) * 0.25).astype(np.float32)
        s[rng.random(s.shape) < 0.1] = -0.0
    else:
        s = rng.standard_normal((H, nq, n)).astype(np.float32)
    return s


TOPK = [
    # (H, n, nq, i0, keep, G, coarse)
    (2, 16, 16, 0, 5, (), False),
    (3, 71, 30, 41, 9, (), True),
    (2, 129, 7, 100, 20, (3, 128, 64), True),
    (2, 200, 50, 10, 200, (), False),      # keep = n
    (2, 200, 50, 10, 1, (), False),        # diagonal only
    (2, 150, 20, 0, 4, (5, 6, 7), False),  # keep = |F| on rows 0..19
    (1, 1000, 12, 988, 100, (), True),
    (2, 4096, 3, 4000, 410, (0, 4095), False),  # the largest n
    (1, 1, 1, 0, 1, (), False),
]


@pytest.mark.parametrize("case", TOPK, ids=lambda c: "n{}_nq{}_i0{}_k{}".format(c[1], c[2], c[3], c[4]))
def test_topk_mask_bit_exact(gpu, case):
    H, n, nq, i0, keep, G, coarse = case
    s = _topk_case(7, H, n, nq, i0, keep, G, coarse)
    # Any L with n blocks works for the mask: block 1, L = n.
    g = sp.Geometry(H, n, 8, 1, i0, i0 + nq, sp.BF16)
    m, sel = sp.sparsp_topk_mask(g, P.to_device(s, "f32"), keep, G)
    om, osel = orc.select_topk(s, keep, i0, G)
    np.testing.assert_array_equal(m.cpu().numpy(), P.words_as_int64(om))
    np.testing.assert_array_equal(sel.cpu().numpy(), osel)


# Shapes the streaming gather does not take (a block's rows or columns do not
# split into groups of eight 16-byte chunks): the windowed gather kernel.
GATHER_ONLY_GEOMS = [
    (2, 700, 20, 12, 3, 20, "f32"),    # d / 4 = 5, block / 4 = 3, ragged last block
    (3, 900, 64, 32, 2, 25, "bf16"),   # block / 8 = 4 sub-blocks per row
    (2, 1000, 128, 16, 0, 63, "bf16"),  # block / 8 = 2, ragged
]


@pytest.mark.parametrize("geo", GEOMS + GATHER_ONLY_GEOMS,
                         ids=lambda g: "H{}L{}d{}b{}_{}-{}_{}".format(*g))
def test_demand_gather_bit_exact(gpu, geo):
    H, L, d, b, i0, i1, dt = geo
    n = -(-L // b)
    nq = i1 - i0
    _, k, v = _rand_inputs(2, H, L, d, dt)
    s = _topk_case(3, H, n, nq, i0, 0, (), False)
    keep = max(2, n // 5)
    om, osel = orc.select_topk(s, keep, i0, ())
    g = P.geometry(H, L, d, b, i0, i1, dt)
    mask = P.torch().from_numpy(P.words_as_int64(om)).cuda()
    out = sp.sparsp_demand_union_gather(g, mask, P.to_device(k, dt), P.to_device(v, dt))
    D = orc.demand_union(om)
    head_off, gather_blk, slot_of = orc.packing_plan(D)
    np.testing.assert_array_equal(out["demand"].cpu().numpy(), P.words_as_int64(D))
    np.testing.assert_array_equal(out["head_off"].cpu().numpy(), head_off)
    np.testing.assert_array_equal(out["slot_of"].cpu().numpy(), slot_of)
    S = int(head_off[-1])
    np.testing.assert_array_equal(out["gather_blk"].cpu().numpy()[:S], gather_blk)
    Kp, Vp = orc.pack_kv(k, v, head_off, gather_blk, L, b)
    np.testing.assert_array_equal(P.from_device_bits(out["K_packed"], dt)[:S], Kp)
    np.testing.assert_array_equal(P.from_device_bits(out["V_packed"], dt)[:S], Vp)


def _pipeline(q, k, v, g, dt, keep, G=()):
    """Oracle scores -> oracle mask, and the same scores -> GPU topk and gather.

    Returns the oracle mask and selection, the GPU selection and the packed buffers.
    """
    L, b, d = g.L, g.block, g.d
    _, _, scores = P.oracle_pooled_scores(q, k, dt, L, b, g.i0, g.i1, d)
    om, osel = orc.select_topk(scores, keep, g.i0, G)
    m, sel = sp.sparsp_topk_mask(g, P.to_device(scores, "f32"), keep, G)
    out = sp.sparsp_demand_union_gather(g, m, P.to_device(k, dt), P.to_device(v, dt))
    return om, osel, sel, out


# The float32 kernel runs P = 4, 2 or 1 lanes per query row for blocks of up
# to 64, 128 and 256 tokens; these cover each P with ragged blocks and odd d.
F32_ATTN_GEOMS = [
    (2, 1000, 20, 48, 1, 12, "f32"),     # P = 4, d = 20, ragged last block
    (2, 1200, 96, 96, 0, 13, "f32"),     # P = 2, ragged (48 tokens)
    (2, 1500, 128, 128, 2, 12, "f32"),   # P = 2, d = 128
    (2, 1700, 64, 200, 0, 9, "f32"),     # P = 1, ragged (100 tokens)
    (1, 2000, 128, 256, 0, 8, "f32"),    # P = 1, the largest block
]


@pytest.mark.parametrize("geo", GEOMS + F32_ATTN_GEOMS,
                         ids=lambda g: "H{}L{}d{}b{}_{}-{}_{}".format(*g))
@pytest.mark.parametrize("keep_frac", [0.3, 1.0])
def test_attention_parity(gpu, geo, keep_frac):
    H, L, d, b, i0, i1, dt = geo
    n = -(-L // b)
    q, k, v = _rand_inputs(4, H, L, d, dt)
    g = P.geometry(H, L, d, b, i0, i1, dt)
    keep = max(1, int(round(keep_frac * n)))
    om, osel, sel, out = _pipeline(q, k, v, g, dt, keep)
    np.testing.assert_array_equal(sel.cpu().numpy(), osel)
    scale = ctypes_scale(d)
    Qd = P.to_device(q, dt)
    outs = [sp.sparsp_block_sparse_attn(g, Qd, sel, out["slot_of"], out["K_packed"],
                                        out["V_packed"], scale, out_dtype=sp.F32)]
    if dt == "bf16":
        outs.append(sp.sparsp_block_sparse_attn(g, Qd, sel, out["slot_of"], out["K_packed"],
                                                out["V_packed"], scale, out_dtype=sp.BF16))
    Qf, Kf, Vf = (orc.decode_input(x, dt) for x in (q, k, v))
    O_ref, lse_ref = orc.sparse_attention(Qf, Kf, Vf, om, L, b, i0, scale)
    for O, lse in outs:
        On = O.float().cpu().numpy()
        P.check_attention(On, O_ref, dt == "bf16", f"{geo} keep={keep} {O.dtype}")
        ln = lse.cpu().numpy()
        fin = np.isfinite(lse_ref)
        assert (np.isneginf(ln) == ~fin).all()
        # Scores come from exact bf16 products with float32 sums: lse is tight too.
        assert np.abs(ln[fin] - lse_ref[fin]).max() <= (1e-4 if dt == "bf16" else 1e-5)


def ctypes_scale(d):
    return float(np.float32(1.0 / math.sqrt(d)))


def test_attention_diagonal_only_equals_local_block_attention(gpu):
    torch = P.torch()
    H, L, d, b = 2, 1000, 128, 128
    q, k, v = _rand_inputs(5, H, L, d, "bf16")
    g = P.geometry(H, L, d, b, 0, 8, "bf16")
    om, _, sel, out = _pipeline(q, k, v, g, "bf16", 1)
    assert (sel.cpu().numpy()[..., 0] == np.arange(8)).all()
    O, _ = sp.sparsp_block_sparse_attn(g, P.to_device(q, "bf16"), sel, out["slot_of"],
                                       out["K_packed"], out["V_packed"], ctypes_scale(d),
                                       out_dtype=sp.F32)
    Qf, Kf, Vf = (torch.from_numpy(orc.decode_input(x, "bf16")) for x in (q, k, v))
    for i in range(8):
        lo, hi = i * b, min((i + 1) * b, L)
        ref = torch.nn.functional.scaled_dot_product_attention(
            Qf[:, lo:hi], Kf[:, lo:hi], Vf[:, lo:hi], scale=ctypes_scale(d)).numpy()
        got = O.cpu().numpy()[:, i * b:i * b + hi - lo]
        assert np.abs(got - ref).max() <= P.BF16_MAX_ABS


def test_outputs_are_deterministic(gpu):
    H, L, d, b, i0, i1, dt = GEOMS[3]
    q, k, v = _rand_inputs(6, H, L, d, dt)
    g = P.geometry(H, L, d, b, i0, i1, dt)
    runs = []
    for _ in range(2):
        Qd, Kd, Vd = (P.to_device(x, dt) for x in (q, k, v))
        pq, pk, sc = sp.sparsp_block_scores(g, Qd, Kd)
        m, sel = sp.sparsp_topk_mask(g, sc, 9)
        out = sp.sparsp_demand_union_gather(g, m, Kd, Vd)
        O, lse = sp.sparsp_block_sparse_attn(g, Qd, sel, out["slot_of"], out["K_packed"],
                                             out["V_packed"], out_dtype=sp.BF16)
        outs = (pq, pk, sc, m, sel, out["demand"], out["slot_of"], O.view(P.torch().int16), lse)
        runs.append([x.cpu().numpy().tobytes() for x in outs])
    assert runs[0] == runs[1]


def test_errors_surface_through_the_binding(gpu):
    torch = P.torch()
    g = sp.Geometry(2, 1024, 128, 128, 0, 8, sp.BF16)
    m = torch.zeros((2, 8, 1), dtype=torch.int64, device="cuda")
    K = torch.zeros((2, 1024, 128), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(sp.SparspError) as ei:
        sp.sparsp_demand_union_gather(g, m, K, K, capacity_blocks=15)
    assert ei.value.code == -4
    sc = torch.zeros((2, 8, 8), dtype=torch.float32, device="cuda")
    with pytest.raises(sp.SparspError) as ei:
        sp.sparsp_topk_mask(g, sc, 9)
    assert ei.value.code == -1


def test_mfma_probe_runs(gpu):
    """The benchmark's measurement probe: every thread writes a finite sum."""
    from paper_2609_32197_amd import probe
    torch = P.torch()
    sink = torch.full((8 * 256,), float("nan"), dtype=torch.float32, device="cuda")
    probe.run(50, 8, sink)
    torch.cuda.synchronize()
    out = sink.cpu()
    assert torch.isfinite(out).all() and (out != 0).any()
    with pytest.raises(ValueError):
        probe.run(50, 9, sink)
