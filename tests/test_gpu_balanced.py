"""Attention with the last round of workgroups balanced
(sparsp_block_sparse_attn_balanced, or the binding's workspace= argument).

The launch runs R = H*nq rows on the P workgroups the device keeps resident;
the S = R mod P rows of the last round are split into k = min(4, P // S)
pieces, merged through the log-sum-exp. So:

* every row outside the last round equals sparsp_block_sparse_attn's bit for
  bit, and the split rows meet the usual bar against the oracle (and differ
  from the unsplit kernel by float32 rounding only);
* without a workspace, or with one too small for two pieces, the call is
  sparsp_block_sparse_attn bit for bit.

The workspace holds the row order first (4 bytes per row, padded to 256),
then one block x (d+1) float32 partial per resident workgroup, so P is read
back from sparsp_attn_workspace_bytes. The rows of the last round are
recomputed from the documented launch order: positions are dealt to the XCDs
in contiguous ranges, and within each head position k holds the row with the
k-th smallest first kept block (ties by row index). Rows the test takes as
whole must then equal the plain call bit for bit, which also checks that
order.
"""

import numpy as np
import pytest

import oracle as orc
import paper_2609_32197_amd as sp
from tests import _parity as P
from tests.test_gpu_kernels import _pipeline, _rand_inputs, ctypes_scale

pytestmark = pytest.mark.gpu


def xcd_row(w, G):
    """Row of workgroup index w: XCD w % 8 takes the (w % 8)-th contiguous range."""
    x, idx, per, rem = w & 7, w >> 3, G >> 3, G & 7
    return x * per + min(x, rem) + idx


def row_sort_bytes(rows):
    return (rows * 4 + 255) // 256 * 256


def sorted_rows(sel, n):
    """Launch position -> row: within each head, rows by first kept block, then index."""
    sel = np.asarray(sel)
    H, nq = sel.shape[:2]
    first = sel[:, :, 0].astype(np.int64)
    first = np.where((first < 0) | (first >= n), n, first)
    return np.concatenate([h * nq + np.lexsort((np.arange(nq), first[h])) for h in range(H)])


def tail_rows(g, keep, sel):
    """Rows (h * nq + r) of the last round that the balanced call splits, and k."""
    nbytes = sp.sparsp_attn_workspace_bytes(g, keep)
    G = g.H * g.nq
    slots = (nbytes - row_sort_bytes(G)) // (g.block * (g.d + 1) * 4)
    S = G % slots if slots else 0
    if S == 0 or slots // S < 2:
        return set(), 1, nbytes
    k = min(4, slots // S)
    row_at = sorted_rows(sel.cpu().numpy() if hasattr(sel, "cpu") else sel, g.n)
    return {int(row_at[xcd_row(G - S + t, G)]) for t in range(S)}, k, nbytes


GEOMS = [
    (3, 9000, 128, 128, 20, 71, "bf16"),   # 128-token kernel, ragged last block
    (2, 4400, 64, 128, 3, 35, "bf16"),     # 128-token kernel, d = 64
    (2, 4500, 64, 64, 30, 71, "bf16"),     # 64-token kernel
    (2, 4100, 128, 64, 0, 40, "bf16"),     # 64-token kernel, d = 128
    (8, 35900, 128, 128, 0, 280, "bf16"),  # more rows than resident workgroups (2,240)
    (12, 16000, 64, 64, 0, 180, "bf16"),   # the same for the 64-token kernel (2,160)
]


@pytest.mark.parametrize("geo", GEOMS, ids=lambda g: "H{}L{}d{}b{}_{}-{}_{}".format(*g))
@pytest.mark.parametrize("keep_frac", [0.05, 0.4])
def test_balanced_attention(gpu, geo, keep_frac):
    torch = P.torch()
    H, L, d, b, i0, i1, dt = geo
    n = -(-L // b)
    q, k, v = _rand_inputs(5, H, L, d, dt)
    g = P.geometry(H, L, d, b, i0, i1, dt)
    keep = max(1, int(round(keep_frac * n)))
    om, osel, sel, out = _pipeline(q, k, v, g, dt, keep)
    split, kk, nbytes = tail_rows(g, keep, sel)
    assert nbytes > 0
    ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    Qd = P.to_device(q, dt)
    args = (g, Qd, sel, out["slot_of"], out["K_packed"], out["V_packed"], ctypes_scale(d))
    nq = i1 - i0
    rows = H * nq
    if len(split) == 0:
        pytest.skip(f"{rows} rows fill every round on this device: nothing to split")
    whole = np.array([r not in split for r in range(rows)])
    for odt in (sp.F32, sp.BF16):
        O0, l0 = sp.sparsp_block_sparse_attn(*args, out_dtype=odt)
        O1, l1 = sp.sparsp_block_sparse_attn(*args, out_dtype=odt, workspace=ws)
        bits = torch.int16 if odt == sp.BF16 else torch.int32
        a0 = O0.view(bits).reshape(H, nq, b, d).reshape(rows, b, d).cpu().numpy()
        a1 = O1.view(bits).reshape(H, nq, b, d).reshape(rows, b, d).cpu().numpy()
        np.testing.assert_array_equal(a1[whole], a0[whole])
        m0 = l0.view(torch.int32).reshape(rows, b).cpu().numpy()
        m1 = l1.view(torch.int32).reshape(rows, b).cpu().numpy()
        np.testing.assert_array_equal(m1[whole], m0[whole])
        # the split rows against the oracle (all of them when there are few)
        Qf, Kf, Vf = (orc.decode_input(x, dt) for x in (q, k, v))
        On = O1.float().cpu().numpy()
        ln = l1.cpu().numpy()
        for row in sorted(split)[:24]:
            h, r = divmod(row, nq)
            o_ref, lse_ref = orc.attend_block(Qf[h], Kf[h], Vf[h], om[h, r], i0 + r, L, b,
                                              ctypes_scale(d))
            P.check_attention(On[h, r * b:(r + 1) * b], o_ref, True,
                              f"balanced {geo} keep={keep} k={kk} row={row}")
            fin = np.isfinite(lse_ref)
            got = ln[h, r * b:(r + 1) * b]
            assert (np.isneginf(got) == ~fin).all()
            assert np.abs(got[fin] - lse_ref[fin]).max() <= 1e-4


@pytest.mark.parametrize("geo", GEOMS[:3], ids=lambda g: "H{}L{}d{}b{}_{}-{}_{}".format(*g))
def test_without_room_the_call_is_unchanged(gpu, geo):
    torch = P.torch()
    H, L, d, b, i0, i1, dt = geo
    q, k, v = _rand_inputs(6, H, L, d, dt)
    g = P.geometry(H, L, d, b, i0, i1, dt)
    keep = 5
    _, _, sel, out = _pipeline(q, k, v, g, dt, keep)
    args = (g, P.to_device(q, dt), sel, out["slot_of"], out["K_packed"], out["V_packed"],
            ctypes_scale(d))
    O0, l0 = sp.sparsp_block_sparse_attn(*args)
    for nbytes in (16, b * (d + 1) * 4):   # too small for two pieces of even one row
        ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        O1, l1 = sp.sparsp_block_sparse_attn(*args, workspace=ws)
        assert torch.equal(O0.view(torch.int16), O1.view(torch.int16))
        assert torch.equal(l0.view(torch.int32), l1.view(torch.int32))


@pytest.mark.parametrize("name", ["wan-share", "hunyuan-share"])
def test_balanced_full_size(gpu, name):
    """The benchmark workloads: rows outside the last round bit-identical, the
    split rows against the oracle (a sample) and against the unsplit kernel."""
    torch = P.torch()
    from workloads import get_workload, make_qkv
    wl = get_workload(name)
    q, k, v = make_qkv(wl)
    g = P.geometry(wl.H, wl.L, wl.d, wl.block, wl.i0, wl.i1, wl.dtype)
    Qd, Kd, Vd = (P.to_device(x, wl.dtype) for x in (q, k, v))
    _, _, sc = sp.sparsp_block_scores(g, Qd, Kd)
    m, sel = sp.sparsp_topk_mask(g, sc, wl.keep, wl.global_blocks)
    out = sp.sparsp_demand_union_gather(g, m, Kd, Vd)
    args = (g, Qd, sel, out["slot_of"], out["K_packed"], out["V_packed"], wl.softmax_scale)
    split, kk, nbytes = tail_rows(g, wl.keep, sel)
    ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device="cuda")
    O0, l0 = sp.sparsp_block_sparse_attn(*args)
    O1, l1 = sp.sparsp_block_sparse_attn(*args, workspace=ws)
    rows, b = wl.H * wl.nq, wl.block
    whole = np.array([r not in split for r in range(rows)])
    a0 = O0.view(torch.int16).reshape(rows, b, wl.d).cpu().numpy()
    a1 = O1.view(torch.int16).reshape(rows, b, wl.d).cpu().numpy()
    np.testing.assert_array_equal(a1[whole], a0[whole])
    if not split:
        return
    d01 = (O1.float() - O0.float()).abs()
    assert float(d01.max()) <= 2e-2 and float(d01.mean()) <= 1e-3
    mask = orc.words_to_mask(m.cpu().numpy().view(np.uint64), g.n)
    On = O1.float().cpu().numpy()
    rng = np.random.default_rng(3)
    for row in rng.choice(sorted(split), size=min(6, len(split)), replace=False):
        h, r = divmod(int(row), wl.nq)
        qf, kf, vf = (orc.decode_input(x[h], wl.dtype) for x in (q, k, v))
        o_ref, _ = orc.attend_block(qf, kf, vf, mask[h, r], wl.i0 + r, wl.L, b, wl.softmax_scale)
        P.check_attention(On[h, r * b:(r + 1) * b], o_ref, True,
                          f"balanced {name} row={row} (k={kk}, {len(split)} split rows)")
