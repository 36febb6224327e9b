"""GPU parity of dependency-aware placement (Section 4.3, Eq. 4) against the oracle.

* sparsp_permute_blocks moves token blocks exactly as oracle.permute_blocks
  (bit for bit, forward and inverse, ragged last block included);
* a rank's pipeline over placed tensors: the mask from the oracle's float32
  scores (rearranged to placed order) is bit-exact, and the demand it yields,
  mapped back to logical blocks, equals Eq. 2's union over the rank's query
  blocks; sparsp_remote_demand equals Eq. 3's block count;
* on the full wan-share layer: the placement round trip is exact.
"""

import numpy as np
import pytest

import oracle as orc
import paper_2609_32197_amd as sp
from tests import _parity as P
from tests.test_gpu_kernels import _rand_inputs

pytestmark = pytest.mark.gpu

# (H, T frames, frame tokens, extra tokens, d, block, ranks, dtype)
CASES = [
    (2, 4, 192, 0, 64, 64, 3, "f32"),     # 3 blocks per frame, 1 per rank
    (3, 5, 320, 40, 64, 64, 2, "bf16"),   # blocks straddle frames, ragged tail
    (2, 3, 1000, 0, 128, 128, 4, "bf16"),
]


def _ids(c):
    return "H{}T{}F{}+{}d{}b{}R{}_{}".format(*c)


@pytest.mark.parametrize("case", CASES, ids=_ids)
def test_permute_matches_oracle(gpu, case):
    H, T, F, extra, d, b, R, dt = case
    L = T * F + extra
    x, _, _ = _rand_inputs(7, H, L, d, dt)
    g = P.geometry(H, L, d, b, 0, 1, dt)
    perm, _ = sp.sparsp_periodic_placement(L, b, F, R)
    import torch
    pd = torch.from_numpy(perm).cuda()
    X = P.to_device(x, dt)
    Y = sp.sparsp_permute_blocks(g, pd, X)
    want = orc.permute_blocks(x, perm.astype(np.int64), L, b)
    np.testing.assert_array_equal(P.from_device_bits(Y, dt), want)
    back = sp.sparsp_permute_blocks(g, pd, Y, inverse=True)
    np.testing.assert_array_equal(P.from_device_bits(back, dt), x)


@pytest.mark.parametrize("case", CASES, ids=_ids)
def test_placed_rank_pipeline_matches_eq2_eq3(gpu, case):
    import torch
    H, T, F, extra, d, b, R, dt = case
    L = T * F + extra
    q, k, v = _rand_inputs(11, H, L, d, dt)
    n = -(-L // b)
    keep = max(1, n // 3)
    owner = orc.periodic_owner(L, b, F, R)
    # oracle: scores of every query block in logical order, the full mask, Eq. 2 per rank
    _, _, s_log = P.oracle_pooled_scores(q, k, dt, L, b, 0, n, d)
    mask_all, _ = orc.select_topk(s_log, keep, 0)
    perm, begin = sp.sparsp_periodic_placement(L, b, F, R)
    pd = torch.from_numpy(perm).cuda()
    gl = P.geometry(H, L, d, b, 0, 1, dt)
    Kp = sp.sparsp_permute_blocks(gl, pd, P.to_device(k, dt))
    Vp = sp.sparsp_permute_blocks(gl, pd, P.to_device(v, dt))
    for r in range(R):
        i0, i1 = int(begin[r]), int(begin[r + 1])
        g = P.geometry(H, L, d, b, i0, i1, dt)
        rows = perm[i0:i1].astype(np.int64)
        s_pl = s_log[:, rows][:, :, perm.astype(np.int64)]  # placed rows and columns
        m, sel = sp.sparsp_topk_mask(g, P.to_device(np.ascontiguousarray(s_pl), "f32"), keep)
        om, _ = orc.select_topk(np.ascontiguousarray(s_pl), keep, i0)
        np.testing.assert_array_equal(P.words_as_int64(om), m.cpu().numpy())
        out = sp.sparsp_demand_union_gather(g, m, Kp, Vp)
        dem_pl = orc.words_to_mask(out["demand"].cpu().numpy().view(np.uint64), n)
        dem_log = np.zeros_like(dem_pl)
        dem_log[:, perm] = dem_pl
        want = orc.rank_demand(mask_all, owner, r)
        np.testing.assert_array_equal(dem_log, want)
        remote, total = sp.sparsp_remote_demand(g, out["demand"])
        assert remote == orc.remote_blocks(want, owner, r)
        assert total == int(want.sum())


def test_wan_share_placement_round_trip(gpu):
    import torch
    from workloads import get_workload, make_qkv
    wl = get_workload("wan-share")
    q, _, _ = make_qkv(wl, heads=range(8))
    T, Hy, W = wl.latent
    g = P.geometry(8, wl.L, wl.d, wl.block, 0, 1, wl.dtype)
    perm, begin = sp.sparsp_periodic_placement(wl.L, wl.block, Hy * W, wl.ranks)
    pd = torch.from_numpy(perm).cuda()
    X = P.to_device(q, wl.dtype)
    Y = sp.sparsp_permute_blocks(g, pd, X)
    assert torch.equal(sp.sparsp_permute_blocks(g, pd, Y, inverse=True), X)
    ybits = P.from_device_bits(Y, wl.dtype)
    b = wl.block
    for kk in (0, int(begin[1]), int(begin[2]) + 5, g.n - 1):
        j = int(perm[kk])
        c = min(b, wl.L - j * b)
        np.testing.assert_array_equal(ybits[:, kk * b:kk * b + c], q[:, j * b:j * b + c])
