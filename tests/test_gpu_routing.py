"""GPU parity of demand-directed routing (Section 5), producer side.

sparsp_pack_for_consumers against oracle.pack_by_consumer, bit for bit: the
cut provide bitsets, the (consumer, head) offsets, the block list and the
packed K and transposed V, for small geometries (fp32 and bf16, ragged last
block, the producer first, middle and last) and for the wan-share layer's
four ranks with demands computed on the GPU; and the consumer's own
derivation of its receive layout from its demand equals the producer's.
"""

import numpy as np
import pytest

import oracle as orc
import paper_2609_32197_amd as sp
from tests import _parity as P
from tests.test_gpu_kernels import _rand_inputs

pytestmark = pytest.mark.gpu

# (H, L, d, block, ranks, dtype)
CASES = [(3, 1000, 64, 64, 4, "f32"), (2, 4500, 64, 64, 3, "bf16"), (2, 9000, 128, 128, 5, "bf16")]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "H{}L{}d{}b{}R{}_{}".format(*c))
def test_pack_for_consumers_matches_oracle(gpu, case):
    import torch
    H, L, d, b, R, dt = case
    _, k, v = _rand_inputs(21, H, L, d, dt)
    n = -(-L // b)
    rng = np.random.default_rng(R)
    demands = [rng.random((H, n)) < 0.3 for _ in range(R)]
    words = np.stack([orc.mask_to_words(x) for x in demands]).view(np.int64)
    g = P.geometry(H, L, d, b, 0, 1, dt)
    Kd, Vd = P.to_device(k, dt), P.to_device(v, dt)
    kf, vf = (x.astype(np.float64) if dt == "f32" else x for x in (k, v))
    for p in sorted({0, R // 2, R - 1}):
        out = sp.sparsp_pack_for_consumers(g, torch.from_numpy(words).cuda(), R, p, Kd, Vd)
        provides = orc.provide_masks(demands, R, p)
        want = orc.pack_by_consumer(provides, k, v, L, b)
        prov = np.concatenate([m for _, m in provides])
        np.testing.assert_array_equal(out["provide"].cpu().numpy(), P.words_as_int64(prov))
        np.testing.assert_array_equal(out["head_off"].cpu().numpy(), want["head_off"])
        S = int(want["head_off"][-1])
        np.testing.assert_array_equal(out["gather_blk"][:S].cpu().numpy(), want["gather_blk"])
        np.testing.assert_array_equal(P.from_device_bits(out["K_packed"][:S], dt),
                                      want["K_packed"])
        np.testing.assert_array_equal(P.from_device_bits(out["V_packed"][:S], dt),
                                      want["V_packed"])


def test_wan_share_producers_and_consumer_view(gpu):
    import torch
    from workloads import get_workload, make_qkv
    wl = get_workload("wan-share")
    heads = list(range(6))
    q, k, v = make_qkv(wl, heads=heads)
    H, R = len(heads), wl.ranks
    Qd, Kd, Vd = (P.to_device(x, wl.dtype) for x in (q, k, v))
    n = -(-wl.L // wl.block)
    dems = []
    for c in range(R):
        lo, hi = orc.local_range(n, R, c)
        g = P.geometry(H, wl.L, wl.d, wl.block, lo, hi, wl.dtype)
        _, _, sc = sp.sparsp_block_scores(g, Qd, Kd)
        m, _ = sp.sparsp_topk_mask(g, sc, wl.keep)
        dems.append(sp.sparsp_demand_union_gather(g, m, Kd, Vd)["demand"].clone())
    D = torch.stack(dems)
    dem_np = [orc.words_to_mask(x.cpu().numpy().view(np.uint64), n) for x in dems]
    g = P.geometry(H, wl.L, wl.d, wl.block, 0, 1, wl.dtype)
    for p in range(R):
        out = sp.sparsp_pack_for_consumers(g, D, R, p, Kd, Vd)
        provides = orc.provide_masks(dem_np, R, p)
        lo, hi = orc.local_range(n, R, p)
        head_off = out["head_off"].cpu().numpy()
        for idx, (c, m) in enumerate(provides):
            c_off, c_blk, _ = orc.packing_plan(m)   # what consumer c derives from its mask
            s0, s1 = head_off[idx * H], head_off[(idx + 1) * H]
            np.testing.assert_array_equal(head_off[idx * H:(idx + 1) * H + 1] - s0, c_off)
            np.testing.assert_array_equal(out["gather_blk"][s0:s1].cpu().numpy(), c_blk)
        # sampled packed blocks against the source rows
        kb = P.from_device_bits(out["K_packed"][:int(head_off[-1])], wl.dtype)
        blk = out["gather_blk"].cpu().numpy()
        rng = np.random.default_rng(p)
        for slot in rng.choice(int(head_off[-1]), 8, replace=False):
            v_head = int(np.searchsorted(head_off, slot, side="right") - 1)
            h, j = v_head % H, int(blk[slot])
            c = min(wl.block, wl.L - j * wl.block)
            np.testing.assert_array_equal(kb[slot, :c], k[h, j * wl.block:j * wl.block + c])
        vol = sp.sparsp_route_volume(g, D, R, p)
        assert vol["direct"] == int(head_off[-1])
        assert vol["direct"] <= vol["relay"] <= vol["dense"]
