"""GPU parity at the full sizes of the benchmark workloads, in the launch
configuration the benchmark times.

For every workload (tiny float32 case; Wan-style rank share; HunyuanVideo-style
rank share, whole layer and its dense twin; the text-token density sweep):

* block scores within the derived bound of tests/_parity.py, every entry;
* masks and selections bit-exact when the GPU gets the oracle's float32 scores;
* demand, offsets, slot maps, gather indices and both packed buffers
  bit-exact, every entry;
* attention within 2e-2 max-abs / 1e-3 mean-abs (bf16) or 1e-5 (float32) on
  sampled query blocks: every head x 16 blocks, always including the first,
  the last and the padded last block of the slice (all blocks for the tiny
  case);
* end to end (GPU scores -> GPU mask), the share of rows whose mask equals the
  oracle's is reported and must stay above 98%: rows can differ only where two
  candidates' float32 scores are within the score error bound of each other.
"""

import functools

import numpy as np
import pytest

import oracle as orc
import paper_2609_32197_amd as sp
from tests import _parity as P
from workloads import get_workload, make_qkv

pytestmark = pytest.mark.gpu

NAMES = ["tiny-f32", "wan-share", "hunyuan-share", "hunyuan-layer", "hunyuan-layer-dense",
         "text-sweep-5", "text-sweep-10", "text-sweep-25", "text-sweep-50", "text-sweep-100"]


@functools.lru_cache(maxsize=1)
def _inputs(config_id, ranks, rank):
    """Raw inputs and oracle pooled scores, shared by workloads with the same data."""
    wl = next(get_workload(n) for n in NAMES
              if get_workload(n).config_id == config_id and get_workload(n).ranks == ranks
              and get_workload(n).rank == rank)
    q, k, v = make_qkv(wl, seed=0)
    pq, pk, sc, aq, ak = P.oracle_pooled_scores(q, k, wl.dtype, wl.L, wl.block, wl.i0, wl.i1,
                                                 wl.d, with_abs=True)
    return q, k, v, pq, pk, sc, aq, ak


class Case:
    def __init__(self, name):
        wl = get_workload(name)
        self.wl = wl
        (self.q, self.k, self.v, self.pq, self.pk, self.scores, self.aq,
         self.ak) = _inputs(wl.config_id, wl.ranks, wl.rank)
        self.g = P.geometry(wl.H, wl.L, wl.d, wl.block, wl.i0, wl.i1, wl.dtype)
        self.Qd, self.Kd, self.Vd = (P.to_device(x, wl.dtype) for x in (self.q, self.k, self.v))
        self.mask, self.sel = orc.select_topk(self.scores, wl.keep, wl.i0, wl.global_blocks)


@pytest.fixture(scope="module", params=NAMES)
def case(request, gpu):
    c = Case(request.param)
    yield c
    del c
    P.torch().cuda.empty_cache()


def test_block_scores(case):
    wl = case.wl
    pq, pk, sc = sp.sparsp_block_scores(case.g, case.Qd, case.Kd)
    err = np.abs(sc.cpu().numpy().astype(np.float64) - case.scores.astype(np.float64))
    tol = P.score_tolerance(case.pq, case.pk, case.aq, case.ak, case.scores, wl.d, wl.block,
                            wl.dtype)
    assert (err <= tol).all(), f"{wl.name}: max excess {(err - tol).max():.3g}"


def test_mask_bit_exact_from_oracle_scores(case):
    wl = case.wl
    m, sel = sp.sparsp_topk_mask(case.g, P.to_device(case.scores, "f32"), wl.keep,
                                 wl.global_blocks)
    np.testing.assert_array_equal(m.cpu().numpy(), P.words_as_int64(case.mask))
    np.testing.assert_array_equal(sel.cpu().numpy(), case.sel)


def test_demand_and_gather_bit_exact(case):
    wl = case.wl
    mask = P.torch().from_numpy(P.words_as_int64(case.mask)).cuda()
    out = sp.sparsp_demand_union_gather(case.g, mask, case.Kd, case.Vd)
    D = orc.demand_union(case.mask)
    head_off, gather_blk, slot_of = orc.packing_plan(D)
    np.testing.assert_array_equal(out["demand"].cpu().numpy(), P.words_as_int64(D))
    np.testing.assert_array_equal(out["head_off"].cpu().numpy(), head_off)
    np.testing.assert_array_equal(out["slot_of"].cpu().numpy(), slot_of)
    S = int(head_off[-1])
    np.testing.assert_array_equal(out["gather_blk"].cpu().numpy()[:S], gather_blk)
    Kp, Vp = orc.pack_kv(case.k, case.v, head_off, gather_blk, wl.L, wl.block)
    np.testing.assert_array_equal(P.from_device_bits(out["K_packed"][:S], wl.dtype), Kp)
    del Kp
    np.testing.assert_array_equal(P.from_device_bits(out["V_packed"][:S], wl.dtype), Vp)


def _sample_pairs(wl, per_head=16, seed=0):
    if wl.H * wl.nq <= 64:
        return [(h, r) for h in range(wl.H) for r in range(wl.nq)]
    rng = np.random.default_rng(seed)
    pairs = []
    for h in range(wl.H):
        rows = {0, wl.nq - 1}
        if wl.i1 == wl.n:  # the padded last block is local
            rows.add(wl.nq - 1)
        rows |= set(rng.choice(wl.nq, size=min(wl.nq, per_head), replace=False).tolist())
        pairs += [(h, int(r)) for r in sorted(rows)[:per_head + 2]]
    return pairs


def test_attention_sampled(case):
    wl = case.wl
    m, sel = sp.sparsp_topk_mask(case.g, P.to_device(case.scores, "f32"), wl.keep,
                                 wl.global_blocks)
    out = sp.sparsp_demand_union_gather(case.g, m, case.Kd, case.Vd)
    out_dtype = sp.BF16 if wl.dtype == "bf16" else sp.F32
    O, lse = sp.sparsp_block_sparse_attn(case.g, case.Qd, sel, out["slot_of"], out["K_packed"],
                                         out["V_packed"], wl.softmax_scale, out_dtype=out_dtype)
    O = O.float().cpu().numpy()
    lse = lse.cpu().numpy()
    b = wl.block
    worst = worst_lse = 0.0
    abs_sum = count = 0.0
    pairs = _sample_pairs(wl)
    for h, r in pairs:
        qf = orc.decode_input(case.q[h], wl.dtype)
        kf = orc.decode_input(case.k[h], wl.dtype)
        vf = orc.decode_input(case.v[h], wl.dtype)
        o_ref, l_ref = orc.attend_block(qf, kf, vf, case.mask[h, r], wl.i0 + r, wl.L, b,
                                        wl.softmax_scale)
        got = O[h, r * b:(r + 1) * b]
        mx, mean = P.check_attention(got, o_ref, wl.dtype == "bf16", f"{wl.name} h={h} r={r}")
        worst = max(worst, mx)
        abs_sum += mean * got.size
        count += got.size
        fin = np.isfinite(l_ref)
        assert (np.isneginf(lse[h, r * b:(r + 1) * b]) == ~fin).all()
        lerr = float(np.abs(lse[h, r * b:(r + 1) * b][fin] - l_ref[fin]).max())
        assert lerr <= 1e-4
        worst_lse = max(worst_lse, lerr)
    print(f"\n[attention error] {wl.name}: {len(pairs)} sampled (head, query block) rows, "
          f"max-abs {worst:.3g}, mean-abs {abs_sum / count:.3g}, lse max {worst_lse:.3g}")


def test_end_to_end_mask_agreement(case):
    wl = case.wl
    _, _, sc = sp.sparsp_block_scores(case.g, case.Qd, case.Kd)
    m, _ = sp.sparsp_topk_mask(case.g, sc, wl.keep, wl.global_blocks)
    rows_equal = (m.cpu().numpy() == P.words_as_int64(case.mask)).all(axis=2)
    frac = float(rows_equal.mean())
    print(f"{wl.name}: {frac:.5f} of rows select the same blocks end to end")
    assert frac >= 0.98
