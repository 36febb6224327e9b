"""GPU parity at the size limits of the path and in its degenerate cases.

* The largest block count the library takes (n = 4096, the last block
  ragged) with every block kept: each row attends over 524,251 keys and its
  kept list fills 16 KB of LDS beside the tiles (32 KB for the float32
  kernel, whose case uses 16-token blocks).
* The largest head count (H = 1024; the head offsets are staged in LDS by the
  offsets and gather kernels).
* A sequence shorter than one block (n = 1: the whole sequence is one partial
  block), for each attention kernel and both gather kernels.

Selections, demand, offsets, slot maps and packed buffers are compared bit for
bit with the oracle given the same float32 scores; attention within the bars
of tests/_parity.py (bf16: 2e-2 max-abs, 1e-3 mean-abs; float32: 1e-5), lse
within 1e-4 (bf16) or 1e-5 (float32).
"""

import numpy as np
import pytest

import oracle as orc
import paper_2609_32197_amd as sp
from tests import _parity as P
from tests.test_gpu_kernels import _pipeline, _rand_inputs, ctypes_scale

pytestmark = pytest.mark.gpu


def _check(geo, keep, seed, heads=None, rows=None):
    H, L, d, b, i0, i1, dt = geo
    q, k, v = _rand_inputs(seed, H, L, d, dt)
    g = P.geometry(H, L, d, b, i0, i1, dt)
    om, osel, sel, out = _pipeline(q, k, v, g, dt, keep)
    np.testing.assert_array_equal(sel.cpu().numpy(), osel)
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
    del Kp, Vp

    scale = ctypes_scale(d)
    Qd = P.to_device(q, dt)
    outs = [sp.sparsp_block_sparse_attn(g, Qd, sel, out["slot_of"], out["K_packed"],
                                        out["V_packed"], scale, out_dtype=sp.F32)]
    if dt == "bf16":
        outs.append(sp.sparsp_block_sparse_attn(g, Qd, sel, out["slot_of"], out["K_packed"],
                                                out["V_packed"], scale, out_dtype=sp.BF16))
    outs = [(O.float().cpu().numpy(), lse.cpu().numpy()) for O, lse in outs]
    nq = i1 - i0
    for h in (range(H) if heads is None else heads):
        Qf, Kf, Vf = (orc.decode_input(x[h], dt) for x in (q, k, v))
        for r in (range(nq) if rows is None else rows):
            o_ref, l_ref = orc.attend_block(Qf, Kf, Vf, om[h, r], i0 + r, L, b, scale)
            for On, ln in outs:
                got = On[h, r * b:(r + 1) * b]
                P.check_attention(got, o_ref, dt == "bf16", f"{geo} h={h} r={r}")
                fin = np.isfinite(l_ref)
                lg = ln[h, r * b:(r + 1) * b]
                assert (np.isneginf(lg) == ~fin).all()
                assert np.abs(lg[fin] - l_ref[fin]).max() <= (1e-4 if dt == "bf16" else 1e-5)


def test_largest_block_count_dense_rows(gpu):
    # n = 4096 blocks of 128 (the last one 91 tokens), the last three query
    # blocks, every block kept
    L = 4095 * 128 + 91
    _check((1, L, 128, 128, 4093, 4096, "bf16"), keep=4096, seed=11)


def test_largest_block_count_dense_rows_f32(gpu):
    # the float32 kernel with n = 4096 blocks of 16 (the last one 7 tokens),
    # every block kept: its kept list (slots and counts) fills 32 KB of LDS
    L = 4095 * 16 + 7
    _check((1, L, 128, 16, 4094, 4096, "f32"), keep=4096, seed=14)


def test_largest_head_count(gpu):
    # H = 1024 heads, n = 10 blocks of 64 (the last one 54 tokens)
    _check((1024, 630, 64, 64, 0, 10, "bf16"), keep=3, seed=12,
           heads=[0, 1, 511, 1022, 1023])


@pytest.mark.parametrize("geo", [
    (2, 5, 128, 128, 0, 1, "bf16"),    # 128-token kernel, 5 valid tokens
    (2, 100, 64, 128, 0, 1, "bf16"),   # 128-token kernel, d = 64
    (2, 37, 64, 64, 0, 1, "bf16"),     # 64-token kernel
    (2, 3, 8, 4, 0, 1, "f32"),         # float32 kernel, windowed gather
    (3, 50, 128, 64, 0, 1, "f32"),     # float32 kernel, streaming gather
], ids=lambda g: "H{}L{}d{}b{}_{}-{}_{}".format(*g))
def test_sequence_shorter_than_one_block(gpu, geo):
    _check(geo, keep=1, seed=13)
