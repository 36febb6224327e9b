"""Longest-first row order and attention launched in a given row order.

sparsp_row_order is a scheduling helper, not a step of the method. What it
fixes is compared exactly: which heads share each of the eight XCD queues
(recomputed here from the documented rule) and that every queue runs longest
first. The rest is checked for validity: the order is a permutation, and rows
of equal count may come in any order.
sparsp_block_sparse_attn_ordered changes only which workgroup computes which
row, so its outputs must equal sparsp_block_sparse_attn's bit for bit, for
every kernel family, under a CDF selection (rows of very unequal length).
"""

import numpy as np
import pytest

import paper_2609_32197_amd as sp
from tests import _parity as P
from tests.test_gpu_kernels import _rand_inputs, ctypes_scale

pytestmark = pytest.mark.gpu


def _queues(counts, n):
    """The head -> queue assignment sparsp_row_order documents, and queue lengths."""
    H, nq = counts.shape
    c = np.clip(counts, 0, n).astype(np.int64)
    tot = c.sum(axis=1)
    room = [H // 8 + (1 if x < H % 8 else 0) for x in range(8)]
    qlen = [r * nq for r in room]
    load = [0] * 8
    q = {}
    for h in sorted(range(H), key=lambda h: (-tot[h], h)):
        best = min((x for x in range(8) if room[x] > 0), key=lambda x: (load[x], x))
        q[h] = best
        load[best] += int(tot[h])
        room[best] -= 1
    return q, qlen


@pytest.mark.parametrize("H,nq,n,lo,hi", [
    (1, 1, 1, 0, 2), (2, 7, 16, 0, 17), (3, 40, 591, 1, 592), (40, 147, 591, 1, 300),
    (2, 300, 4096, 0, 4097), (5, 11, 64, -3, 70), (19, 9, 128, 1, 129),
    # more rows than the kernel keeps in LDS (14,336): counts read from memory
    (24, 929, 929, 0, 930), (1024, 16, 64, 0, 65), (112, 128, 256, 0, 257)])
def test_row_order_balances_heads_and_sorts_rows(gpu, H, nq, n, lo, hi):
    torch = P.torch()
    rng = np.random.default_rng(H * 1000 + nq)
    counts = rng.integers(lo, hi, size=(H, nq)).astype(np.int32)
    counts.flat[:: max(1, counts.size // 5)] = counts.flat[0]  # ties
    g = P.geometry(H, n * 64, 64, 64, 0, nq, "f32")
    order = sp.sparsp_row_order(g, torch.from_numpy(counts).cuda()).cpu().numpy()
    assert sorted(order.tolist()) == list(range(H * nq))          # a permutation
    q, qlen = _queues(counts, n)
    clamped = np.clip(counts.reshape(-1), 0, n)
    # walk the round-robin interleave back into the eight queues
    queues, pos = [[] for _ in range(8)], 0
    for k in range(max(qlen) if qlen else 0):
        for x in range(8):
            if k < qlen[x]:
                queues[x].append(int(order[pos]))
                pos += 1
    for x in range(8):
        rows = queues[x]
        assert {r // nq for r in rows} == {h for h, y in q.items() if y == x}
        seq = clamped[rows]
        np.testing.assert_array_equal(seq, np.sort(seq)[::-1])  # longest first


GEOMS = [
    (3, 9000, 128, 128, 20, 71, "bf16"),   # 128-token kernel
    (2, 4400, 64, 128, 3, 35, "bf16"),     # 128-token kernel, d = 64
    (2, 4500, 64, 64, 30, 71, "bf16"),     # 64-token kernel
    (3, 1000, 64, 64, 5, 16, "f32"),       # float32 kernel
]


@pytest.mark.parametrize("geo", GEOMS, ids=lambda g: "H{}L{}d{}b{}_{}-{}_{}".format(*g))
def test_ordered_attention_is_bit_identical(gpu, geo):
    torch = P.torch()
    H, L, d, b, i0, i1, dt = geo
    q, k, v = _rand_inputs(21, H, L, d, dt)
    g = P.geometry(H, L, d, b, i0, i1, dt)
    Q, K, V = (P.to_device(x, dt) for x in (q, k, v))
    _, _, sc = sp.sparsp_block_scores(g, Q, K)
    m, sel, cnt = sp.sparsp_cdf_mask(g, sc, 0.9)
    out = sp.sparsp_demand_union_gather(g, m, K, V)
    args = (g, Q, sel, out["slot_of"], out["K_packed"], out["V_packed"], ctypes_scale(d))
    odts = [sp.F32] + ([sp.BF16] if dt == "bf16" else [])
    longest = sp.sparsp_row_order(g, cnt)
    shuffled = torch.from_numpy(np.random.default_rng(2).permutation(H * (i1 - i0)).astype(np.int32)).cuda()
    for odt in odts:
        O0, l0 = sp.sparsp_block_sparse_attn(*args, out_dtype=odt)
        for order in (longest, shuffled):
            O1, l1 = sp.sparsp_block_sparse_attn(*args, out_dtype=odt, row_order=order)
            assert torch.equal(O0.view(torch.int16) if odt == sp.BF16 else O0.view(torch.int32),
                               O1.view(torch.int16) if odt == sp.BF16 else O1.view(torch.int32))
            assert torch.equal(l0.view(torch.int32), l1.view(torch.int32))


def test_ordered_attention_full_size_wan_share(gpu):
    torch = P.torch()
    from workloads import get_workload, make_qkv
    wl = get_workload("wan-share")
    q, k, v = make_qkv(wl)
    g = P.geometry(wl.H, wl.L, wl.d, wl.block, wl.i0, wl.i1, wl.dtype)
    Q, K, V = (P.to_device(x, wl.dtype) for x in (q, k, v))
    _, _, sc = sp.sparsp_block_scores(g, Q, K)
    m, sel, cnt = sp.sparsp_cdf_mask(g, sc, 0.9)
    out = sp.sparsp_demand_union_gather(g, m, K, V)
    args = (g, Q, sel, out["slot_of"], out["K_packed"], out["V_packed"], wl.softmax_scale)
    O0, l0 = sp.sparsp_block_sparse_attn(*args)
    order = sp.sparsp_row_order(g, cnt)
    assert sorted(order.cpu().numpy().tolist()) == list(range(wl.H * (wl.i1 - wl.i0)))
    O1, l1 = sp.sparsp_block_sparse_attn(*args, row_order=order)
    assert torch.equal(O0.view(torch.int16), O1.view(torch.int16))
    assert torch.equal(l0.view(torch.int32), l1.view(torch.int32))
