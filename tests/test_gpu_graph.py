"""The four-call step captured in a HIP graph (torch.cuda.CUDAGraph) and
replayed.

The library issues kernels only on the caller's stream: no memset, copy,
allocation or synchronisation. A captured step must therefore reproduce the
eager step bit for bit on every replay. The attention call is the
allocation-free balanced variant (the binding's fixed_scratch=True), the one
meant for callers under graph capture; its device-array address is looked up
by an eager call before the capture.

Before each replay the outputs are overwritten (torch's fill kernel, outside
the graph), so a replay that skipped a write would show. Between replays the
same step runs eagerly into other buffers, with a synchronisation, and must
match too.
"""

import pytest

import paper_2609_32197_amd as sp
from tests import _parity as P
from tests.test_gpu_kernels import _rand_inputs

pytestmark = pytest.mark.gpu

# (H, L, d, block, i0, i1, dtype, keep)
CASES = [
    (2, 4500, 128, 128, 0, 36, "bf16", 9),    # 128-token kernel, ragged last block (20 tokens)
    (3, 4100, 64, 64, 5, 60, "bf16", 12),     # 64-token kernel, ragged (4 tokens)
]


def _outputs(g, keep, Q):
    torch = P.torch()
    cap = g.H * g.n
    dev = Q.device
    e = lambda shape, dt: torch.empty(shape, dtype=dt, device=dev)
    return {
        "pooled_q": e((g.H, g.nq, g.d), torch.float32),
        "pooled_k": e((g.H, g.n, g.d), torch.float32),
        "scores": e((g.H, g.nq, g.n), torch.float32),
        "mask": e((g.H, g.nq, g.W), torch.int64),
        "sel": e((g.H, g.nq, keep), torch.int32),
        "packed": {
            "demand": e((g.H, g.W), torch.int64), "head_off": e((g.H + 1,), torch.int32),
            "slot_of": e((g.H, g.n), torch.int32), "gather_blk": e((cap,), torch.int32),
            "K_packed": e((cap, g.block, g.d), Q.dtype), "V_packed": e((cap, g.d, g.block), Q.dtype),
        },
        "O": e((g.H, g.nq * g.block, g.d), torch.bfloat16),
        "lse": e((g.H, g.nq * g.block), torch.float32),
    }


def _step(g, Q, K, V, keep, o):
    sp.sparsp_block_scores(g, Q, K, o["pooled_q"], o["pooled_k"], o["scores"])
    sp.sparsp_topk_mask(g, o["scores"], keep, (), mask=o["mask"], sel=o["sel"])
    p = sp.sparsp_demand_union_gather(g, o["mask"], K, V, out=o["packed"])
    sp.sparsp_block_sparse_attn(g, Q, o["sel"], p["slot_of"], p["K_packed"], p["V_packed"],
                                out_dtype=sp.BF16, O=o["O"], lse=o["lse"], fixed_scratch=True)


def _flat(o):
    out = {k: v for k, v in o.items() if k != "packed"}
    out.update({"packed." + k: v for k, v in o["packed"].items() if hasattr(v, "view")})
    return out


def _bits(t):
    torch = P.torch()
    return t.view(torch.int16) if t.element_size() == 2 else t.view(torch.int32) \
        if t.element_size() == 4 else t.view(torch.int64)


def _assert_same(got, ref, what):
    torch = P.torch()
    S = int(ref["packed.head_off"][-1].item())
    for k, r in ref.items():
        a, b = got[k], r
        if k in ("packed.gather_blk", "packed.K_packed", "packed.V_packed"):
            a, b = a[:S], b[:S]  # slots past the demanded ones are not written
        assert torch.equal(_bits(a), _bits(b)), f"{what}: {k} differs"


@pytest.mark.parametrize("case", CASES, ids=lambda c: "H{}L{}d{}b{}_{}-{}_{}_k{}".format(*c))
def test_captured_step_replays_bit_exact(gpu, case):
    torch = P.torch()
    H, L, d, b, i0, i1, dt, keep = case
    q, k, v = _rand_inputs(21, H, L, d, dt)
    g = P.geometry(H, L, d, b, i0, i1, dt)
    Q, K, V = (P.to_device(x, dt) for x in (q, k, v))

    ref = _outputs(g, keep, Q)
    _step(g, Q, K, V, keep, ref)  # eager; also looks up the fixed array's address
    torch.cuda.synchronize()
    ref = _flat(ref)

    bufs = _outputs(g, keep, Q)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        _step(g, Q, K, V, keep, bufs)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        _step(g, Q, K, V, keep, bufs)
    torch.cuda.synchronize()

    flat = _flat(bufs)
    for rep in range(3):
        for t in flat.values():
            _bits(t).fill_(-1)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        _assert_same(flat, ref, f"replay {rep}")
        eager = _outputs(g, keep, Q)
        _step(g, Q, K, V, keep, eager)
        torch.cuda.synchronize()
        _assert_same(_flat(eager), ref, f"eager run after replay {rep}")
