"""The attention entry point that allocates nothing
(sparsp_block_sparse_attn_balanced_noalloc), called through the C ABI.

Its last-round split writes float32 partials to the library's fixed device
array instead of a caller workspace, so its outputs must equal those of
sparsp_block_sparse_attn_balanced with a workspace of
sparsp_attn_workspace_bytes bytes, bit for bit (same kernels, same split).
Two calls run in a row on geometries whose last round is split, the second
smaller than the first, so the second finds the first call's partials in the
array and must not depend on them. Neither call is given a workspace; the
outputs are preallocated, so the calls themselves allocate nothing.
"""

import ctypes

import numpy as np
import pytest

import paper_2609_32197_amd as sp
from tests import _parity as P
from tests.test_gpu_kernels import _pipeline, _rand_inputs, ctypes_scale

pytestmark = pytest.mark.gpu

# (H, L, d, block, i0, i1, dtype, keep fraction): rows against resident slots
# (512 for 128-token blocks, 1,024 for 64-token blocks on a 256-CU part)
CALLS = [
    (8, 35900, 128, 128, 0, 280, "bf16", 0.3),   # 2,240 rows: a partial last round
    (3, 9000, 128, 128, 20, 71, "bf16", 0.4),    # 153 rows: every row split in pieces
    (12, 16000, 64, 64, 0, 180, "bf16", 0.2),    # 64-token kernel, 2,160 rows
    (2, 4100, 64, 64, 5, 60, "bf16", 0.5),       # smaller again, 110 rows
]


def _call(lib, fn, g, args, extra_ws=None):
    gs = g.c_struct()
    (Q, sel, keep, slot_of, Kp, Vp, cap, scale, O, odt, lse, stream) = args
    if extra_ws is None:
        return getattr(lib, fn)(ctypes.byref(gs), Q, sel, keep, slot_of, Kp, Vp, cap, scale, O,
                                odt, lse, stream)
    ws, nbytes = extra_ws
    return getattr(lib, fn)(ctypes.byref(gs), Q, sel, keep, slot_of, Kp, Vp, cap, scale, ws,
                            nbytes, O, odt, lse, stream)


def test_noalloc_equals_balanced_twice(gpu):
    torch = P.torch()
    lib = sp.load_library()
    for H, L, d, b, i0, i1, dt, frac in CALLS:
        n = -(-L // b)
        keep = max(1, int(round(frac * n)))
        q, k, v = _rand_inputs(11, H, L, d, dt)
        g = P.geometry(H, L, d, b, i0, i1, dt)
        _, _, sel, out = _pipeline(q, k, v, g, dt, keep)
        Qd = P.to_device(q, dt)
        nq = i1 - i0
        nbytes = sp.sparsp_attn_workspace_bytes(g, keep)
        assert 0 < nbytes <= (36 << 20), nbytes
        ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        results = {}
        for fn in ("sparsp_block_sparse_attn_balanced", "sparsp_block_sparse_attn_balanced_noalloc"):
            O = torch.full((H, nq * b, d), float("nan"), dtype=torch.bfloat16, device="cuda")
            lse = torch.full((H, nq * b), float("nan"), dtype=torch.float32, device="cuda")
            stream = torch.cuda.current_stream().cuda_stream
            args = (Qd.data_ptr(), sel.data_ptr(), keep, out["slot_of"].data_ptr(),
                    out["K_packed"].data_ptr(), out["V_packed"].data_ptr(),
                    int(out["K_packed"].shape[0]), ctypes_scale(d), O.data_ptr(), sp.BF16,
                    lse.data_ptr(), stream)
            rc = _call(lib, fn, g, args,
                       (ws.data_ptr(), nbytes) if fn.endswith("balanced") else None)
            assert rc == 0, (fn, rc, lib.sparsp_last_error())
            torch.cuda.synchronize()
            results[fn] = (O.view(torch.int16).cpu().numpy(), lse.view(torch.int32).cpu().numpy())
        (o0, l0), (o1, l1) = results.values()
        np.testing.assert_array_equal(o1, o0)
        np.testing.assert_array_equal(l1, l0)
        print(f"H{H} L{L} d{d} b{b} rows {H * nq} keep {keep}: equal bit for bit "
              f"(workspace of the balanced call {nbytes} B)")
