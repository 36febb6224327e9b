"""The C ABI without a GPU: the library loads, exports what include/sparsp.h
declares, and rejects bad arguments on the host before launching anything.

Every call here fails argument checking, so no kernel is launched and the
dummy device addresses are never touched.
"""

import ctypes
import os
import re

import pytest

import paper_2609_32197_amd as sp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sparsp.h")

E_INVALID, E_DTYPE, E_UNSUPPORTED, E_CAPACITY = -1, -2, -3, -4
P = 1 << 20  # a 16-byte aligned dummy device address (never dereferenced)


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(sp.lib_path()):
        pytest.fail("libsparsp.so is not built; run python -m paper_2609_32197_amd.build")
    return sp.load_library()


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:int|const char\*)\s+(sparsp_\w+)\s*\(", text, re.M)))


def test_header_declares_the_four_steps():
    names = declared_functions()
    for want in ("sparsp_block_scores", "sparsp_topk_mask", "sparsp_demand_union_gather",
                 "sparsp_block_sparse_attn", "sparsp_last_error", "sparsp_version"):
        assert want in names


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_version(lib):
    assert lib.sparsp_version() == 100


def geom(H=2, L=1024, d=128, block=128, i0=0, i1=8, dtype=sp.BF16):
    return sp.Geometry(H, L, d, block, i0, i1, dtype).c_struct()


def scores_call(lib, g):
    return lib.sparsp_block_scores(ctypes.byref(g) if g is not None else None, P, P, P, P, P, None)


def test_geometry_rejected(lib):
    assert lib.sparsp_block_scores(None, P, P, P, P, P, None) == E_INVALID
    assert b"NULL" in lib.sparsp_last_error()
    assert scores_call(lib, geom(H=0)) == E_INVALID
    assert scores_call(lib, geom(L=-5)) == E_INVALID
    assert scores_call(lib, geom(dtype=7)) == E_DTYPE
    assert scores_call(lib, geom(i0=3, i1=3)) == E_INVALID
    assert scores_call(lib, geom(i0=0, i1=9)) == E_INVALID  # n = 8
    assert scores_call(lib, geom(i0=-1, i1=2)) == E_INVALID
    assert scores_call(lib, geom(L=4097 * 16, block=16, i1=1)) == E_UNSUPPORTED  # n > 4096
    assert scores_call(lib, geom(d=100)) == E_UNSUPPORTED  # d % 8 for bf16
    assert scores_call(lib, geom(d=320)) == E_UNSUPPORTED
    assert lib.sparsp_block_scores(ctypes.byref(geom()), P + 4, P, P, P, P, None) == E_INVALID
    assert lib.sparsp_block_scores(ctypes.byref(geom()), P, 0, P, P, P, None) == E_INVALID
    assert b"" != lib.sparsp_last_error()


def topk_call(lib, g, keep, glob=(), n_global=None):
    arr = (ctypes.c_int32 * max(1, len(glob)))(*glob)
    ng = len(glob) if n_global is None else n_global
    return lib.sparsp_topk_mask(ctypes.byref(g), P, keep, arr if glob else None, ng, P, P, None)


def test_topk_rejected(lib):
    g = geom(L=1024, block=128, i0=2, i1=6)  # n = 8
    assert topk_call(lib, g, 9) == E_INVALID  # keep > n
    assert topk_call(lib, g, 0) == E_INVALID  # keep < |{diagonal}|
    assert topk_call(lib, g, 2, glob=(7, 0)) == E_INVALID  # |F| = 3 for every row
    assert topk_call(lib, g, 2, glob=(8,)) == E_INVALID  # out of range
    assert topk_call(lib, g, 2, glob=(-1,)) == E_INVALID
    assert topk_call(lib, g, 2, n_global=3) == E_INVALID  # NULL list with n_global > 0
    big = geom(L=128 * 100, block=128, i0=0, i1=4)
    assert topk_call(lib, big, 90, glob=tuple(range(10, 75))) == E_UNSUPPORTED  # > 64 globals
    assert lib.sparsp_topk_mask(ctypes.byref(g), None, 3, None, 0, P, P, None) == E_INVALID


def gather_call(lib, g, cap, K=P):
    return lib.sparsp_demand_union_gather(ctypes.byref(g), P, K, P, P, P, P, P, P, P, cap, None)


def test_demand_gather_rejected(lib):
    g = geom(H=3, L=1000, block=128, i0=0, i1=8)  # n = 8
    assert gather_call(lib, g, 23) == E_CAPACITY
    assert b"capacity" in lib.sparsp_last_error()
    assert gather_call(lib, g, 24, K=P + 8) == E_INVALID
    assert gather_call(lib, geom(H=3, L=1000, block=100, i1=10), 1000) == E_UNSUPPORTED
    assert gather_call(lib, geom(dtype=sp.F32, d=64, block=30, L=300, i1=10), 1000) == E_UNSUPPORTED


def attn_call(lib, g, keep=2, cap=16, scale=0.125, out=sp.BF16, Q=P):
    return lib.sparsp_block_sparse_attn(ctypes.byref(g), Q, P, keep, P, P, P, cap, scale, P, out,
                                        None, None)


def test_attention_rejected(lib):
    assert attn_call(lib, geom(), keep=0) == E_INVALID
    assert attn_call(lib, geom(), keep=9) == E_INVALID
    assert attn_call(lib, geom(), cap=0) == E_CAPACITY
    assert attn_call(lib, geom(), scale=0.0) == E_INVALID
    assert attn_call(lib, geom(), scale=float("nan")) == E_INVALID
    assert attn_call(lib, geom(), out=3) == E_DTYPE
    assert attn_call(lib, geom(d=96)) == E_UNSUPPORTED  # bf16 MFMA variants: d in {64, 128}
    assert attn_call(lib, geom(block=32, L=256)) == E_UNSUPPORTED
    assert attn_call(lib, geom(dtype=sp.F32, d=192), out=sp.F32) == E_UNSUPPORTED
    assert attn_call(lib, geom(dtype=sp.F32, d=64), out=sp.BF16) == E_DTYPE
    assert attn_call(lib, geom(dtype=sp.F32, d=64, block=512, L=4096), out=sp.F32) == E_UNSUPPORTED
    assert attn_call(lib, geom(), Q=0) == E_INVALID


def test_binding_rejects_host_tensors():
    torch = pytest.importorskip("torch")
    g = sp.Geometry(1, 128, 64, 64, 0, 2, sp.F32)
    Q = torch.zeros(1, 128, 64)
    with pytest.raises(ValueError, match="GPU"):
        sp.sparsp_block_scores(g, Q, Q, pooled_q=Q, pooled_k=Q, scores=Q)


def test_binding_reports_status_names(lib):
    e = sp.SparspError(-4, "capacity_blocks too small")
    assert e.status == "SPARSP_E_CAPACITY" and "capacity" in str(e)
