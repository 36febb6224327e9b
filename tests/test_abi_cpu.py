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
    return sorted(set(re.findall(r"^\s*(?:int|int64_t|const char\*)\s+(sparsp_\w+)\s*\(", text,
                                 re.M)))


def test_header_declares_the_four_steps():
    names = declared_functions()
    for want in ("sparsp_block_scores", "sparsp_topk_mask", "sparsp_demand_union_gather",
                 "sparsp_block_sparse_attn", "sparsp_last_error", "sparsp_version"):
        assert want in names


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_header_declares_the_shard_by_shard_calls():
    names = declared_functions()
    for want in ("sparsp_chunk_plan", "sparsp_block_sparse_attn_part", "sparsp_lse_merge",
                 "sparsp_chunked_attn"):
        assert want in names


def test_version(lib):
    assert lib.sparsp_version() == 200


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


# ---------------------------------------------------------------------------
# the chunk schedule is host code: it runs here, against the oracle
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(8))
def test_chunk_plan_matches_the_oracle(lib, seed):
    import numpy as np
    import oracle as orc
    rng = np.random.default_rng(100 + seed)
    H = int(rng.integers(1, 12))
    block = 16
    n = int(rng.integers(2, 150))
    L = n * block - int(rng.integers(0, block))
    ranks = int(rng.integers(1, min(n, 9) + 1))
    rank = int(rng.integers(0, ranks))
    hpc, tail = int(rng.integers(1, 6)), int(rng.integers(1, 4))
    demand = rng.random((H, n)) < rng.uniform(0.05, 0.9)
    g = sp.Geometry(H, L, 64, block, 0, 1, sp.F32)
    got = [c.astuple() for c in sp.sparsp_chunk_plan(g, orc.mask_to_words(demand), ranks, rank,
                                                     hpc, tail)]
    assert got == orc.chunk_plan(demand, ranks, rank, hpc, tail)


def test_chunk_plan_rejected(lib):
    import numpy as np
    g = geom(H=4, L=1024, block=128, i0=0, i1=8)  # n = 8
    dem = np.zeros((4, 1), dtype=np.uint64)
    arr = (sp.Chunk * 64)()
    call = lambda ranks, rank, a, b, cap=64: lib.sparsp_chunk_plan(
        ctypes.byref(g), dem.ctypes.data, ranks, rank, a, b, arr, cap)
    assert call(0, 0, 1, 1) == E_INVALID
    assert call(9, 0, 1, 1) == E_INVALID  # more ranks than blocks
    assert call(4, 4, 1, 1) == E_INVALID
    assert call(4, -1, 1, 1) == E_INVALID
    assert call(4, 0, 0, 1) == E_INVALID
    assert call(4, 0, 1, 0) == E_INVALID
    assert call(4, 0, 1, 1, cap=12) == E_CAPACITY  # needs 1 + 3 * 4 = 13
    assert b"13" in lib.sparsp_last_error()
    assert call(4, 0, 1, 1, cap=13) == 13
    assert call(1, 0, 1, 1) == 1
    assert lib.sparsp_chunk_plan(ctypes.byref(g), None, 4, 0, 1, 1, arr, 64) == E_INVALID


def test_part_and_merge_rejected(lib):
    g = geom()  # H = 2, n = 8
    part = lambda lo, hi, h0, h1, lse=P: lib.sparsp_block_sparse_attn_part(
        ctypes.byref(g), P, P, 2, P, P, P, 16, 0.125, lo, hi, h0, h1, P, lse, 0, None)
    assert part(0, 9, 0, 2) == E_INVALID
    assert part(-1, 4, 0, 2) == E_INVALID
    assert part(5, 4, 0, 2) == E_INVALID
    assert part(0, 8, 1, 1) == E_INVALID
    assert part(0, 8, 0, 3) == E_INVALID
    assert part(0, 8, 0, 2, lse=None) == E_INVALID  # lse is required
    merge = lambda h0, h1, a=P, b=P + 4096: lib.sparsp_lse_merge(
        ctypes.byref(g), h0, h1, a, a + 8192, b, b + 8192, None)
    assert merge(0, 3) == E_INVALID
    assert merge(1, 1) == E_INVALID
    assert merge(0, 2, b=P) == E_INVALID  # part aliases the accumulator
    assert merge(0, 2, a=P + 4) == E_INVALID  # misaligned
    bad = (sp.Chunk * 1)(sp.Chunk(0, 0, 9, 0, 2, 0))
    assert lib.sparsp_chunked_attn(ctypes.byref(g), P, P, 2, P, P, P, 16, 0.125, bad, 1, P, P,
                                   None) == E_INVALID


# ---------------------------------------------------------------------------
# placement and the Eq. 3 count are host code: they run here, against the oracle
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(8))
def test_periodic_placement_matches_the_oracle(lib, seed):
    import numpy as np
    import oracle as orc
    rng = np.random.default_rng(200 + seed)
    block = int(rng.choice([8, 16, 64, 128]))
    F = int(rng.integers(block // 2 + 1, 40 * block))
    L = int(rng.integers(2 * block, 3000 * 8))
    n = -(-L // block)
    if n > 4096:
        L = 4096 * block
        n = 4096
    ranks = int(rng.integers(1, min(n, 9) + 1))
    perm, begin = sp.sparsp_periodic_placement(L, block, F, ranks)
    operm, obegin = orc.placement_permutation(orc.periodic_owner(L, block, F, ranks), ranks)
    assert perm.tolist() == operm.tolist() and begin.tolist() == obegin.tolist()


@pytest.mark.parametrize("seed", range(6))
def test_remote_demand_matches_the_oracle(lib, seed):
    import numpy as np
    import oracle as orc
    rng = np.random.default_rng(300 + seed)
    H, n = int(rng.integers(1, 9)), int(rng.integers(2, 300))
    ranks = int(rng.integers(1, min(n, 8) + 1))
    r = int(rng.integers(0, ranks))
    lo, hi = orc.local_range(n, ranks, r)
    demand = rng.random((H, n)) < 0.3
    g = sp.Geometry(H, n * 16, 64, 16, lo, hi, sp.F32)
    remote, total = sp.sparsp_remote_demand(g, orc.mask_to_words(demand))
    assert remote == orc.remote_blocks(demand, orc.contiguous_owner(n, ranks), r)
    assert total == int(demand.sum())


def test_placement_and_permute_rejected(lib):
    import numpy as np
    perm = np.zeros(64, dtype=np.int32)
    begin = np.zeros(9, dtype=np.int32)
    call = lambda L, b, F, R: lib.sparsp_periodic_placement(L, b, F, R, perm.ctypes.data,
                                                           begin.ctypes.data)
    assert call(0, 8, 64, 2) == E_INVALID
    assert call(64, 0, 64, 2) == E_INVALID
    assert call(64, 8, 0, 2) == E_INVALID
    assert call(64, 8, 64, 0) == E_INVALID
    assert call(64, 8, 64, 9) == E_INVALID  # more ranks than blocks
    assert lib.sparsp_periodic_placement(64, 8, 64, 2, None, begin.ctypes.data) == E_INVALID
    g = geom()
    assert lib.sparsp_permute_blocks(ctypes.byref(g), P, P, P, 0, None) == E_INVALID  # X == Y
    assert lib.sparsp_permute_blocks(ctypes.byref(g), P, P, P + 8, 0, None) == E_INVALID
    assert lib.sparsp_permute_blocks(ctypes.byref(g), None, P, P + 4096, 0, None) == E_INVALID


def test_cdf_mask_rejected(lib):
    g = geom(L=1024, block=128, i0=2, i1=6)  # n = 8
    call = lambda tau, glob=(), ng=None: lib.sparsp_cdf_mask(
        ctypes.byref(g), P, tau, (ctypes.c_int32 * max(1, len(glob)))(*glob) if glob else None,
        len(glob) if ng is None else ng, P, P, P, None)
    assert call(0.0) == E_INVALID
    assert call(-0.5) == E_INVALID
    assert call(1.01) == E_INVALID
    assert call(float("nan")) == E_INVALID
    assert call(0.9, glob=(8,)) == E_INVALID
    assert call(0.9, ng=2) == E_INVALID
    assert lib.sparsp_cdf_mask(ctypes.byref(g), P, 0.9, None, 0, P, P, None, None) == E_INVALID


# ---------------------------------------------------------------------------
# demand-directed routing: the volume counter is host code
# ---------------------------------------------------------------------------

def test_route_volume_reproduces_the_paper_example(lib):
    import json
    import numpy as np
    import oracle as orc
    ex = json.load(open(os.path.join(ROOT, "tests", "golden", "cross_ring_example.json")))
    R, names = ex["ranks"], ex["blocks"]
    n = R * len(names)
    dem = [np.zeros((1, n), dtype=bool) for _ in range(R)]
    for c, blocks in ex["demand"].items():
        for name in blocks:
            dem[int(c)][0, names.index(name)] = True
    words = np.stack([orc.mask_to_words(d) for d in dem])
    g = sp.Geometry(1, n * 8, 64, 8, 0, 1, sp.F32)
    vol = sp.sparsp_route_volume(g, words, R, ex["producer"])
    assert vol["relay"] == ex["relay_block_hops"] and vol["direct"] == ex["direct_blocks"]
    assert vol["dense"] == (R - 1) * len(names)


@pytest.mark.parametrize("seed", range(6))
def test_route_volume_matches_the_oracle(lib, seed):
    import numpy as np
    import oracle as orc
    rng = np.random.default_rng(400 + seed)
    H, n = int(rng.integers(1, 7)), int(rng.integers(2, 200))
    R = int(rng.integers(2, min(n, 9) + 1))
    p = int(rng.integers(0, R))
    demands = [rng.random((H, n)) < rng.uniform(0.05, 0.6) for _ in range(R)]
    words = np.stack([orc.mask_to_words(d) for d in demands])
    g = sp.Geometry(H, n * 16, 64, 16, 0, 1, sp.F32)
    lo, hi = orc.local_range(n, R, p)
    assert sp.sparsp_route_volume(g, words, R, p) == orc.route_volume(
        orc.provide_masks(demands, R, p), hi - lo)


def test_routing_rejected(lib):
    g = geom(H=4, L=1024, block=128, i0=0, i1=8)  # n = 8
    pack = lambda R, p, cap=1 << 20, K=P: lib.sparsp_pack_for_consumers(
        ctypes.byref(g), P, R, p, K, P, P, P, P, P, P, P, cap, None)
    assert pack(1, 0) == E_INVALID
    assert pack(9, 0) == E_INVALID
    assert pack(4, 4) == E_INVALID
    assert pack(4, 0, cap=23) == E_CAPACITY  # 3 consumers x 4 heads x 2 shard blocks = 24
    assert pack(4, 0, K=P + 8) == E_INVALID
    big = geom(H=300, L=1024, block=128, i0=0, i1=8)
    assert lib.sparsp_pack_for_consumers(ctypes.byref(big), P, 8, 0, P, P, P, P, P, P, P, P,
                                         1 << 30, None) == E_UNSUPPORTED  # 7 * 300 > 1024
    z = ctypes.c_int64()
    assert lib.sparsp_route_volume(ctypes.byref(g), P, 1, 0, ctypes.byref(z), ctypes.byref(z),
                                   ctypes.byref(z)) == E_INVALID


def test_mfma_probe_is_outside_the_abi(lib):
    """The benchmark's MFMA probe lives in its own library, not in libsparsp."""
    from paper_2609_32197_amd import probe
    assert not hasattr(lib, "sparsp_mfma_probe")
    assert probe.status(0, 4, P) == E_INVALID
    assert probe.status(10, 0, P) == E_INVALID
    assert probe.status(10, (1 << 20) + 1, P) == E_INVALID
    assert probe.status(10, 4, None) == E_INVALID
    # the unit probes beside it reject bad arguments before any launch
    u = probe._load().unit_probe_run
    assert not hasattr(lib, "unit_probe_run")
    assert u(3, 10, 4, P, None) == E_INVALID     # no such probe
    assert u(-1, 10, 4, P, None) == E_INVALID
    assert u(0, 0, 4, P, None) == E_INVALID      # iters < 1
    assert u(2, 10, 0, P, None) == E_INVALID     # no workgroups
    assert u(1, 10, (1 << 20) + 1, P, None) == E_INVALID
    assert u(1, 10, 4, None, None) == E_INVALID  # no sink


def test_row_order_and_ordered_attention_rejected(lib):
    g = geom(H=2, L=1024, block=128, i0=0, i1=8)
    assert lib.sparsp_row_order(ctypes.byref(g), None, P, None) == E_INVALID
    assert lib.sparsp_row_order(ctypes.byref(g), P, None, None) == E_INVALID
    bad = geom(H=2, L=1024, block=128, i0=3, i1=3)
    assert lib.sparsp_row_order(ctypes.byref(bad), P, P, None) == E_INVALID
    gb = geom(H=2, L=1024, d=128, block=128, i0=0, i1=8, dtype=sp.BF16)
    attn = lambda order, keep=4: lib.sparsp_block_sparse_attn_ordered(
        ctypes.byref(gb), P, P, keep, P, P, P, 16, 0.1, order, P, sp.BF16, None, None)
    assert attn(None) == E_INVALID
    assert attn(P, keep=0) == E_INVALID
    assert attn(P, keep=9) == E_INVALID


def test_balanced_attention_rejected(lib):
    g = geom(H=2, L=1024, d=128, block=128, i0=0, i1=8, dtype=sp.BF16)

    def call(ws=P, ws_bytes=1 << 20, keep=4, out=sp.BF16):
        return lib.sparsp_block_sparse_attn_balanced(ctypes.byref(g), P, P, keep, P, P, P, 16, 0.1,
                                                     ws, ws_bytes, P, out, None, None)
    assert call(ws=P + 8) == E_INVALID        # misaligned workspace
    assert call(ws_bytes=-1) == E_INVALID
    assert call(keep=0) == E_INVALID
    assert call(keep=9) == E_INVALID
    assert call(out=7) == E_DTYPE
    assert lib.sparsp_attn_workspace_bytes(ctypes.byref(g), 0) == E_INVALID
    bad = geom(i0=3, i1=3)
    assert lib.sparsp_attn_workspace_bytes(ctypes.byref(bad), 1) == E_INVALID
    gf = geom(H=2, L=1000, d=64, block=64, i0=0, i1=4, dtype=sp.F32)
    assert lib.sparsp_attn_workspace_bytes(ctypes.byref(gf), 4) == 0   # float32: no split
