"""Python binding of libsparsp: one rank's share of SparSP sparse attention on MI355X.

The four calls mirror the C ABI in include/sparsp.h one to one and only
marshal arguments: tensors are torch tensors on the GPU (torch provides the
device memory and the stream), every step of the computation runs in the
library's HIP kernels. There is no fallback: if the library is not built, or
a tensor is not on the GPU, the call raises.

    sparsp_block_scores         pooled Q/K tiles and block scores (Section 4.2)
    sparsp_topk_mask            top-k block mask with forced diagonal (Section 4.1)
    sparsp_demand_union_gather  per-head demand (Eq. 2) and packed K/V (Section 5.2)
    sparsp_block_sparse_attn    attention of the local query blocks (Eq. 1)
    sparsp_cdf_mask             CDF-mode block mask (Section 8.1), instead of top-k
    sparsp_block_sparse_attn(..., workspace=)  attention with the last round balanced

Shard-by-shard attention (Section 2.3, Section 7):

    sparsp_chunk_plan              the chunk schedule of one rank (host)
    sparsp_block_sparse_attn_part  attention over one shard for a run of heads
    sparsp_lse_merge               online-softmax merge of two partial results
    sparsp_chunked_attn            a whole schedule, attended and merged

Dependency-aware placement (Section 4.3, Eq. 4):

    sparsp_periodic_placement      placed order of the blocks per rank (host)
    sparsp_permute_blocks          token blocks into placed order and back
    sparsp_remote_demand           Eq. 3's remote block count of a rank (host)

Demand-directed KV routing (Section 5):

    sparsp_pack_for_consumers      a producer's packed blocks for every consumer
    sparsp_route_volume            dense / relay / direct block-hops (host)

Short aliases without the prefix are provided as well.
"""

from __future__ import annotations

import ctypes
import math
import os
import threading
from dataclasses import dataclass
from typing import Optional, Sequence

__all__ = [
    "SparspError",
    "Geometry",
    "lib_path",
    "load_library",
    "version",
    "sparsp_block_scores",
    "sparsp_topk_mask",
    "sparsp_demand_union_gather",
    "sparsp_block_sparse_attn",
    "block_scores",
    "topk_mask",
    "demand_union_gather",
    "block_sparse_attn",
    "Chunk",
    "sparsp_chunk_plan",
    "sparsp_block_sparse_attn_part",
    "sparsp_lse_merge",
    "sparsp_chunked_attn",
    "chunk_plan",
    "block_sparse_attn_part",
    "lse_merge",
    "chunked_attn",
    "sparsp_cdf_mask",
    "cdf_mask",
    "sparsp_periodic_placement",
    "sparsp_permute_blocks",
    "sparsp_remote_demand",
    "sparsp_pack_for_consumers",
    "sparsp_route_volume",
    "sparsp_row_order",
    "sparsp_attn_workspace_bytes",
    "row_order",
    "attn_workspace_bytes",
    "pack_for_consumers",
    "route_volume",
    "periodic_placement",
    "permute_blocks",
    "remote_demand",
    "F32",
    "BF16",
    "STATUS",
]

F32, BF16 = 0, 1
STATUS = {0: "SPARSP_OK", -1: "SPARSP_E_INVALID", -2: "SPARSP_E_DTYPE",
          -3: "SPARSP_E_UNSUPPORTED", -4: "SPARSP_E_CAPACITY", -5: "SPARSP_E_HIP"}

_HERE = os.path.dirname(os.path.abspath(__file__))
_LOCK = threading.Lock()
_LIB = None


def lib_path() -> str:
    return os.path.join(_HERE, "libsparsp.so")


class SparspError(RuntimeError):
    def __init__(self, code: int, message: str):
        self.code = code
        self.status = STATUS.get(code, str(code))
        super().__init__(f"{self.status}: {message}")


class _Geom(ctypes.Structure):
    _fields_ = [("H", ctypes.c_int32), ("L", ctypes.c_int32), ("d", ctypes.c_int32),
                ("block", ctypes.c_int32), ("q_blk_begin", ctypes.c_int32),
                ("q_blk_end", ctypes.c_int32), ("dtype", ctypes.c_int32)]


@dataclass(frozen=True)
class Geometry:
    """sparsp_geom: Q/K/V are [H, L, d]; local query blocks [i0, i1) of n = ceil(L/block)."""

    H: int
    L: int
    d: int
    block: int
    i0: int
    i1: int
    dtype: int  # F32 or BF16

    @property
    def n(self) -> int:
        return -(-self.L // self.block)

    @property
    def nq(self) -> int:
        return self.i1 - self.i0

    @property
    def W(self) -> int:
        return -(-self.n // 64)

    def c_struct(self) -> _Geom:
        return _Geom(self.H, self.L, self.d, self.block, self.i0, self.i1, self.dtype)


class Chunk(ctypes.Structure):
    """sparsp_chunk: shard [kv_blk_begin, kv_blk_end) of `owner`, heads [head_begin, head_end)."""

    _fields_ = [("owner", ctypes.c_int32), ("kv_blk_begin", ctypes.c_int32),
                ("kv_blk_end", ctypes.c_int32), ("head_begin", ctypes.c_int32),
                ("head_end", ctypes.c_int32), ("blocks", ctypes.c_int32)]

    def astuple(self) -> tuple:
        return (self.owner, self.kv_blk_begin, self.kv_blk_end, self.head_begin, self.head_end,
                self.blocks)


_VP = ctypes.c_void_p
_I32 = ctypes.c_int32
_SIGNATURES = {
    "sparsp_block_scores": [ctypes.POINTER(_Geom), _VP, _VP, _VP, _VP, _VP, _VP],
    "sparsp_topk_mask": [ctypes.POINTER(_Geom), _VP, ctypes.c_int32,
                         ctypes.POINTER(ctypes.c_int32), ctypes.c_int32, _VP, _VP, _VP],
    "sparsp_demand_union_gather": [ctypes.POINTER(_Geom), _VP, _VP, _VP, _VP, _VP, _VP, _VP,
                                   _VP, _VP, ctypes.c_int64, _VP],
    "sparsp_block_sparse_attn": [ctypes.POINTER(_Geom), _VP, _VP, ctypes.c_int32, _VP, _VP, _VP,
                                 ctypes.c_int64, ctypes.c_float, _VP, ctypes.c_int32, _VP, _VP],
    "sparsp_chunk_plan": [ctypes.POINTER(_Geom), _VP, _I32, _I32, _I32, _I32,
                          ctypes.POINTER(Chunk), _I32],
    "sparsp_block_sparse_attn_part": [ctypes.POINTER(_Geom), _VP, _VP, _I32, _VP, _VP, _VP,
                                      ctypes.c_int64, ctypes.c_float, _I32, _I32, _I32, _I32,
                                      _VP, _VP, _I32, _VP],
    "sparsp_lse_merge": [ctypes.POINTER(_Geom), _I32, _I32, _VP, _VP, _VP, _VP, _VP],
    "sparsp_chunked_attn": [ctypes.POINTER(_Geom), _VP, _VP, _I32, _VP, _VP, _VP, ctypes.c_int64,
                            ctypes.c_float, ctypes.POINTER(Chunk), _I32, _VP, _VP, _VP],
    "sparsp_periodic_placement": [_I32, _I32, _I32, _I32, _VP, _VP],
    "sparsp_cdf_mask": [ctypes.POINTER(_Geom), _VP, ctypes.c_float,
                        ctypes.POINTER(ctypes.c_int32), _I32, _VP, _VP, _VP, _VP],
    "sparsp_permute_blocks": [ctypes.POINTER(_Geom), _VP, _VP, _VP, _I32, _VP],
    "sparsp_remote_demand": [ctypes.POINTER(_Geom), _VP, ctypes.POINTER(ctypes.c_int64),
                             ctypes.POINTER(ctypes.c_int64)],
    "sparsp_pack_for_consumers": [ctypes.POINTER(_Geom), _VP, _I32, _I32, _VP, _VP, _VP, _VP, _VP,
                                  _VP, _VP, _VP, ctypes.c_int64, _VP],
    "sparsp_route_volume": [ctypes.POINTER(_Geom), _VP, _I32, _I32,
                            ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_int64),
                            ctypes.POINTER(ctypes.c_int64)],
    "sparsp_row_order": [ctypes.POINTER(_Geom), _VP, _VP, _VP],
    "sparsp_block_sparse_attn_ordered": [ctypes.POINTER(_Geom), _VP, _VP, ctypes.c_int32, _VP, _VP,
                                         _VP, ctypes.c_int64, ctypes.c_float, _VP, _VP,
                                         ctypes.c_int32, _VP, _VP],
    "sparsp_attn_workspace_bytes": [ctypes.POINTER(_Geom), _I32],
    "sparsp_block_sparse_attn_balanced": [ctypes.POINTER(_Geom), _VP, _VP, ctypes.c_int32, _VP,
                                          _VP, _VP, ctypes.c_int64, ctypes.c_float, _VP,
                                          ctypes.c_int64, _VP, ctypes.c_int32, _VP, _VP],
    "sparsp_block_sparse_attn_balanced_noalloc": [ctypes.POINTER(_Geom), _VP, _VP, ctypes.c_int32,
                                                  _VP, _VP, _VP, ctypes.c_int64, ctypes.c_float,
                                                  _VP, ctypes.c_int32, _VP, _VP],
}
_RESTYPES = {"sparsp_attn_workspace_bytes": ctypes.c_int64}


def load_library(path: Optional[str] = None) -> ctypes.CDLL:
    """Load libsparsp.so (built in-tree); raises if it is missing."""
    global _LIB
    with _LOCK:
        if _LIB is not None and path is None:
            return _LIB
        p = path or lib_path()
        if not os.path.exists(p):
            raise RuntimeError(f"{p} is not built: run `python -m paper_2609_32197_amd.build`")
        lib = ctypes.CDLL(p)
        for name, args in _SIGNATURES.items():
            fn = getattr(lib, name)
            fn.argtypes = args
            fn.restype = _RESTYPES.get(name, ctypes.c_int)
        lib.sparsp_last_error.argtypes = []
        lib.sparsp_last_error.restype = ctypes.c_char_p
        lib.sparsp_version.argtypes = []
        lib.sparsp_version.restype = ctypes.c_int
        if path is None:
            _LIB = lib
        return lib


def version() -> int:
    return load_library().sparsp_version()


def _check(rc: int):
    if rc < 0:
        msg = load_library().sparsp_last_error().decode(errors="replace")
        raise SparspError(rc, msg)


# ---------------------------------------------------------------------------
# tensor marshalling
# ---------------------------------------------------------------------------

def _torch():
    import torch
    return torch


def _elem_dtype(geom: Geometry):
    torch = _torch()
    return torch.bfloat16 if geom.dtype == BF16 else torch.float32


def _dev(t, name, dtype=None, shape=None):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on the GPU (got {t.device})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype} (got {t.dtype})")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)} (got {tuple(t.shape)})")
    return t.data_ptr()


def _stream(stream, device):
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return ctypes.c_void_p(stream.cuda_stream)


def _empty(shape, dtype, like):
    return _torch().empty(shape, dtype=dtype, device=like.device)


# ---------------------------------------------------------------------------
# the four calls
# ---------------------------------------------------------------------------

def sparsp_block_scores(geom: Geometry, Q, K, pooled_q=None, pooled_k=None, scores=None,
                        stream=None):
    """Pooled tiles and block scores. Returns (pooled_q [H,nq,d], pooled_k [H,n,d], scores [H,nq,n])."""
    torch = _torch()
    g = geom
    et = _elem_dtype(g)
    pq = pooled_q if pooled_q is not None else _empty((g.H, g.nq, g.d), torch.float32, Q)
    pk = pooled_k if pooled_k is not None else _empty((g.H, g.n, g.d), torch.float32, Q)
    sc = scores if scores is not None else _empty((g.H, g.nq, g.n), torch.float32, Q)
    args = (
        _dev(Q, "Q", et, (g.H, g.L, g.d)), _dev(K, "K", et, (g.H, g.L, g.d)),
        _dev(pq, "pooled_q", torch.float32, (g.H, g.nq, g.d)),
        _dev(pk, "pooled_k", torch.float32, (g.H, g.n, g.d)),
        _dev(sc, "scores", torch.float32, (g.H, g.nq, g.n)),
    )
    gs = g.c_struct()
    _check(load_library().sparsp_block_scores(ctypes.byref(gs), *args, _stream(stream, Q.device)))
    return pq, pk, sc


def sparsp_topk_mask(geom: Geometry, scores, keep: int, global_blocks: Sequence[int] = (),
                     mask=None, sel=None, stream=None):
    """Top-k block mask. Returns (mask uint64-as-int64 [H,nq,W], sel int32 [H,nq,keep])."""
    torch = _torch()
    g = geom
    m = mask if mask is not None else _empty((g.H, g.nq, g.W), torch.int64, scores)
    s = sel if sel is not None else _empty((g.H, g.nq, max(int(keep), 0)), torch.int32, scores)
    gb = list(int(x) for x in global_blocks)
    arr = (ctypes.c_int32 * max(1, len(gb)))(*gb)
    args = (
        _dev(scores, "scores", torch.float32, (g.H, g.nq, g.n)), ctypes.c_int32(int(keep)),
        arr if gb else None, ctypes.c_int32(len(gb)),
        _dev(m, "mask", torch.int64, (g.H, g.nq, g.W)),
        _dev(s, "sel", torch.int32, (g.H, g.nq, max(int(keep), 0))),
    )
    gs = g.c_struct()
    _check(load_library().sparsp_topk_mask(ctypes.byref(gs), *args, _stream(stream, scores.device)))
    return m, s


def sparsp_cdf_mask(geom: Geometry, scores, tau: float, global_blocks: Sequence[int] = (),
                    mask=None, sel=None, counts=None, stream=None):
    """CDF-mode block mask. Returns (mask [H,nq,W], sel int32 [H,nq,n] padded with -1,
    counts int32 [H,nq]); pass sel (its width n is the `keep`) to attention as usual."""
    torch = _torch()
    g = geom
    m = mask if mask is not None else _empty((g.H, g.nq, g.W), torch.int64, scores)
    s = sel if sel is not None else _empty((g.H, g.nq, g.n), torch.int32, scores)
    c = counts if counts is not None else _empty((g.H, g.nq), torch.int32, scores)
    gb = list(int(x) for x in global_blocks)
    arr = (ctypes.c_int32 * max(1, len(gb)))(*gb)
    args = (
        _dev(scores, "scores", torch.float32, (g.H, g.nq, g.n)), ctypes.c_float(float(tau)),
        arr if gb else None, ctypes.c_int32(len(gb)),
        _dev(m, "mask", torch.int64, (g.H, g.nq, g.W)),
        _dev(s, "sel", torch.int32, (g.H, g.nq, g.n)),
        _dev(c, "counts", torch.int32, (g.H, g.nq)),
    )
    gs = g.c_struct()
    _check(load_library().sparsp_cdf_mask(ctypes.byref(gs), *args, _stream(stream, scores.device)))
    return m, s, c


def sparsp_demand_union_gather(geom: Geometry, mask, K, V, capacity_blocks: Optional[int] = None,
                               out=None, stream=None):
    """Per-head demand and packed K/V.

    Returns a dict with demand [H,W] (uint64 bits in int64), head_off [H+1],
    slot_of [H,n], gather_blk [capacity], K_packed [capacity,block,d] and
    V_packed [capacity,d,block] (transposed blocks). ``out`` may supply
    preallocated tensors under the same keys.
    """
    torch = _torch()
    g = geom
    et = _elem_dtype(g)
    cap = int(capacity_blocks if capacity_blocks is not None else g.H * g.n)
    o = dict(out or {})
    o.setdefault("demand", _empty((g.H, g.W), torch.int64, K))
    o.setdefault("head_off", _empty((g.H + 1,), torch.int32, K))
    o.setdefault("slot_of", _empty((g.H, g.n), torch.int32, K))
    o.setdefault("gather_blk", _empty((cap,), torch.int32, K))
    o.setdefault("K_packed", _empty((cap, g.block, g.d), et, K))
    o.setdefault("V_packed", _empty((cap, g.d, g.block), et, K))
    args = (
        _dev(mask, "mask", torch.int64, (g.H, g.nq, g.W)),
        _dev(K, "K", et, (g.H, g.L, g.d)), _dev(V, "V", et, (g.H, g.L, g.d)),
        _dev(o["demand"], "demand", torch.int64, (g.H, g.W)),
        _dev(o["head_off"], "head_off", torch.int32, (g.H + 1,)),
        _dev(o["slot_of"], "slot_of", torch.int32, (g.H, g.n)),
        _dev(o["gather_blk"], "gather_blk", torch.int32),
        _dev(o["K_packed"], "K_packed", et), _dev(o["V_packed"], "V_packed", et),
    )
    if o["gather_blk"].numel() < cap or o["K_packed"].numel() < cap * g.block * g.d \
            or o["V_packed"].numel() < cap * g.block * g.d:
        raise ValueError("output buffers smaller than capacity_blocks")
    gs = g.c_struct()
    _check(load_library().sparsp_demand_union_gather(ctypes.byref(gs), *args, ctypes.c_int64(cap),
                                                    _stream(stream, K.device)))
    o["capacity_blocks"] = cap
    return o


def sparsp_block_sparse_attn(geom: Geometry, Q, sel, slot_of, K_packed, V_packed,
                             softmax_scale: Optional[float] = None, out_dtype: Optional[int] = None,
                             O=None, lse=None, want_lse: bool = True, stream=None, row_order=None,
                             workspace=None, fixed_scratch: bool = False):
    """Block-sparse attention. Returns (O [H, nq*block, d], lse [H, nq*block] or None).

    With row_order (int32 [H*nq], e.g. from sparsp_row_order) the rows are
    launched in that order (sparsp_block_sparse_attn_ordered); the outputs are
    the same bit for bit. With workspace (a device tensor, e.g. of
    sparsp_attn_workspace_bytes(geom, keep) bytes) the rows of the last round
    of workgroups are split to fill the GPU (sparsp_block_sparse_attn_balanced).
    With fixed_scratch the same split uses the library's fixed device array
    instead (sparsp_block_sparse_attn_balanced_noalloc; pass O and lse as well
    for a call that allocates nothing)."""
    torch = _torch()
    g = geom
    et = _elem_dtype(g)
    keep = int(sel.shape[-1])
    if out_dtype is None:
        out_dtype = g.dtype
    odt = torch.bfloat16 if out_dtype == BF16 else torch.float32
    if softmax_scale is None:
        softmax_scale = ctypes.c_float(1.0 / math.sqrt(g.d)).value
    o = O if O is not None else _empty((g.H, g.nq * g.block, g.d), odt, Q)
    ls = lse if lse is not None else (
        _empty((g.H, g.nq * g.block), torch.float32, Q) if want_lse else None)
    if K_packed.dim() != 3 or V_packed.dim() != 3:
        raise ValueError("K_packed and V_packed must be 3-D")
    cap = int(K_packed.shape[0])
    if tuple(K_packed.shape[1:]) != (g.block, g.d) or tuple(V_packed.shape) != (cap, g.d, g.block):
        raise ValueError("packed buffers must be [cap, block, d] and [cap, d, block]")
    args = (
        _dev(Q, "Q", et, (g.H, g.L, g.d)), _dev(sel, "sel", torch.int32, (g.H, g.nq, keep)),
        ctypes.c_int32(keep), _dev(slot_of, "slot_of", torch.int32, (g.H, g.n)),
        _dev(K_packed, "K_packed", et), _dev(V_packed, "V_packed", et), ctypes.c_int64(cap),
        ctypes.c_float(softmax_scale), _dev(o, "O", odt, (g.H, g.nq * g.block, g.d)),
        ctypes.c_int32(out_dtype),
        _dev(ls, "lse", torch.float32, (g.H, g.nq * g.block)) if ls is not None else None,
    )
    gs = g.c_struct()
    lib = load_library()
    if sum(x is not None and x is not False for x in (row_order, workspace, fixed_scratch)) > 1:
        raise ValueError("row_order, workspace and fixed_scratch cannot be combined")
    if fixed_scratch:
        _check(lib.sparsp_block_sparse_attn_balanced_noalloc(ctypes.byref(gs), *args,
                                                             _stream(stream, Q.device)))
    elif workspace is not None:
        if not workspace.is_cuda or not workspace.is_contiguous():
            raise ValueError("workspace must be a contiguous cuda tensor")
        _check(lib.sparsp_block_sparse_attn_balanced(
            ctypes.byref(gs), *args[:8], workspace.data_ptr(),
            ctypes.c_int64(workspace.numel() * workspace.element_size()), *args[8:],
            _stream(stream, Q.device)))
    elif row_order is None:
        _check(lib.sparsp_block_sparse_attn(ctypes.byref(gs), *args, _stream(stream, Q.device)))
    else:
        ro = _dev(row_order, "row_order", torch.int32, (g.H * g.nq,))
        _check(lib.sparsp_block_sparse_attn_ordered(ctypes.byref(gs), *args[:8], ro, *args[8:],
                                                    _stream(stream, Q.device)))
    return o, ls


def sparsp_attn_workspace_bytes(geom: Geometry, keep: int) -> int:
    """Workspace bytes sparsp_block_sparse_attn(..., workspace=) can use (0: none applies)."""
    gs = geom.c_struct()
    nbytes = int(load_library().sparsp_attn_workspace_bytes(ctypes.byref(gs), int(keep)))
    _check(nbytes if nbytes < 0 else 0)
    return nbytes


def sparsp_row_order(geom: Geometry, counts, order=None, stream=None):
    """Rows h*nq + r sorted by counts (int32 [H, nq]) descending, as int32 [H*nq]."""
    torch = _torch()
    g = geom
    o = order if order is not None else _empty((g.H * g.nq,), torch.int32, counts)
    gs = g.c_struct()
    _check(load_library().sparsp_row_order(ctypes.byref(gs),
                                           _dev(counts, "counts", torch.int32, (g.H, g.nq)),
                                           _dev(o, "order", torch.int32, (g.H * g.nq,)),
                                           _stream(stream, counts.device)))
    return o


# ---------------------------------------------------------------------------
# shard-by-shard attention
# ---------------------------------------------------------------------------

def sparsp_chunk_plan(geom: Geometry, demand, ranks: int, rank: int, heads_per_chunk: int,
                      tail_heads_per_chunk: int) -> list:
    """The chunk schedule of rank `rank` (host). demand: [H, W] uint64 bits (any device).

    Returns a list of Chunk structures in execution order.
    """
    import numpy as np
    g = geom
    if hasattr(demand, "detach"):
        demand = demand.detach().cpu().numpy()
    dem = np.ascontiguousarray(np.asarray(demand).view(np.uint64).reshape(g.H, g.W))
    cap = 1 + max(0, int(ranks) - 1) * g.H
    arr = (Chunk * cap)()
    gs = g.c_struct()
    rc = load_library().sparsp_chunk_plan(ctypes.byref(gs), dem.ctypes.data, int(ranks), int(rank),
                                          int(heads_per_chunk), int(tail_heads_per_chunk), arr, cap)
    _check(rc)
    return [Chunk(*arr[i].astuple()) for i in range(rc)]


def _packed_args(g, K_packed, V_packed, et):
    if K_packed.dim() != 3 or V_packed.dim() != 3:
        raise ValueError("K_packed and V_packed must be 3-D")
    cap = int(K_packed.shape[0])
    if tuple(K_packed.shape[1:]) != (g.block, g.d) or tuple(V_packed.shape) != (cap, g.d, g.block):
        raise ValueError("packed buffers must be [cap, block, d] and [cap, d, block]")
    return _dev(K_packed, "K_packed", et), _dev(V_packed, "V_packed", et), ctypes.c_int64(cap)


def _scale(g, softmax_scale):
    if softmax_scale is None:
        softmax_scale = ctypes.c_float(1.0 / math.sqrt(g.d)).value
    return ctypes.c_float(softmax_scale)


def sparsp_block_sparse_attn_part(geom: Geometry, Q, sel, slot_of, K_packed, V_packed,
                                  kv_blocks: tuple, heads: tuple,
                                  softmax_scale: Optional[float] = None, O=None, lse=None,
                                  accumulate: bool = False, stream=None):
    """Attention over the kept blocks in kv_blocks = (lo, hi) for heads = (h0, h1).

    Returns (O float32 [H, nq*block, d], lse float32 [H, nq*block]); only the
    rows of heads h0..h1-1 are touched. With accumulate, (O, lse) must be given
    and hold a running result that the part is folded into.
    """
    if accumulate and (O is None or lse is None):
        raise ValueError("accumulate needs the running (O, lse)")
    torch = _torch()
    g = geom
    et = _elem_dtype(g)
    keep = int(sel.shape[-1])
    o = O if O is not None else _empty((g.H, g.nq * g.block, g.d), torch.float32, Q)
    ls = lse if lse is not None else _empty((g.H, g.nq * g.block), torch.float32, Q)
    kp, vp, cap = _packed_args(g, K_packed, V_packed, et)
    args = (
        _dev(Q, "Q", et, (g.H, g.L, g.d)), _dev(sel, "sel", torch.int32, (g.H, g.nq, keep)),
        ctypes.c_int32(keep), _dev(slot_of, "slot_of", torch.int32, (g.H, g.n)), kp, vp, cap,
        _scale(g, softmax_scale), int(kv_blocks[0]), int(kv_blocks[1]), int(heads[0]),
        int(heads[1]), _dev(o, "O", torch.float32, (g.H, g.nq * g.block, g.d)),
        _dev(ls, "lse", torch.float32, (g.H, g.nq * g.block)), int(bool(accumulate)),
    )
    gs = g.c_struct()
    _check(load_library().sparsp_block_sparse_attn_part(ctypes.byref(gs), *args,
                                                       _stream(stream, Q.device)))
    return o, ls


def sparsp_lse_merge(geom: Geometry, heads: tuple, O_acc, lse_acc, O_part, lse_part, stream=None):
    """Folds (O_part, lse_part) into (O_acc, lse_acc) in place for heads (h0, h1)."""
    torch = _torch()
    g = geom
    so, sl = (g.H, g.nq * g.block, g.d), (g.H, g.nq * g.block)
    args = (
        int(heads[0]), int(heads[1]),
        _dev(O_acc, "O_acc", torch.float32, so), _dev(lse_acc, "lse_acc", torch.float32, sl),
        _dev(O_part, "O_part", torch.float32, so), _dev(lse_part, "lse_part", torch.float32, sl),
    )
    gs = g.c_struct()
    _check(load_library().sparsp_lse_merge(ctypes.byref(gs), *args, _stream(stream, O_acc.device)))
    return O_acc, lse_acc


def sparsp_chunked_attn(geom: Geometry, Q, sel, slot_of, K_packed, V_packed, plan: Sequence,
                        softmax_scale: Optional[float] = None, O=None, lse=None, stream=None):
    """Runs a chunk schedule (a list of Chunk or 6-tuples). Returns (O, lse), float32."""
    torch = _torch()
    g = geom
    et = _elem_dtype(g)
    keep = int(sel.shape[-1])
    so, sl = (g.H, g.nq * g.block, g.d), (g.H, g.nq * g.block)
    o = O if O is not None else _empty(so, torch.float32, Q)
    ls = lse if lse is not None else _empty(sl, torch.float32, Q)
    chunks = [c if isinstance(c, Chunk) else Chunk(*[int(x) for x in c]) for c in plan]
    arr = (Chunk * max(1, len(chunks)))(*chunks)
    kp, vp, cap = _packed_args(g, K_packed, V_packed, et)
    args = (
        _dev(Q, "Q", et, (g.H, g.L, g.d)), _dev(sel, "sel", torch.int32, (g.H, g.nq, keep)),
        ctypes.c_int32(keep), _dev(slot_of, "slot_of", torch.int32, (g.H, g.n)), kp, vp, cap,
        _scale(g, softmax_scale), arr, len(chunks),
        _dev(o, "O", torch.float32, so), _dev(ls, "lse", torch.float32, sl),
    )
    gs = g.c_struct()
    _check(load_library().sparsp_chunked_attn(ctypes.byref(gs), *args, _stream(stream, Q.device)))
    return o, ls


# ---------------------------------------------------------------------------
# dependency-aware placement
# ---------------------------------------------------------------------------

def sparsp_periodic_placement(L: int, block: int, frame_tokens: int, ranks: int) -> tuple:
    """Eq. 4's placed order (host). Returns (perm int32 [n], rank_begin int32 [ranks+1]) as numpy."""
    import numpy as np
    n = -(-int(L) // int(block))
    perm = np.empty(n, dtype=np.int32)
    begin = np.empty(int(ranks) + 1, dtype=np.int32)
    _check(load_library().sparsp_periodic_placement(int(L), int(block), int(frame_tokens),
                                                    int(ranks), perm.ctypes.data,
                                                    begin.ctypes.data))
    return perm, begin


def sparsp_permute_blocks(geom: Geometry, perm, X, Y=None, inverse: bool = False, stream=None):
    """Token blocks of X [H, L, d] into placed order (or back, with inverse). perm: int32 [n] on the GPU."""
    torch = _torch()
    g = geom
    et = _elem_dtype(g)
    y = Y if Y is not None else torch.empty_like(X)
    args = (_dev(perm, "perm", torch.int32, (g.n,)), _dev(X, "X", et, (g.H, g.L, g.d)),
            _dev(y, "Y", et, (g.H, g.L, g.d)), int(bool(inverse)))
    gs = g.c_struct()
    _check(load_library().sparsp_permute_blocks(ctypes.byref(gs), *args, _stream(stream, X.device)))
    return y


def sparsp_remote_demand(geom: Geometry, demand) -> tuple:
    """(remote blocks outside [i0, i1), all demanded blocks) from demand [H, W] (any device)."""
    import numpy as np
    g = geom
    if hasattr(demand, "detach"):
        demand = demand.detach().cpu().numpy()
    dem = np.ascontiguousarray(np.asarray(demand).view(np.uint64).reshape(g.H, g.W))
    rem, alld = ctypes.c_int64(), ctypes.c_int64()
    gs = g.c_struct()
    _check(load_library().sparsp_remote_demand(ctypes.byref(gs), dem.ctypes.data,
                                               ctypes.byref(rem), ctypes.byref(alld)))
    return rem.value, alld.value


# ---------------------------------------------------------------------------
# demand-directed routing
# ---------------------------------------------------------------------------

def sparsp_pack_for_consumers(geom: Geometry, demands, ranks: int, producer: int, K, V, out=None,
                              stream=None):
    """Producer `producer`'s packed blocks for every other rank, in ring order.

    demands: int64 (uint64 bits) [ranks, H, W] on the GPU. Returns a dict with
    provide [(R-1)*H, W], head_off [(R-1)*H+1], slot_of [(R-1)*H, n],
    gather_blk, K_packed, V_packed and capacity_blocks.
    """
    torch = _torch()
    g = geom
    et = _elem_dtype(g)
    R = int(ranks)
    nv = (R - 1) * g.H
    lo, hi = (int(producer) * g.n) // R, ((int(producer) + 1) * g.n) // R
    cap = max(1, nv * (hi - lo))
    o = dict(out or {})
    o.setdefault("provide", _empty((nv, g.W), torch.int64, K))
    o.setdefault("head_off", _empty((nv + 1,), torch.int32, K))
    o.setdefault("slot_of", _empty((nv, g.n), torch.int32, K))
    o.setdefault("gather_blk", _empty((cap,), torch.int32, K))
    o.setdefault("K_packed", _empty((cap, g.block, g.d), et, K))
    o.setdefault("V_packed", _empty((cap, g.d, g.block), et, K))
    args = (
        _dev(demands, "demands", torch.int64, (R, g.H, g.W)), R, int(producer),
        _dev(K, "K", et, (g.H, g.L, g.d)), _dev(V, "V", et, (g.H, g.L, g.d)),
        _dev(o["provide"], "provide", torch.int64, (nv, g.W)),
        _dev(o["head_off"], "head_off", torch.int32, (nv + 1,)),
        _dev(o["slot_of"], "slot_of", torch.int32, (nv, g.n)),
        _dev(o["gather_blk"], "gather_blk", torch.int32),
        _dev(o["K_packed"], "K_packed", et), _dev(o["V_packed"], "V_packed", et),
    )
    cap = min(o["gather_blk"].numel(), o["K_packed"].shape[0], o["V_packed"].shape[0])
    gs = g.c_struct()
    _check(load_library().sparsp_pack_for_consumers(ctypes.byref(gs), *args, ctypes.c_int64(cap),
                                                   _stream(stream, K.device)))
    o["capacity_blocks"] = cap
    return o


def sparsp_route_volume(geom: Geometry, demands, ranks: int, producer: int) -> dict:
    """Block-hops of the producer's shard: {'dense', 'relay', 'direct'} (demands: [R, H, W], any device)."""
    import numpy as np
    g = geom
    if hasattr(demands, "detach"):
        demands = demands.detach().cpu().numpy()
    dem = np.ascontiguousarray(np.asarray(demands).view(np.uint64).reshape(int(ranks), g.H, g.W))
    dense, relay, direct = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    gs = g.c_struct()
    _check(load_library().sparsp_route_volume(ctypes.byref(gs), dem.ctypes.data, int(ranks),
                                              int(producer), ctypes.byref(dense),
                                              ctypes.byref(relay), ctypes.byref(direct)))
    return {"dense": dense.value, "relay": relay.value, "direct": direct.value}


block_scores = sparsp_block_scores
row_order = sparsp_row_order
attn_workspace_bytes = sparsp_attn_workspace_bytes
topk_mask = sparsp_topk_mask
demand_union_gather = sparsp_demand_union_gather
block_sparse_attn = sparsp_block_sparse_attn
chunk_plan = sparsp_chunk_plan
block_sparse_attn_part = sparsp_block_sparse_attn_part
lse_merge = sparsp_lse_merge
chunked_attn = sparsp_chunked_attn
cdf_mask = sparsp_cdf_mask
periodic_placement = sparsp_periodic_placement
permute_blocks = sparsp_permute_blocks
remote_demand = sparsp_remote_demand
pack_for_consumers = sparsp_pack_for_consumers
route_volume = sparsp_route_volume
