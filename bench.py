#!/usr/bin/env python3
"""Benchmark of one rank's share of SparSP sparse attention on one MI355X.

One step is the whole per-rank hot path over one batch of synthetic input
already resident in HBM: pooled scores -> top-k mask -> demand union and
compaction -> block-sparse attention, the four calls of libsparsp.

    python bench.py [--steps K] [--warmup W] [--workload wan-share]

Prints ONE JSON line on stdout. `value` is the whole step's throughput in
TFLOP/s of algorithmic attention work over the kept (unmasked) tiles,
4 * d * c_i * c_j FLOPs per kept (query block i, KV block j) pair with c the
valid token counts; `ms_per_step` is the layer time. The `roofline` object
is for the dominant kernel (attention), timed with HIP events on the stream
it runs on. `cpu_baseline` is the float64 oracle timed on a bounded sample of
the same workload on the host cores.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "block-sparse attn ms/layer + TFLOP/s on unmasked tiles (% MFMA peak), 1 GPU"
PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3    # MI355X fp32 (vector / matrix)
PEAK_HBM_GBPS = 8000.0     # MI355X HBM3E
ATTN_SRC = os.path.join(ROOT, "paper_2609_32197_amd", "csrc", "attn_bf16.hip")
COUNTERS = os.path.join(ROOT, "profiles", "attn_bf16_wan-share_counters.md")


def parse_args(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="wan-share")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="wall-clock budget of the oracle sample")
    ap.add_argument("--cache-dir", default=None,
                    help="keep generated inputs as .npy files here and reuse them")
    ap.add_argument("--chunk-heads", type=int, default=8,
                    help="heads per chunk of a remote shard (shard-by-shard attention)")
    ap.add_argument("--tail-chunk-heads", type=int, default=2,
                    help="heads per chunk of the last remote shard")
    ap.add_argument("--no-flush", action="store_true",
                    help="do not overwrite a 512 MiB buffer between steps (it evicts the "
                         "Infinity Cache and L2 so each step starts cold)")
    ap.add_argument("--extensions", action="store_true",
                    help="also measure shard-by-shard attention, CDF selection, routing and placement")
    ap.add_argument("--unit-probes", action="store_true",
                    help="also measure the exponential, FMA and 16-byte LDS read issue rates "
                         "against the register-only MFMA rate")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of this many MiB (for counter calibration)")
    return ap.parse_args(argv)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def copy_calibration(mib: int):
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    log(f"copied {mib} MiB x 5")


def load_inputs(wl, seed, cache_dir, make_qkv):
    """Generate the workload's inputs, or reuse a copy saved by an earlier run."""
    import numpy as np
    if cache_dir:
        paths = [os.path.join(cache_dir, f"{wl.config_id}_{seed}_{t}.npy") for t in "qkv"]
        if all(os.path.exists(p) for p in paths):
            return tuple(np.load(p) for p in paths)
    q, k, v = make_qkv(wl, seed=seed)
    if cache_dir:
        os.makedirs(cache_dir, exist_ok=True)
        for p, x in zip(paths, (q, k, v)):
            np.save(p, x)
    return q, k, v


def code_sha(path):
    """sha256[:16] of a HIP source with its comments and blank lines removed: the
    counters stay valid across comment edits and are dropped on any code change."""
    with open(path) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    lines = [line.rstrip() for line in text.splitlines() if line.strip()]
    return hashlib.sha256("\n".join(lines).encode()).hexdigest()[:16]


def read_traffic():
    """HBM bytes per attention launch from the committed counter summary, if current."""
    if not os.path.exists(COUNTERS):
        return None, "no counter summary"
    text = open(COUNTERS).read()
    m_sha = re.search(r"code sha256\[:16\][^`]*`([0-9a-f]{16})`", text)
    m_b = re.search(r"HBM bytes per launch \(calibrated\):\s*([0-9.eE+]+)", text)
    if not m_sha or not m_b:
        return None, "counter summary unreadable"
    if m_sha.group(1) != code_sha(ATTN_SRC):
        return None, "kernel changed since the counters were taken"
    return float(m_b.group(1)), "ok"


def measured_peaks(sp, torch, copy_bytes: int, stream):
    """Practical ceilings on this part, beside the data-sheet peaks: the bf16
    MFMA rate with register operands (the benchmark's probe kernel in
    paper_2609_32197_amd.probe, outside libsparsp; best of three ~20 ms
    launches) and a plain device-to-device copy of copy_bytes
    (read + write, mean of five)."""
    wgs, iters = 1024, 60000
    sink = torch.empty(wgs * 256, dtype=torch.float32, device="cuda")
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    from paper_2609_32197_amd import probe
    probe.run(1000, wgs, sink, stream=stream)
    best = 0.0
    for _ in range(3):
        e0.record(stream)
        probe.run(iters, wgs, sink, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        best = max(best, wgs * iters * 524288 / (e0.elapsed_time(e1) * 1e-3) / 1e12)
    del sink
    n = max(1, copy_bytes // 2)
    src = torch.empty(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    with torch.cuda.stream(stream):
        dst.copy_(src)
        e0.record(stream)
        for _ in range(5):
            dst.copy_(src)
        e1.record(stream)
    torch.cuda.synchronize()
    copy_gbps = 2 * n * 5 / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del src, dst
    return best, copy_gbps


def measure_unit_probes(torch, stream, mfma_tflops: float, cus: int):
    """Issue rates the attention kernel's softmax and operand reads depend on,
    each best of three launches of its probe kernel (paper_2609_32197_amd.probe),
    expressed per SIMD (per CU for LDS) and per matrix-core slot: the time one
    v_mfma_f32_32x32x16_bf16 takes on a SIMD at the register-only MFMA rate of
    the same process (32 cycles at that clock). The probes draw less power than
    the MFMA probe, so their clock can run higher: the per-slot figures are
    upper bounds for work that shares the SIMD with MFMAs."""
    from paper_2609_32197_amd import probe
    simds = 4 * cus
    mfma_per_simd_s = mfma_tflops * 1e12 / 32768 / simds
    out = {"mfma_tflops": mfma_tflops, "mfma_per_simd_per_s": mfma_per_simd_s}
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for kind, wgs, iters in (("exp", 8 * cus, 4000), ("fma", 8 * cus, 20000), ("lds", 2 * cus, 4000)):
        sink = torch.empty(wgs * 256, dtype=torch.float32, device="cuda")
        probe.run_unit(kind, 10, wgs, sink, stream=stream)
        best = float("inf")
        for _ in range(3):
            e0.record(stream)
            probe.run_unit(kind, iters, wgs, sink, stream=stream)
            e1.record(stream)
            torch.cuda.synchronize()
            best = min(best, e0.elapsed_time(e1) * 1e-3)
        if kind == "lds":
            per_cu_s = wgs * 4 * iters * 32 * 1024 / best / cus  # bytes per CU per second
            out["lds"] = {"bytes_per_cu_per_s": per_cu_s,
                          "bytes_per_cu_per_mfma_slot": per_cu_s / mfma_per_simd_s,
                          "bytes_per_cycle_per_cu": per_cu_s / mfma_per_simd_s / 32,
                          "workgroups": wgs, "seconds": best}
        else:
            per_simd_s = wgs * 4 * iters * 16 / best / simds  # wave instructions per SIMD per second
            out[kind] = {"wave_instr_per_simd_per_s": per_simd_s,
                         "per_mfma_slot": per_simd_s / mfma_per_simd_s,
                         "cycles_per_wave_instr": 32 * mfma_per_simd_s / per_simd_s,
                         "workgroups": wgs, "seconds": best}
        del sink
    return out


def attention_flops(sel, L, block, i0, d):
    import numpy as np
    n = -(-L // block)
    c = np.minimum(block, L - block * np.arange(n)).astype(np.int64)
    H, nq, keep = sel.shape
    kv = c[sel].sum(axis=2)                       # valid keys per row
    ci = c[i0:i0 + nq]
    return int(4 * d * (kv * ci[None, :]).sum())


def attention_flops_sel(sel, L, block, i0, d):
    """attention_flops for a sel padded with -1 (CDF mode): padded entries count nothing."""
    import numpy as np
    n = -(-L // block)
    c = np.minimum(block, L - block * np.arange(n)).astype(np.int64)
    c_pad = np.concatenate([c, [0]])
    H, nq, _ = sel.shape
    kv = c_pad[np.where(sel >= 0, sel, n)].sum(axis=2)
    ci = c[i0:i0 + nq]
    return int(4 * d * (kv * ci[None, :]).sum())


def gather_bytes(slot_of, L, block, d, w):
    """Algorithmic bytes of the compaction: read valid K and V rows, write whole packed blocks."""
    import numpy as np
    n = -(-L // block)
    c = np.minimum(block, L - block * np.arange(n)).astype(np.int64)
    dem = slot_of >= 0
    reads = int((dem * c[None, :]).sum()) * 2 * d * w
    writes = int(dem.sum()) * 2 * block * d * w
    return reads + writes + slot_of.size * 4


def cpu_baseline(wl, q, k, v, budget_s):
    """Time the float64 oracle over whole heads of the same workload until the budget is spent."""
    import numpy as np
    import oracle as orc
    blas = "unknown"
    try:
        from threadpoolctl import threadpool_info
        pools = [p for p in threadpool_info() if p.get("user_api") == "blas"]
        threads = max([p.get("num_threads", 1) for p in pools] or [1])
        if pools:
            blas = ", ".join(f"{p.get('internal_api')} {p.get('version')} "
                             f"({p.get('num_threads')} threads)" for p in pools)
    except Exception:  # threadpoolctl missing: numpy's default pool
        threads = os.cpu_count() or 1
    flops = 0
    spent = 0.0
    heads = 0
    for h in range(wl.H):
        t0 = time.perf_counter()
        Qh, Kh, Vh = (orc.decode_input(x[h:h + 1], wl.dtype) for x in (q, k, v))
        pq = orc.pool_blocks(Qh, wl.L, wl.block, range(wl.i0, wl.i1))
        pk = orc.pool_blocks(Kh, wl.L, wl.block)
        s = orc.block_scores(pq, pk, wl.d)
        mask, _ = orc.select_topk(s, wl.keep, wl.i0, wl.global_blocks)
        D = orc.demand_union(mask)
        head_off, gather_blk, _ = orc.packing_plan(D)
        orc.pack_kv(k[h:h + 1], v[h:h + 1], head_off, gather_blk, wl.L, wl.block)
        orc.sparse_attention(Qh, Kh, Vh, mask, wl.L, wl.block, wl.i0, wl.softmax_scale)
        spent += time.perf_counter() - t0
        flops += orc.attention_flops(mask, wl.L, wl.block, wl.i0, wl.d)
        heads += 1
        if spent >= budget_s:
            break
    return {
        "value": flops / spent / 1e12,
        "unit": "TFLOP/s",
        "cores": int(threads),
        "host_cpu_count": os.cpu_count(),
        "host_cpus_usable": len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else None,
        "blas": blas,
        "kind": "oracle",
        "sample": f"{heads} of {wl.H} heads, whole pipeline (pool, score, select, union, pack, "
                  f"attend) per head, {spent:.1f} s",
    }


def time_calls(fn, reps, stream):
    """Mean milliseconds of fn() over reps calls, HIP events on `stream`, after one warm call."""
    import torch
    fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def measure_chunked(sp, g, wl, Q, bufs, packed, stream, a):
    """Shard-by-shard attention of this rank (Section 2.3, Section 7): the chunk
    schedule run with sparsp_chunked_attn against one unchunked call with the
    same float32 output, and the log-sum-exp merge on its own over every head."""
    import torch
    plan = sp.sparsp_chunk_plan(g, packed["demand"], wl.ranks, wl.rank, a.chunk_heads,
                                a.tail_chunk_heads)
    f32 = torch.float32
    so, sl = (wl.H, wl.nq * wl.block, wl.d), (wl.H, wl.nq * wl.block)
    O, lse, Op, lp = (torch.empty(x, dtype=f32, device="cuda") for x in (so, sl, so, sl))
    reps = 5

    def chunked():
        sp.sparsp_chunked_attn(g, Q, bufs["sel"], packed["slot_of"], packed["K_packed"],
                               packed["V_packed"], plan, wl.softmax_scale, O=O, lse=lse,
                               stream=stream)

    def whole():
        sp.sparsp_block_sparse_attn(g, Q, bufs["sel"], packed["slot_of"], packed["K_packed"],
                                    packed["V_packed"], wl.softmax_scale, out_dtype=sp.F32, O=Op,
                                    lse=lp, stream=stream)

    def merge():
        sp.sparsp_lse_merge(g, (0, wl.H), O, lse, Op, lp, stream=stream)

    c0 = plan[0]

    def local():
        sp.sparsp_block_sparse_attn_part(g, Q, bufs["sel"], packed["slot_of"], packed["K_packed"],
                                         packed["V_packed"], (c0.kv_blk_begin, c0.kv_blk_end),
                                         (c0.head_begin, c0.head_end), wl.softmax_scale, O=Op,
                                         lse=lp, stream=stream)

    t_chunked = time_calls(chunked, reps, stream)
    t_local = time_calls(local, reps, stream)
    t_whole = time_calls(whole, reps, stream)
    t_merge = time_calls(merge, reps, stream)
    rows = wl.H * wl.nq * wl.block
    mbytes = rows * (12 * wl.d + 12)  # read both O and lse, write the accumulator
    return {
        "ranks": wl.ranks, "rank": wl.rank, "heads_per_chunk": a.chunk_heads,
        "tail_heads_per_chunk": a.tail_chunk_heads, "chunks": len(plan),
        "chunked_ms": t_chunked, "local_shard_ms": t_local,
        "remote_chunks_ms": t_chunked - t_local, "unchunked_f32_out_ms": t_whole,
        "overhead_frac": t_chunked / t_whole - 1.0,
        "merge": {"rows": rows, "ms": t_merge, "algorithmic_bytes": mbytes,
                  "GBps": mbytes / (t_merge * 1e-3) / 1e9,
                  "frac_of_hbm_peak": mbytes / (t_merge * 1e-3) / 1e9 / PEAK_HBM_GBPS},
    }


def measure_placement(sp, g, wl, Q, K, V, bufs, packed, stream, ranks_list=(4, 8)):
    """Dependency-aware placement (Section 4.3, Eq. 4) against contiguous slices.

    For each R, every rank r runs scores, top-k and demand over its own query
    blocks, with the tensors in logical order (contiguous slices) or in Eq. 4's
    placed order; the sums over ranks of the demanded blocks (sum of U_h) and
    of Eq. 3's remote blocks are reported, with the largest V_r in bytes. The
    block permutation kernel is timed on Q.
    """
    import torch
    T, Hy, W = wl.latent
    F = Hy * W
    b, d, w = wl.block, wl.d, wl.bytes_per_elem
    Qp, Kp = torch.empty_like(Q), torch.empty_like(K)
    res = {"frame_tokens": F}

    def rank_stats(Qx, Kx, begin):
        demanded, remote, worst = 0, 0, 0
        for r in range(len(begin) - 1):
            gr = sp.Geometry(wl.H, wl.L, wl.d, wl.block, int(begin[r]), int(begin[r + 1]), g.dtype)
            _, _, sc = sp.sparsp_block_scores(gr, Qx, Kx, stream=stream)
            m, _ = sp.sparsp_topk_mask(gr, sc, wl.keep, wl.global_blocks, stream=stream)
            sp.sparsp_demand_union_gather(gr, m, Kx, Kx, wl.H * wl.n, out=packed, stream=stream)
            rem, tot = sp.sparsp_remote_demand(gr, packed["demand"])
            demanded += tot
            remote += rem
            worst = max(worst, rem)
        return {"demanded_blocks": demanded, "remote_blocks": remote,
                "max_rank_remote_blocks": worst, "max_rank_V_bytes": 2 * b * d * w * worst,
                "total_V_bytes": 2 * b * d * w * remote}

    for R in ranks_list:
        if R > wl.n:
            continue
        contiguous = [(p * wl.n) // R for p in range(R + 1)]
        perm, begin = sp.sparsp_periodic_placement(wl.L, b, F, R)
        pd = torch.from_numpy(perm).cuda()
        sp.sparsp_permute_blocks(g, pd, Q, Qp, stream=stream)
        sp.sparsp_permute_blocks(g, pd, K, Kp, stream=stream)
        c = rank_stats(Q, K, contiguous)
        pr = rank_stats(Qp, Kp, begin)
        res[f"R{R}"] = {
            "contiguous": c, "periodic": pr,
            "remote_reduction": 1.0 - pr["remote_blocks"] / max(1, c["remote_blocks"]),
            "demand_reduction": 1.0 - pr["demanded_blocks"] / max(1, c["demanded_blocks"]),
            "periodic_rank_blocks": [int(begin[p + 1] - begin[p]) for p in range(R)],
        }
        if "permute" not in res:
            ms = time_calls(lambda: sp.sparsp_permute_blocks(g, pd, Q, Qp, stream=stream), 5, stream)
            nbytes = 2 * wl.H * wl.L * wl.d * w
            res["permute"] = {"ms": ms, "bytes": nbytes, "GBps": nbytes / (ms * 1e-3) / 1e9,
                              "frac_of_hbm_peak": nbytes / (ms * 1e-3) / 1e9 / PEAK_HBM_GBPS}
    del Qp, Kp
    return res


def measure_cdf(sp, g, wl, Q, bufs, packed, stream, taus=(0.85, 0.9, 0.95)):
    """CDF-mode selection (Section 8.1) in place of top-k: the mask kernel's time, the
    kept blocks per row, and the layer with that selection (scores, CDF mask, demand
    and gather, attention over the n-wide padded sel)."""
    import numpy as np
    import torch
    res = {}
    K = packed["_K"]
    V = packed["_V"]
    for tau in taus:
        m, sel, cnt = sp.sparsp_cdf_mask(g, bufs["scores"], tau, wl.global_blocks, stream=stream)
        t_mask = time_calls(lambda: sp.sparsp_cdf_mask(g, bufs["scores"], tau, wl.global_blocks,
                                                       mask=m, sel=sel, counts=cnt, stream=stream),
                            5, stream)
        c = cnt.cpu().numpy()
        O = torch.empty((wl.H, wl.nq * wl.block, wl.d), dtype=Q.dtype, device="cuda")
        cap = wl.H * wl.n

        def layer():
            sp.sparsp_block_scores(g, Q, K, bufs["pooled_q"], bufs["pooled_k"], bufs["scores"],
                                   stream=stream)
            sp.sparsp_cdf_mask(g, bufs["scores"], tau, wl.global_blocks, mask=m, sel=sel,
                               counts=cnt, stream=stream)
            sp.sparsp_demand_union_gather(g, m, K, V, cap, out=packed, stream=stream)
            sp.sparsp_block_sparse_attn(g, Q, sel, packed["slot_of"], packed["K_packed"],
                                        packed["V_packed"], wl.softmax_scale, O=O, lse=bufs["lse"],
                                        stream=stream)

        order = torch.empty((wl.H * wl.nq,), dtype=torch.int32, device="cuda")

        def layer_longest_first():
            sp.sparsp_block_scores(g, Q, K, bufs["pooled_q"], bufs["pooled_k"], bufs["scores"],
                                   stream=stream)
            sp.sparsp_cdf_mask(g, bufs["scores"], tau, wl.global_blocks, mask=m, sel=sel,
                               counts=cnt, stream=stream)
            sp.sparsp_demand_union_gather(g, m, K, V, cap, out=packed, stream=stream)
            sp.sparsp_row_order(g, cnt, order=order, stream=stream)
            sp.sparsp_block_sparse_attn(g, Q, sel, packed["slot_of"], packed["K_packed"],
                                        packed["V_packed"], wl.softmax_scale, O=O, lse=bufs["lse"],
                                        stream=stream, row_order=order)

        t_layer = time_calls(layer, 3, stream)
        t_layer_lf = time_calls(layer_longest_first, 3, stream)
        attn = lambda ro: sp.sparsp_block_sparse_attn(
            g, Q, sel, packed["slot_of"], packed["K_packed"], packed["V_packed"], wl.softmax_scale,
            O=O, lse=bufs["lse"], stream=stream, row_order=ro)
        t_attn = time_calls(lambda: attn(None), 3, stream)
        t_attn_lf = time_calls(lambda: attn(order), 3, stream)
        flops = attention_flops_sel(sel.cpu().numpy(), wl.L, wl.block, wl.i0, wl.d)
        res[str(tau)] = {"mask_ms": t_mask, "mean_kept_blocks": float(c.mean()),
                         "min_kept_blocks": int(c.min()), "max_kept_blocks": int(c.max()),
                         "kept_fraction": float(c.mean()) / wl.n, "layer_ms": t_layer,
                         "attention_tflop": flops / 1e12,
                         "layer_tflops": flops / (t_layer * 1e-3) / 1e12,
                         "attention_ms": t_attn, "attention_tflops": flops / (t_attn * 1e-3) / 1e12,
                         "layer_ms_longest_first": t_layer_lf,
                         "layer_tflops_longest_first": flops / (t_layer_lf * 1e-3) / 1e12,
                         "attention_ms_longest_first": t_attn_lf,
                         "attention_tflops_longest_first": flops / (t_attn_lf * 1e-3) / 1e12}
    return res


def measure_routing(sp, g, wl, Q, K, V, packed, stream):
    """Demand-directed routing (Section 5) at the workload's rank count R: every
    rank's demand from its own query blocks (contiguous slices), then for each
    producer the per-consumer packing (sparsp_pack_for_consumers: timed, with its
    algorithmic bytes) and the dense-ring / relay / direct block-hop counts."""
    import numpy as np
    import torch
    R = wl.ranks
    dems = []
    for c in range(R):
        gr = sp.Geometry(wl.H, wl.L, wl.d, wl.block, (c * wl.n) // R, ((c + 1) * wl.n) // R,
                         g.dtype)
        _, _, sc = sp.sparsp_block_scores(gr, Q, K, stream=stream)
        m, _ = sp.sparsp_topk_mask(gr, sc, wl.keep, wl.global_blocks, stream=stream)
        sp.sparsp_demand_union_gather(gr, m, K, V, wl.H * wl.n, out=packed, stream=stream)
        dems.append(packed["demand"].clone())
    D = torch.stack(dems)
    c_valid = np.minimum(wl.block, wl.L - wl.block * np.arange(wl.n)).astype(np.int64)
    row = wl.d * wl.bytes_per_elem
    per = []
    for p in range(R):
        out = sp.sparsp_pack_for_consumers(g, D, R, p, K, V, stream=stream)
        ms = time_calls(lambda: sp.sparsp_pack_for_consumers(g, D, R, p, K, V, out=out,
                                                             stream=stream), 3, stream)
        S = int(out["head_off"][-1].item())
        blk = out["gather_blk"][:S].cpu().numpy()
        nbytes = int(2 * row * c_valid[blk].sum() + 2 * S * wl.block * row)
        vol = sp.sparsp_route_volume(g, D, R, p)
        per.append({"producer": p, "slots": S, "pack_ms": ms, "bytes": nbytes,
                    "GBps": nbytes / (ms * 1e-3) / 1e9, **vol})
        del out
    blk_bytes = 2 * wl.block * wl.d * wl.bytes_per_elem  # K and V of one block
    tot = {k: sum(x[k] for x in per) for k in ("dense", "relay", "direct")}
    return {"ranks": R, "producers": per,
            "block_hops": tot,
            "bytes": {k: v * blk_bytes for k, v in tot.items()},
            "relay_over_direct": tot["relay"] / max(1, tot["direct"]),
            "dense_over_direct": tot["dense"] / max(1, tot["direct"])}


def main(argv=None) -> int:
    a = parse_args(argv)
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if a.gpus != 1 or world != 1:
        print(json.dumps({"error": "this benchmark runs one rank's share on ONE GPU; "
                                   f"--gpus {a.gpus} (WORLD_SIZE={world}) is not supported",
                          "n_gpus": a.gpus}))
        return 2

    import numpy as np
    import torch

    if a.copy_calibration:
        copy_calibration(a.copy_calibration)
        return 0

    import paper_2609_32197_amd as sp
    from workloads import get_workload, make_qkv

    wl = get_workload(a.workload)
    t0 = time.time()
    q, k, v = load_inputs(wl, a.seed, a.cache_dir, make_qkv)
    log(f"[bench] {wl.name} inputs ready in {time.time() - t0:.1f}s")

    def dev(x):
        if wl.dtype == "bf16":
            return torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(x).cuda()

    Q, K, V = dev(q), dev(k), dev(v)
    g = sp.Geometry(wl.H, wl.L, wl.d, wl.block, wl.i0, wl.i1,
                    sp.BF16 if wl.dtype == "bf16" else sp.F32)
    f32, i32, i64 = torch.float32, torch.int32, torch.int64
    cap = wl.H * wl.n
    et = Q.dtype
    bufs = dict(
        pooled_q=torch.empty((wl.H, wl.nq, wl.d), dtype=f32, device="cuda"),
        pooled_k=torch.empty((wl.H, wl.n, wl.d), dtype=f32, device="cuda"),
        scores=torch.empty((wl.H, wl.nq, wl.n), dtype=f32, device="cuda"),
        mask=torch.empty((wl.H, wl.nq, g.W), dtype=i64, device="cuda"),
        sel=torch.empty((wl.H, wl.nq, wl.keep), dtype=i32, device="cuda"),
        O=torch.empty((wl.H, wl.nq * wl.block, wl.d), dtype=et, device="cuda"),
        lse=torch.empty((wl.H, wl.nq * wl.block), dtype=f32, device="cuda"),
    )
    packed = dict(
        demand=torch.empty((wl.H, g.W), dtype=i64, device="cuda"),
        head_off=torch.empty((wl.H + 1,), dtype=i32, device="cuda"),
        slot_of=torch.empty((wl.H, wl.n), dtype=i32, device="cuda"),
        gather_blk=torch.empty((cap,), dtype=i32, device="cuda"),
        K_packed=torch.empty((cap, wl.block, wl.d), dtype=et, device="cuda"),
        V_packed=torch.empty((cap, wl.d, wl.block), dtype=et, device="cuda"),
    )
    out_dtype = sp.BF16 if wl.dtype == "bf16" else sp.F32
    stream = torch.cuda.current_stream()
    # Workspace that lets the attention call split the rows of its last, partial
    # round of workgroups (sparsp_block_sparse_attn_balanced); empty for float32.
    ws_bytes = sp.sparsp_attn_workspace_bytes(g, wl.keep)
    attn_ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda") if ws_bytes > 0 else None

    def step(ev=None):
        if ev: ev[0].record(stream)
        sp.sparsp_block_scores(g, Q, K, bufs["pooled_q"], bufs["pooled_k"], bufs["scores"],
                               stream=stream)
        if ev: ev[1].record(stream)
        sp.sparsp_topk_mask(g, bufs["scores"], wl.keep, wl.global_blocks, bufs["mask"],
                            bufs["sel"], stream=stream)
        if ev: ev[2].record(stream)
        sp.sparsp_demand_union_gather(g, bufs["mask"], K, V, cap, out=packed, stream=stream)
        if ev: ev[3].record(stream)
        sp.sparsp_block_sparse_attn(g, Q, bufs["sel"], packed["slot_of"], packed["K_packed"],
                                    packed["V_packed"], wl.softmax_scale, out_dtype=out_dtype,
                                    O=bufs["O"], lse=bufs["lse"], stream=stream,
                                    workspace=attn_ws)
        if ev: ev[4].record(stream)

    # Between steps a 512 MiB buffer is overwritten on the same stream, so every
    # step starts with the Infinity Cache (256 MB) and the L2s holding none of
    # its inputs. The overwrite lies outside the stage events.
    flush = None if a.no_flush else torch.empty(512 << 20, dtype=torch.uint8, device="cuda")

    def cold():
        if flush is not None:
            flush.fill_(0x5A)

    for _ in range(a.warmup):
        cold()
        step()
    torch.cuda.synchronize()

    # Timed region: K steps, per-stage HIP events on the same stream.
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(a.steps)]
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    for s in range(a.steps):
        cold()
        step(evs[s])
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t_wall) * 1e3 / a.steps
    stage_names = ["block_scores", "topk_mask", "demand_union_gather", "block_sparse_attn"]
    stage_ms = {nm: float(np.mean([evs[s][i].elapsed_time(evs[s][i + 1]) for s in range(a.steps)]))
                for i, nm in enumerate(stage_names)}
    ms_per_step = float(np.mean([evs[s][0].elapsed_time(evs[s][4]) for s in range(a.steps)]))
    stage_ms_median = {
        nm: float(np.median([evs[s][i].elapsed_time(evs[s][i + 1]) for s in range(a.steps)]))
        for i, nm in enumerate(stage_names)}

    sel = bufs["sel"].cpu().numpy()
    slot_of = packed["slot_of"].cpu().numpy()
    flops = attention_flops(sel, wl.L, wl.block, wl.i0, wl.d)
    gbytes = gather_bytes(slot_of, wl.L, wl.block, wl.d, wl.bytes_per_elem)
    attn_tflops = flops / (stage_ms["block_sparse_attn"] * 1e-3) / 1e12
    peak = PEAK_BF16_TFLOPS if wl.dtype == "bf16" else PEAK_F32_TFLOPS
    demanded = int((slot_of >= 0).sum())
    traffic, traffic_note = read_traffic() if wl.name == "wan-share" else (None, "other workload")
    mfma_meas, copy_meas = measured_peaks(sp, torch, gbytes, stream)
    unit = None
    if a.unit_probes:
        cus = torch.cuda.get_device_properties(0).multi_processor_count
        unit = measure_unit_probes(torch, stream, mfma_meas, cus)

    rec = {
        "metric": METRIC,
        "value": flops / (ms_per_step * 1e-3) / 1e12,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic (seeded generator standing in for the paper's video-DiT activations)",
        "config": {
            "workload": wl.name, "H": wl.H, "d": wl.d, "block": wl.block, "L": wl.L,
            "n_blocks": wl.n, "local_blocks": [wl.i0, wl.i1], "keep": wl.keep,
            "global_blocks": len(wl.global_blocks), "seed": a.seed,
        },
        "stages_ms": stage_ms,
        "stages_statistic": "mean over the timed steps of HIP events recorded on the calls' stream",
        "stages_ms_median": stage_ms_median,
        "wall_ms_per_step": wall_ms,
        "cache_flushed_between_steps": flush is not None,
        "attention": {
            "call": "sparsp_block_sparse_attn_balanced" if attn_ws is not None
                    else "sparsp_block_sparse_attn",
            "algorithmic_tflop": flops / 1e12,
            "kernel_ms": stage_ms["block_sparse_attn"],
            "tflops": attn_tflops,
            "frac_of_mfma_peak": attn_tflops / peak if wl.dtype == "bf16" else None,
            "frac_of_fp32_peak": attn_tflops / peak if wl.dtype != "bf16" else None,
            "measured_mfma_peak_tflops": mfma_meas,
            "frac_of_measured_mfma_peak": attn_tflops / mfma_meas if wl.dtype == "bf16" else None,
        },
        "gather": {
            "demanded_blocks": demanded,
            "union_fraction": demanded / (wl.H * wl.n),
            "algorithmic_bytes": gbytes,
            "call_ms": stage_ms["demand_union_gather"],
            "GBps": gbytes / (stage_ms["demand_union_gather"] * 1e-3) / 1e9,
            "frac_of_hbm_peak": gbytes / (stage_ms["demand_union_gather"] * 1e-3) / 1e9 / PEAK_HBM_GBPS,
            "measured_copy_GBps": copy_meas,
            "frac_of_measured_copy": gbytes / (stage_ms["demand_union_gather"] * 1e-3) / 1e9 / copy_meas,
        },
        "roofline": {
            # the float32 path runs vector FMAs, not the matrix cores
            "bound": "mfma" if wl.dtype == "bf16" else "alu",
            "achieved": attn_tflops,
            "peak": peak,
            "unit": "TFLOP/s",
            "frac": attn_tflops / peak,
            "traffic": traffic,
            "traffic_note": traffic_note,
        },
        "cpu_baseline": None,
    }
    if unit is not None:
        rec["unit_probes"] = unit
    if a.extensions and wl.ranks > 1:
        rec["chunked_attention"] = measure_chunked(sp, g, wl, Q, bufs, packed, stream, a)
        c = rec["chunked_attention"]
        log(f"[bench] shard-by-shard: {c['chunks']} chunks {c['chunked_ms']:.3f} ms vs "
            f"{c['unchunked_f32_out_ms']:.3f} ms unchunked; merge {c['merge']['GBps']:.0f} GB/s")
    if a.extensions and flush is not None:
        # The gather call alone right after the cache flush, so that none of
        # K and V can come from the Infinity Cache or the L2s (in the step,
        # pooling has just streamed K).
        gms = []
        for _ in range(10):
            cold()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            sp.sparsp_demand_union_gather(g, bufs["mask"], K, V, cap, out=packed, stream=stream)
            e1.record(stream)
            torch.cuda.synchronize()
            gms.append(e0.elapsed_time(e1))
        g_ms = float(np.median(gms))
        rec["gather_cold"] = {"call_ms_median": g_ms, "GBps": gbytes / (g_ms * 1e-3) / 1e9,
                              "frac_of_hbm_peak": gbytes / (g_ms * 1e-3) / 1e9 / PEAK_HBM_GBPS}
        log(f"[bench] gather alone after a cache flush: {g_ms:.4f} ms = "
            f"{rec['gather_cold']['GBps']:.0f} GB/s")
    if a.extensions and wl.dtype == "bf16":
        packed["_K"], packed["_V"] = K, V
        rec["cdf_selection"] = measure_cdf(sp, g, wl, Q, bufs, packed, stream)
        del packed["_K"], packed["_V"]
        for tau, res in rec["cdf_selection"].items():
            log(f"[bench] CDF tau={tau}: {res['mean_kept_blocks']:.1f} blocks/row, mask "
                f"{res['mask_ms']:.3f} ms, layer {res['layer_ms']:.3f} ms ({res['layer_tflops']:.0f} TFLOP/s), "
                f"attention {res['attention_ms']:.3f} ms; longest-first: layer "
                f"{res['layer_ms_longest_first']:.3f} ms, attention {res['attention_ms_longest_first']:.3f} ms "
                f"({res['attention_tflops_longest_first']:.0f} TFLOP/s)")
    if a.extensions and wl.ranks > 1:
        # (reuses the step's packed buffers: after the measurements that read them)
        rec["routing"] = measure_routing(sp, g, wl, Q, K, V, packed, stream)
        rt = rec["routing"]
        log(f"[bench] routing R={rt['ranks']}: block-hops dense {rt['block_hops']['dense']} relay "
            f"{rt['block_hops']['relay']} direct {rt['block_hops']['direct']}; pack "
            f"{np.mean([x['GBps'] for x in rt['producers']]):.0f} GB/s")
    if a.extensions and wl.ranks > 1 and not wl.global_blocks:
        # (reuses the step's packed buffers: runs last)
        rec["placement"] = measure_placement(sp, g, wl, Q, K, V, bufs, packed, stream)
        for key, val in rec["placement"].items():
            if key.startswith("R"):
                log(f"[bench] placement {key}: remote blocks contiguous "
                    f"{val['contiguous']['remote_blocks']} -> periodic {val['periodic']['remote_blocks']}"
                    f" ({-100 * val['remote_reduction']:+.1f}%)")
    log(f"[bench] {wl.name}: {ms_per_step:.3f} ms/layer, attention {stage_ms['block_sparse_attn']:.3f} ms "
        f"= {attn_tflops:.0f} TFLOP/s ({100 * attn_tflops / peak:.1f}% of peak, "
        f"{100 * attn_tflops / mfma_meas:.1f}% of the measured {mfma_meas:.0f}), gather "
        f"{rec['gather']['GBps']:.0f} GB/s (copy {copy_meas:.0f}), stages {stage_ms}")
    if not a.no_cpu_baseline:
        del Q, K, V, bufs, packed
        torch.cuda.empty_cache()
        log(f"[bench] timing the oracle on the host for ~{a.cpu_seconds:.0f}s")
        rec["cpu_baseline"] = cpu_baseline(wl, q, k, v, a.cpu_seconds)
    print(json.dumps(rec), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
