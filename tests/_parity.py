"""Shared plumbing of the GPU parity tests: inputs to the device, oracle runs
on the same bits, and the comparisons with their tolerances.

Tolerances (the floating-point parts):

* block scores: the GPU sums in float32, the oracle in float64 (u = 2^-24).
  A pooled value is a block sum split over G row groups of at most b/G rows,
  the G partial sums added in a fixed order, then one division:
  |error| <= (ceil(b/G) + G + 1) u sum|x| / c = e_p u A, with A the mean of
  |x| over the block and G = 256 / (d / elements per 16 bytes). A score is a
  d-term float32 FMA chain times the scale, then compared with the float64
  value rounded to float32: |error| <= scale ((d + 2) u sum_c |qbar_c kbar_c|
  + e_p u sum_c (A^q_c |kbar_c| + |qbar_c| A^k_c)) + u |s|. The test allows
  twice that.
* attention: bf16 path within 2e-2 max-abs and 1e-3 mean-abs of the float64
  oracle; float32 path within 1e-5 max-abs.
"""

from __future__ import annotations

import math

import numpy as np

import oracle as orc
import paper_2609_32197_amd as sp

BF16_MAX_ABS = 2e-2
BF16_MEAN_ABS = 1e-3
F32_MAX_ABS = 1e-5


def torch():
    import torch as _t
    return _t


def to_device(arr: np.ndarray, dtype: str):
    """Generator arrays -> device tensors carrying the same bits."""
    t = torch()
    if dtype == "bf16":
        return t.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(t.bfloat16).cuda()
    return t.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).cuda()


def from_device_bits(t, dtype: str) -> np.ndarray:
    """Device tensor -> numpy with the raw element bits (uint16 for bf16)."""
    tt = torch()
    if dtype == "bf16":
        return t.view(tt.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def geometry(H, L, d, block, i0, i1, dtype: str) -> sp.Geometry:
    return sp.Geometry(H, L, d, block, i0, i1, sp.BF16 if dtype == "bf16" else sp.F32)


def oracle_pooled_scores(q_raw, k_raw, dtype, L, block, i0, i1, d, with_abs=False):
    """Pooled Q (local blocks), pooled K (all blocks), fp32 scores, head by head.

    With with_abs, also the block means of |Q| and |K| (for the error bound).
    """
    pqs, pks, aqs, aks = [], [], [], []
    for h in range(q_raw.shape[0]):
        qh = orc.decode_input(q_raw[h:h + 1], dtype)
        kh = orc.decode_input(k_raw[h:h + 1], dtype)
        pqs.append(orc.pool_blocks(qh, L, block, range(i0, i1)))
        pks.append(orc.pool_blocks(kh, L, block))
        if with_abs:
            aqs.append(orc.pool_blocks(np.abs(qh), L, block, range(i0, i1)))
            aks.append(orc.pool_blocks(np.abs(kh), L, block))
    pq = np.concatenate(pqs)
    pk = np.concatenate(pks)
    s = orc.block_scores(pq, pk, d)
    if with_abs:
        return pq, pk, s, np.concatenate(aqs), np.concatenate(aks)
    return pq, pk, s


def score_tolerance(pq, pk, aq, ak, s32, d, block, dtype):
    u = 2.0 ** -24
    scale = 1.0 / math.sqrt(d)
    groups = 256 // (d // (8 if dtype == "bf16" else 4))
    e_p = -(-block // groups) + groups + 1
    kt = np.swapaxes
    absdot = np.matmul(np.abs(pq), kt(np.abs(pk), 1, 2))
    pool_err = np.matmul(aq, kt(np.abs(pk), 1, 2)) + np.matmul(np.abs(pq), kt(ak, 1, 2))
    bound = scale * ((d + 2) * u * absdot + e_p * u * pool_err) + u * np.abs(s32.astype(np.float64))
    return 2.0 * bound


def words_as_int64(mask_bool: np.ndarray) -> np.ndarray:
    return orc.mask_to_words(mask_bool).view(np.int64)


def check_attention(O_gpu: np.ndarray, O_ref: np.ndarray, bf16: bool, what: str):
    err = np.abs(O_gpu.astype(np.float64) - O_ref)
    assert np.isfinite(O_gpu).all(), f"{what}: non-finite output"
    mx, mean = float(err.max()), float(err.mean())
    if bf16:
        assert mx <= BF16_MAX_ABS and mean <= BF16_MEAN_ABS, f"{what}: max {mx:.3g} mean {mean:.3g}"
    else:
        assert mx <= F32_MAX_ABS, f"{what}: max {mx:.3g}"
    return mx, mean


def check_every_row(q, k, v, mask, O_gpu: np.ndarray, lse_gpu: np.ndarray, wl, i0: int,
                    nq: int, bf16: bool, what: str, lse_tol: float):
    """Every (head, local query block) row of a full-size attention result against
    the oracle's Eq. 1 over the given mask (the GPU's own), O at the parity bar,
    lse within lse_tol, padded query rows lse = -inf. Heads run on a pool of host
    threads, each with a single-threaded BLAS. Returns the largest max-abs error."""
    import os
    from concurrent.futures import ThreadPoolExecutor
    from threadpoolctl import threadpool_limits
    b = wl.block

    def head(h):
        qf, kf, vf = (orc.decode_input(x[h], wl.dtype) for x in (q, k, v))
        worst = 0.0
        for r in range(nq):
            o_ref, l_ref = orc.attend_block(qf, kf, vf, mask[h, r], i0 + r, wl.L, b,
                                            wl.softmax_scale)
            mx, _ = check_attention(O_gpu[h, r * b:(r + 1) * b], o_ref, bf16, f"{what} h={h} r={r}")
            fin = np.isfinite(l_ref)
            lg = lse_gpu[h, r * b:(r + 1) * b]
            assert (np.isneginf(lg) == ~fin).all(), f"{what} h={h} r={r}: padded rows"
            err = float(np.abs(lg[fin] - l_ref[fin]).max()) if fin.any() else 0.0
            assert err <= lse_tol, f"{what} h={h} r={r}: lse off by {err:.3g}"
            worst = max(worst, mx)
        return worst

    workers = min(16, len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else 4)
    with threadpool_limits(1), ThreadPoolExecutor(workers) as ex:
        return max(ex.map(head, range(wl.H)))
