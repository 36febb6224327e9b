"""Synthetic stand-ins for the paper's video-DiT attention workloads.

The paper evaluates on LTX-Video, LTX-2 and HunyuanVideo at 768x1536 and
768x1280 (Section 8.1). Their weights and prompts are not available, so these
seeded generators produce Q/K/V of the same shapes instead: tokens in t-h-w
raster order (index = (t*Hy + y)*W + x), per-head [L, d] matrices, iid N(0,1)
values, and for the locality workload a shared low-frequency 3-D sinusoidal
feature in Q and K so that attention concentrates on spatio-temporal
neighbourhoods, the diagonal / multi-diagonal structure the paper reports in
Section 4.3. Text tokens, where present, are appended after the video tokens.

Values are drawn in float64, rounded to float32 (round to nearest even) and,
for bf16 workloads, rounded again to bfloat16 (round to nearest even). Every
consumer receives these exact bits.

Random streams: numpy PCG64 seeded from SeedSequence([seed, config_id]); the
root spawns one child per tensor (Q noise, K noise, V noise, feature
parameters) and each child one grandchild per head, so any subset of heads can
be regenerated on its own and heads can be generated in parallel.
"""

from __future__ import annotations

import dataclasses
import math
from concurrent.futures import ThreadPoolExecutor
from typing import Optional, Sequence

import numpy as np

__all__ = [
    "Workload",
    "CONFIGS",
    "get_workload",
    "workload_names",
    "make_qkv",
    "bf16_round_bits",
]


@dataclasses.dataclass(frozen=True)
class Workload:
    """Geometry of one rank's share of a sparse attention layer.

    Q, K and V are [H, L, d] with d contiguous. Tokens are cut into
    n = ceil(L / block) blocks; the local query blocks are the contiguous
    slice [i0, i1) owned by rank ``rank`` of ``ranks``
    (i0 = floor(rank*n/ranks)). ``keep`` counts all kept KV blocks of a row,
    forced ones included.
    """

    name: str
    config_id: int
    H: int
    d: int
    block: int
    latent: tuple  # (T, Hy, W) video latent grid
    text_tokens: int
    dtype: str  # "f32" or "bf16"
    keep_pct: Optional[int]  # keep = ceil(keep_pct * n / 100) when keep_abs is None
    keep_abs: Optional[int]
    ranks: int
    rank: int
    feature: str  # "iid", "sinusoid" or "sinusoid-spatial"

    # ---- derived geometry -------------------------------------------------
    @property
    def video_tokens(self) -> int:
        t, y, x = self.latent
        return t * y * x

    @property
    def L(self) -> int:
        return self.video_tokens + self.text_tokens

    @property
    def n(self) -> int:
        return -(-self.L // self.block)

    @property
    def i0(self) -> int:
        return self.rank * self.n // self.ranks

    @property
    def i1(self) -> int:
        return (self.rank + 1) * self.n // self.ranks

    @property
    def nq(self) -> int:
        return self.i1 - self.i0

    @property
    def keep(self) -> int:
        if self.keep_abs is not None:
            return self.keep_abs
        return -(-(self.keep_pct * self.n) // 100)

    @property
    def global_blocks(self) -> tuple:
        """Blocks holding at least one text token: always-kept global KV blocks."""
        if self.text_tokens == 0:
            return ()
        first = self.video_tokens // self.block
        return tuple(range(first, self.n))

    @property
    def bytes_per_elem(self) -> int:
        return 4 if self.dtype == "f32" else 2

    @property
    def softmax_scale(self) -> float:
        """d**-0.5 rounded to float32: the value both sides are handed."""
        return float(np.float32(1.0 / math.sqrt(self.d)))

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)

    def describe(self) -> dict:
        return {
            "workload": self.name,
            "H": self.H,
            "d": self.d,
            "block": self.block,
            "L": self.L,
            "n_blocks": self.n,
            "local_blocks": [self.i0, self.i1],
            "keep": self.keep,
            "global_blocks": list(self.global_blocks),
            "dtype": self.dtype,
        }


def _cfg(**kw) -> Workload:
    base = dict(text_tokens=0, keep_pct=None, keep_abs=None, ranks=1, rank=0, feature="iid")
    base.update(kw)
    return Workload(**base)


CONFIGS = {
    # Tiny fp32 case: 4x16x16 latent, 16 blocks of 64, top-4 plus the diagonal.
    "tiny-f32": _cfg(name="tiny-f32", config_id=1, H=2, d=64, block=64, latent=(4, 16, 16),
                     dtype="f32", keep_abs=5),
    # Wan-style layer share: rank 0 of 4, ~15% kept, locality from a shared sinusoid.
    "wan-share": _cfg(name="wan-share", config_id=2, H=40, d=128, block=128, latent=(21, 45, 80),
                      dtype="bf16", keep_pct=15, ranks=4, feature="sinusoid"),
    # HunyuanVideo-style layer share: rank 0 of 8, ~10% kept.
    "hunyuan-share": _cfg(name="hunyuan-share", config_id=3, H=24, d=128, block=128,
                          latent=(33, 45, 80), dtype="bf16", keep_pct=10, ranks=8),
    # The whole HunyuanVideo-style layer on one GPU, ~10% kept, and its dense twin.
    "hunyuan-layer": _cfg(name="hunyuan-layer", config_id=4, H=24, d=128, block=128,
                          latent=(33, 45, 80), dtype="bf16", keep_pct=10),
    "hunyuan-layer-dense": _cfg(name="hunyuan-layer-dense", config_id=4, H=24, d=128, block=128,
                                latent=(33, 45, 80), dtype="bf16", keep_pct=100),
}
# The wan-style layer with a frame-independent feature (no temporal frequency):
# attention then depends on the in-frame position alone, the multi-diagonal
# pattern of Section 4.3. Used only to study placement.
CONFIGS["wan-share-multidiag"] = dataclasses.replace(
    CONFIGS["wan-share"], name="wan-share-multidiag", config_id=6, feature="sinusoid-spatial")
# Density / text-token sweep: 13x30x45 video + 226 text tokens, rank 0 of 2.
for _pct in (5, 10, 25, 50, 100):
    CONFIGS[f"text-sweep-{_pct}"] = _cfg(
        name=f"text-sweep-{_pct}", config_id=5, H=48, d=64, block=64, latent=(13, 30, 45),
        text_tokens=226, dtype="bf16", keep_pct=_pct, ranks=2)


def workload_names() -> list:
    return list(CONFIGS)


def get_workload(name: str) -> Workload:
    try:
        return CONFIGS[name]
    except KeyError:
        raise KeyError(f"unknown workload {name!r}; known: {', '.join(CONFIGS)}") from None


# ---------------------------------------------------------------------------
# rounding
# ---------------------------------------------------------------------------

def bf16_round_bits(x32: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest even.

    Inputs here are finite, so no NaN special case is needed.
    """
    u = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


# ---------------------------------------------------------------------------
# generation
# ---------------------------------------------------------------------------

_Q, _K, _V, _FEAT = range(4)


def _head_streams(wl: Workload, seed: int):
    root = np.random.SeedSequence([int(seed), int(wl.config_id)])
    per_tensor = root.spawn(4)
    return [t.spawn(wl.H) for t in per_tensor]


def _sinusoid_feature(wl: Workload, ss: np.random.SeedSequence) -> np.ndarray:
    """f[tok, c] = sqrt(2) cos(2 pi (nu_t t/T + nu_y y/Hy + nu_x x/W) + phi) on video tokens.

    With the "sinusoid-spatial" feature nu_t is 0: the same in every frame.
    """
    rng = np.random.Generator(np.random.PCG64(ss))
    nu = rng.uniform(0.0, 2.0, size=(wl.d, 3))
    if wl.feature == "sinusoid-spatial":
        nu[:, 0] = 0.0
    phi = rng.uniform(0.0, 2.0 * np.pi, size=wl.d)
    T, Hy, W = wl.latent
    t = np.arange(T, dtype=np.float64)[:, None, None] / T
    y = np.arange(Hy, dtype=np.float64)[None, :, None] / Hy
    x = np.arange(W, dtype=np.float64)[None, None, :] / W
    f = np.zeros((wl.L, wl.d), dtype=np.float64)
    for c in range(wl.d):
        arg = 2.0 * np.pi * (nu[c, 0] * t + nu[c, 1] * y + nu[c, 2] * x) + phi[c]
        f[: wl.video_tokens, c] = np.sqrt(2.0) * np.cos(arg).reshape(-1)
    return f


def _finish(x64: np.ndarray, dtype: str) -> np.ndarray:
    x32 = x64.astype(np.float32)
    if dtype == "f32":
        return x32
    return bf16_round_bits(x32)


def _one_head(wl: Workload, streams, h: int):
    out = []
    feat = None
    if wl.feature in ("sinusoid", "sinusoid-spatial"):
        feat = _sinusoid_feature(wl, streams[_FEAT][h])
    for t in (_Q, _K, _V):
        rng = np.random.Generator(np.random.PCG64(streams[t][h]))
        x = rng.standard_normal((wl.L, wl.d))
        if feat is not None and t in (_Q, _K):
            x += 2.0 * feat
        out.append(_finish(x, wl.dtype))
    return out


def make_qkv(wl: Workload, seed: int = 0, heads: Optional[Sequence[int]] = None,
             threads: int = 8):
    """Return (Q, K, V) for the heads listed (all by default).

    bf16 workloads come back as uint16 bit patterns, f32 workloads as float32;
    each array is [len(heads), L, d], C-contiguous.
    """
    if heads is None:
        heads = list(range(wl.H))
    heads = [int(h) for h in heads]
    for h in heads:
        if not 0 <= h < wl.H:
            raise ValueError(f"head {h} out of range for H={wl.H}")
    streams = _head_streams(wl, seed)
    dt = np.float32 if wl.dtype == "f32" else np.uint16
    shape = (len(heads), wl.L, wl.d)
    q, k, v = (np.empty(shape, dtype=dt) for _ in range(3))

    def work(idx_h):
        idx, h = idx_h
        qh, kh, vh = _one_head(wl, streams, h)
        q[idx], k[idx], v[idx] = qh, kh, vh

    jobs = list(enumerate(heads))
    if threads > 1 and len(jobs) > 1:
        with ThreadPoolExecutor(max_workers=min(threads, len(jobs))) as ex:
            list(ex.map(work, jobs))
    else:
        for j in jobs:
            work(j)
    return q, k, v
