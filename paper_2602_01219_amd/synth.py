"""Seeded synthetic inputs for the MiTA forward workloads.

This module only draws random tensors and describes workload shapes. It holds
none of the method's arithmetic (no pooling, scoring, selection, routing or
attention), so both the HIP path and the CPU oracle can be fed from it without
sharing any computation.

The workloads stand in for the paper's image and long-sequence settings
(Sec. 4.1: 224px / patch 16 gives a 14x14 grid; Sec. 4.2: dense prediction at
higher resolution; Sec. 4.3: long sequences). No dataset item is used.

Tensors are laid out [B, H, N, d], row-major, token t of a grid_h x grid_w
patch grid at position (t // grid_w, t % grid_w).

Recipe (numpy PCG64, seed = 20260201 + workload number; fixed draw order
centres -> cluster map -> noise Q, K, V -> outliers):
  * Q and K of one (b, h) share one set of cluster centres c ~ N(0, I_d);
    V has its own centres. The cluster map z is per batch element and shared
    by heads and by Q/K/V.
  * x_t = (c_{z_t} + std * eps_t) / sqrt(d), eps ~ N(0, I_d), drawn in
    float64, then rounded to float32 (and from float32 to bfloat16 with
    round-to-nearest-even for the bf16 workloads).
  * cluster map: iid uniform, or a Voronoi map over the patch grid (sites
    uniform in [0, gh) x [0, gw), a token at (r + 1/2, c + 1/2) takes its
    nearest site, ties to the lower site).
  * outliers: a fixed fraction of tokens per batch element (without
    replacement, shared across heads) have q, k and v multiplied by a factor.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Optional

import numpy as np

BASE_SEED = 20260201


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    grid_h: int
    grid_w: int
    d: int
    lm_h: int
    lm_w: int
    k: int
    dtype: str                 # "f32" or "bf16"
    clusters: int
    std: float
    cluster_map: str           # "iid" or "voronoi"
    outlier_frac: float = 0.0
    outlier_scale: float = 1.0
    seed: int = BASE_SEED
    use_shared: int = 1
    use_routed: int = 1
    note: str = ""

    @property
    def N(self) -> int:
        return self.grid_h * self.grid_w

    @property
    def M(self) -> int:
        return self.lm_h * self.lm_w

    @property
    def BH(self) -> int:
        return self.B * self.H

    @property
    def tokens(self) -> int:
        # one token = one sequence position across all heads
        return self.B * self.N

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


def lm_grid(M: int) -> tuple[int, int]:
    """Landmark grid for M landmarks: lm_h = largest divisor of M <= sqrt(M)."""
    h = int(np.floor(np.sqrt(M)))
    while M % h:
        h -= 1
    return h, M // h


def _wl(idx, name, B, H, g, d, M, k, dtype, clusters, std, cmap, **kw):
    lh, lw = lm_grid(M)
    return Workload(name=name, B=B, H=H, grid_h=g, grid_w=g, d=d, lm_h=lh,
                    lm_w=lw, k=k, dtype=dtype, clusters=clusters, std=std,
                    cluster_map=cmap, seed=BASE_SEED + idx, **kw)


# The five workloads (ViT-shaped to long-sequence) and the dense-equivalence mode.
WORKLOADS = {
    "tiny_f32": _wl(1, "tiny_f32", 1, 1, 14, 64, 16, 32, "f32", 8, 1.0, "iid",
                    note="single head, 14x14 grid, fp32"),
    "vits_bf16": _wl(2, "vits_bf16", 64, 6, 14, 64, 16, 49, "bf16", 16, 0.5, "iid",
                     note="ViT-S shape, 14x14 grid"),
    "vitb_hr_bf16": _wl(3, "vitb_hr_bf16", 8, 12, 64, 64, 64, 256, "bf16", 32, 0.5,
                        "voronoi", note="ViT-B shape, 64x64 grid"),
    "dense_pred_bf16": _wl(4, "dense_pred_bf16", 2, 12, 128, 64, 128, 512, "bf16", 64,
                           0.5, "voronoi", outlier_frac=0.05, outlier_scale=4.0,
                           note="dense prediction, 128x128 grid, 5% outliers"),
    "long_bf16": _wl(5, "long_bf16", 1, 16, 256, 128, 256, 1024, "bf16", 128, 0.5,
                     "iid", note="long sequence, 256x256 grid, d=128"),
    "dense_equiv_bf16": _wl(6, "dense_equiv_bf16", 1, 16, 64, 128, 256, 4096, "bf16",
                            128, 0.5, "iid", use_shared=0,
                            note="route-only with k = N: equals full attention"),
}

def _wl1d(idx, name, B, H, N, d, M, k, dtype, clusters, std, **kw):
    """A 1-D sequence (grid 1 x N, landmark grid 1 x M: 1-D pooling)."""
    return Workload(name=name, B=B, H=H, grid_h=1, grid_w=N, d=d, lm_h=1, lm_w=M, k=k,
                    dtype=dtype, clusters=clusters, std=std, cluster_map="iid",
                    seed=BASE_SEED + idx, **kw)


# The paper's own operating points (m = k), at batch sizes that fill one GPU:
#  * image classification, 224 px / patch 16 (14 x 14 tokens), m = k = 25
#    (Sec. 4.1, Tab. ablation default; 5 x 5 landmarks: windows overlap);
#  * semantic segmentation at 512 px and 640 px (32 x 32 and 40 x 40 tokens),
#    m = k = 49 (Sec. 4.2; 7 x 7 landmarks: windows overlap);
#  * long sequences of 1K, 2K and 4K tokens, m = k = 128 (Sec. 4.3, the
#    long-range setting and its wall-clock comparison; 1-D pooling), two heads
#    of 64 (model width 128), B * N = 262144 tokens.
OPERATING_POINTS = {
    "vit_m25_bf16": _wl(7, "vit_m25_bf16", 64, 6, 14, 64, 25, 25, "bf16", 16, 0.5, "iid",
                        note="ViT-S image shape, 14x14 grid, m = k = 25"),
    "seg512_m49_bf16": _wl(8, "seg512_m49_bf16", 16, 6, 32, 64, 49, 49, "bf16", 32, 0.5,
                           "voronoi", note="segmentation at 512 px, 32x32 grid, m = k = 49"),
    "seg640_m49_bf16": _wl(9, "seg640_m49_bf16", 16, 6, 40, 64, 49, 49, "bf16", 32, 0.5,
                           "voronoi", note="segmentation at 640 px, 40x40 grid, m = k = 49"),
    "seq1k_m128_bf16": _wl1d(10, "seq1k_m128_bf16", 256, 2, 1024, 64, 128, 128, "bf16", 32, 0.5,
                             note="1-D sequence of 1024 tokens, m = k = 128"),
    "seq2k_m128_bf16": _wl1d(11, "seq2k_m128_bf16", 128, 2, 2048, 64, 128, 128, "bf16", 32, 0.5,
                             note="1-D sequence of 2048 tokens, m = k = 128"),
    "seq4k_m128_bf16": _wl1d(12, "seq4k_m128_bf16", 64, 2, 4096, 64, 128, 128, "bf16", 32, 0.5,
                             note="1-D sequence of 4096 tokens, m = k = 128"),
}
OPERATING_ORDER = list(OPERATING_POINTS)
WORKLOADS.update(OPERATING_POINTS)


def dense_reference(wl: Workload) -> Workload:
    """Route-only with one landmark and k = N on the same inputs: every query
    attends over every key, i.e. full softmax attention."""
    return wl.with_(lm_h=1, lm_w=1, k=wl.N, use_shared=0, use_routed=1)


WORKLOAD_ORDER = ["tiny_f32", "vits_bf16", "vitb_hr_bf16", "dense_pred_bf16",
                  "long_bf16", "dense_equiv_bf16"]
HEADLINE = "dense_pred_bf16"


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = u + 0x7FFF + ((u >> 16) & 1)
    return (u >> 16).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


@dataclass
class Inputs:
    """q, k, v in their storage form: float32 arrays, or uint16 bf16 bit patterns."""
    wl: Workload
    q: np.ndarray
    k: np.ndarray
    v: np.ndarray

    def as_f64(self):
        if self.wl.dtype == "f32":
            return tuple(x.astype(np.float64) for x in (self.q, self.k, self.v))
        return tuple(bf16_bits_to_f32(x).astype(np.float64) for x in (self.q, self.k, self.v))

    def as_f32(self):
        if self.wl.dtype == "f32":
            return self.q, self.k, self.v
        return tuple(bf16_bits_to_f32(x) for x in (self.q, self.k, self.v))


def _voronoi_map(rng, gh, gw, C):
    sites = rng.uniform(0.0, 1.0, size=(C, 2)) * np.array([gh, gw], dtype=np.float64)
    r = np.arange(gh, dtype=np.float64)[:, None] + 0.5
    c = np.arange(gw, dtype=np.float64)[None, :] + 0.5
    best = np.zeros((gh, gw), dtype=np.int64)
    bestd = np.full((gh, gw), np.inf)
    for s in range(C):  # ascending site order: strict < keeps the lower site on ties
        dd = (r - sites[s, 0]) ** 2 + (c - sites[s, 1]) ** 2
        upd = dd < bestd
        best[upd] = s
        bestd[upd] = dd[upd]
    return best.reshape(-1)


def generate(wl: Workload, seed: Optional[int] = None, B: Optional[int] = None,
             H: Optional[int] = None) -> Inputs:
    """Draw the seeded inputs of a workload (optionally only the first B / H slices
    are kept, which still consumes the same random stream for those slices only
    when B/H equal the workload's; reduced B/H draw a smaller, different stream)."""
    Bv = wl.B if B is None else B
    Hv = wl.H if H is None else H
    rng = np.random.Generator(np.random.PCG64(wl.seed if seed is None else seed))
    N, d, C = wl.N, wl.d, wl.clusters
    cen_qk = rng.standard_normal((Bv, Hv, C, d))
    cen_v = rng.standard_normal((Bv, Hv, C, d))
    if wl.cluster_map == "voronoi":
        z = np.stack([_voronoi_map(rng, wl.grid_h, wl.grid_w, C) for _ in range(Bv)])
    else:
        z = rng.integers(0, C, size=(Bv, N))
    inv = 1.0 / np.sqrt(d)
    out = []
    for cen in (cen_qk, cen_qk, cen_v):
        eps = rng.standard_normal((Bv, Hv, N, d))
        x = np.empty((Bv, Hv, N, d), dtype=np.float32)
        for b in range(Bv):
            x[b] = ((cen[b][:, z[b], :] + wl.std * eps[b]) * inv).astype(np.float32)
        del eps
        out.append(x)
    if wl.outlier_frac > 0.0:
        n_out = int(round(wl.outlier_frac * N))
        for b in range(Bv):
            sel = rng.choice(N, size=n_out, replace=False)
            for x in out:
                x[b][:, sel, :] *= np.float32(wl.outlier_scale)
    if wl.dtype == "bf16":
        out = [f32_to_bf16_bits(x) for x in out]
    wl2 = wl if (Bv == wl.B and Hv == wl.H) else wl.with_(B=Bv, H=Hv)
    return Inputs(wl2, *out)


def small(wl: Workload, **kw) -> Workload:
    """A reduced copy of a workload for tests (same recipe, other sizes)."""
    return wl.with_(**kw)


def landmark_draw(wl: Workload, seed: Optional[int] = None) -> np.ndarray:
    """Random-selection landmark draw (the method's random numbers, passed in as
    an input): for every (b, h) slice, M distinct token indices drawn uniformly
    without replacement, in draw order. Returns int32 [B, H, M]."""
    rng = np.random.Generator(np.random.PCG64((wl.seed if seed is None else seed) + 7919))
    out = np.empty((wl.B, wl.H, wl.M), dtype=np.int32)
    for b in range(wl.B):
        for h in range(wl.H):
            out[b, h] = rng.permutation(wl.N)[:wl.M]
    return out
