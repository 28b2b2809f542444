"""Helpers for the GPU parity tests: host<->device conversion, the selection
validation bounds, and the error metric. No method arithmetic lives here
beyond the comparison itself (the oracle computes every expected value)."""
from __future__ import annotations

import functools
import os
import subprocess
import sys

import numpy as np
import torch

from paper_2602_01219_amd import synth

U = 2.0 ** -24  # unit roundoff of fp32


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_dev(x: np.ndarray, dtype: str) -> torch.Tensor:
    if dtype == "f32":
        return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.uint16).view(np.int16)).view(torch.bfloat16).cuda()


def from_dev(t: torch.Tensor) -> np.ndarray:
    """Device tensor -> float64 numpy (exact widening)."""
    if t.dtype == torch.bfloat16:
        return synth.bf16_bits_to_f32(t.view(torch.int16).cpu().numpy().view(np.uint16)).astype(np.float64)
    if t.dtype == torch.float32:
        return t.cpu().numpy().astype(np.float64)
    return t.cpu().numpy()


def inputs_to_dev(inp: synth.Inputs):
    return tuple(to_dev(x, inp.wl.dtype) for x in (inp.q, inp.k, inp.v))


def maxrel(got: np.ndarray, ref: np.ndarray) -> float:
    """Normwise max-relative error of one slice: max|got - ref| / max|ref|."""
    return float(np.max(np.abs(got - ref)) / max(np.max(np.abs(ref)), 1e-30))


def tol_for(dtype: str) -> float:
    return 1e-5 if dtype == "f32" else 2e-2


def landmark_error(q_win_abs: np.ndarray, q_lm: np.ndarray, window: np.ndarray, dtype: str) -> np.ndarray:
    """Bound on |q_lm_gpu - q_lm_exact| per element: fp32 summation of a
    W-token window costs at most 2 W u times the mean of |q| over the window;
    rounding the mean to bf16 adds 2^-9 of its magnitude (2^-8 used)."""
    e = 2.0 * (window[:, None] + 2) * U * q_win_abs
    if dtype == "bf16":
        e = e + 2.0 ** -8 * (np.abs(q_lm) + e)
    return e


def dot_bound(a_abs: np.ndarray, a_err: np.ndarray, b: np.ndarray, scale: float) -> np.ndarray:
    """Bound tau[i, n] on |fl32(a_gpu_i . b_n) * scale - (a_i . b_n) * scale| when
    |a_gpu - a| <= a_err: the perturbation of a plus 2 (d + 2) u of the
    absolute dot product (fp32 products and accumulation, then the scaling)."""
    d = b.shape[1]
    ba = np.abs(b)
    return scale * (a_err @ ba.T) + scale * 2.0 * (d + 2) * U * ((a_abs + a_err) @ ba.T) + 1e-30


def window_stats(q: np.ndarray, gh, gw, lh, lw):
    """Mean of |q| over each landmark window and the window sizes (for bounds)."""
    from oracle import mita_oracle as O
    N, d = q.shape
    grid = np.abs(q).reshape(gh, gw, d)
    rows, cols = O.pool_windows(gh, lh), O.pool_windows(gw, lw)
    qa = np.empty((lh * lw, d))
    W = np.empty(lh * lw)
    for a, (r0, r1) in enumerate(rows):
        for b, (c0, c1) in enumerate(cols):
            qa[a * lw + b] = grid[r0:r1, c0:c1].reshape(-1, d).mean(0)
            W[a * lw + b] = (r1 - r0) * (c1 - c0)
    return qa, W


def check_selection(S_ref: np.ndarray, tau: np.ndarray, idx_gpu: np.ndarray, k: int):
    """Every GPU-selected token must be within the rounding budget of every
    unselected one: min_sel(S + tau) >= max_unsel(S - tau), per landmark row.
    Returns the number of rows whose set equals the oracle's own top-k set."""
    M, N = S_ref.shape
    assert idx_gpu.shape == (M, k)
    same = 0
    for i in range(M):
        sel = np.zeros(N, dtype=bool)
        sel[idx_gpu[i]] = True
        assert sel.sum() == k, "duplicate indices"
        assert (np.diff(idx_gpu[i]) > 0).all(), "indices not ascending"
        if k < N:
            lo = np.min(S_ref[i, sel] + tau[i, sel])
            hi = np.max(S_ref[i, ~sel] - tau[i, ~sel])
            assert lo >= hi, f"row {i}: selection outside the rounding budget ({lo} < {hi})"
        order = np.lexsort((np.arange(N), -S_ref[i]))
        same += int(set(order[:k].tolist()) == set(idx_gpu[i].tolist()))
    return same


def check_routing(L_ref: np.ndarray, tau: np.ndarray, expert_gpu: np.ndarray):
    """GPU argmax within the rounding budget: L[n, e] + tau >= max_j (L[n, j] - tau)."""
    N, M = L_ref.shape
    assert expert_gpu.min() >= 0 and expert_gpu.max() < M
    got = L_ref[np.arange(N), expert_gpu] + tau[np.arange(N), expert_gpu]
    best = np.max(L_ref - tau, axis=1)
    assert (got >= best).all(), f"routing outside the rounding budget at {np.nonzero(got < best)[0][:5]}"
    return int((np.argmax(L_ref, axis=1) == expert_gpu).sum())


@functools.lru_cache(maxsize=None)
def _region_tool(tmpdir: str) -> str:
    here = os.path.dirname(os.path.abspath(__file__))
    exe = os.path.join(tmpdir, "ws_float_regions")
    r = subprocess.run(["g++", "-std=c++17", "-O1", "-I", os.path.join(here, "..", "include"),
                        os.path.join(here, "host", "ws_float_regions.cpp"), "-o", exe], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return exe


def float_regions(cfg, tmpdir: str, forward: bool):
    """Byte ranges (kind, begin, end) of the floating-point regions of the
    forward's or the backward's workspace (kind "f32" or "io"), from the
    library's own layout header built for the host."""
    from paper_2602_01219_amd import mita
    args = [cfg.B, cfg.H, cfg.grid_h, cfg.grid_w, cfg.d, cfg.lm_h, cfg.lm_w, cfg.k, cfg.use_shared, cfg.use_routed,
            int(cfg.dtype == "bf16"), cfg.s, int(forward)]
    r = subprocess.run([_region_tool(tmpdir), *map(str, args)], capture_output=True, text=True)
    assert r.returncode == 0, r.stdout + r.stderr
    out = [l.split() for l in r.stdout.splitlines()]
    total = int(next(l[1] for l in out if l[0] == "total"))
    assert total == mita.workspace_size(cfg, mita.WS_FORWARD if forward else mita.WS_BACKWARD)
    return [(l[0], int(l[1]), int(l[2])) for l in out if l[0] != "total"]


def fill_float_regions(ws, regions, io_dtype):
    """Zero the workspace, then fill its floating-point regions with NaN."""
    ws.zero_()
    for kind, a, b in regions:
        if b > a:
            ws[a:b].view(torch.float32 if kind == "f32" else io_dtype).fill_(float("nan"))
