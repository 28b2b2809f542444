"""GPU parity of the backward pass (mita_backward) against the oracle's
backward_slice, through the C ABI.

The GPU recomputes the forward's top-k sets and routing; they are read back
through the stage entry points (which the forward tests show equal to the
forward's own), validated against the oracle's float64 scores and logits
within their rounding budget, and given to the oracle. dq, dk, dv are then
compared per (b, h) slice, every row: max|g_gpu - g_ref| / max|g_ref| <= 1e-4
(fp32) / 3e-2 (bf16). The bf16 bound: the softmax weights and their
gradients enter the products rounded to bf16 (relative 2^-9 each), dZ = P (dP
- D) can lose up to a few bits where dP is close to D, and the upstream
gradient of the landmark values is rounded to bf16 for the landmark-value
backward; the sums themselves are fp32.
"""
from __future__ import annotations

import dataclasses
import functools
import shutil

import numpy as np
import pytest
import torch

from oracle import mita_oracle as O
from paper_2602_01219_amd import mita, synth
from tests.gpu_helpers import (check_routing, check_selection, fill_float_regions, float_regions, from_dev, log,
                               maxrel, to_dev)
from tests.test_gpu_parity import _bounds

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "bf16": 3e-2}


@functools.lru_cache(maxsize=None)
def _inputs(name, B=None, H=None):
    return synth.generate(synth.WORKLOADS[name], B=B, H=H)


def _slice64(inp, b, h):
    if inp.wl.dtype == "f32":
        return tuple(x[b, h].astype(np.float64) for x in (inp.q, inp.k, inp.v))
    return tuple(synth.bf16_bits_to_f32(x[b, h]).astype(np.float64) for x in (inp.q, inp.k, inp.v))


def _upstream(wl, seed=17):
    r = np.random.default_rng(wl.seed + seed)
    x = (r.standard_normal((wl.B, wl.H, wl.N, wl.d)) / np.sqrt(wl.d)).astype(np.float32)
    return x if wl.dtype == "f32" else synth.f32_to_bf16_bits(x)


def _check_backward(cfg, inp, slices):
    wl = inp.wl
    q, k, v = (to_dev(x, wl.dtype) for x in (inp.q, inp.k, inp.v))
    dO_h = _upstream(wl)
    dO = to_dev(dO_h, wl.dtype)
    o = mita.forward(cfg, q, k, v)
    dq, dk, dv = mita.backward(cfg, q, k, v, o, dO)
    # the discrete choices the backward recomputed (equal to the forward's)
    q_lm = mita.landmarks(cfg, q)
    idx_all = exp_all = None
    if cfg.use_routed:
        S, _ = mita.scores(cfg, q_lm, k, v, want_v_lm=False)
        idx_all = mita.topk(cfg, S).cpu().numpy().astype(np.int64)
        exp_all = mita.route(cfg, q, q_lm)[0].cpu().numpy().astype(np.int64)
    torch.cuda.synchronize()
    g_all = [from_dev(t) for t in (dq, dk, dv)]
    dO64 = dO_h.astype(np.float64) if wl.dtype == "f32" else synth.bf16_bits_to_f32(dO_h).astype(np.float64)
    tol = TOL[wl.dtype]
    worst = 0.0
    for (b, h) in slices:
        qs, ks, vs = _slice64(inp, b, h)
        fi = fe = None
        if cfg.use_routed:
            q_lm_ref = O.landmarks(qs, cfg.grid_h, cfg.grid_w, cfg.lm_h, cfg.lm_w)
            tau_s, tau_r = _bounds(qs, ks, q_lm_ref, cfg, wl.dtype)
            check_selection(O.scores(q_lm_ref, ks, cfg.eff_scale), tau_s, idx_all[b, h], cfg.k)
            check_routing((qs @ q_lm_ref.T) * cfg.eff_scale, tau_r, exp_all[b, h])
            fi, fe = idx_all[b, h], exp_all[b, h]
        ref = O.backward_slice(qs, ks, vs, dO64[b, h], cfg.grid_h, cfg.grid_w, cfg.lm_h, cfg.lm_w, cfg.k, None,
                               cfg.use_shared, cfg.use_routed, force_idx=fi, force_expert=fe)
        errs = [maxrel(g[b, h], r) for g, r in zip(g_all, (ref.dq, ref.dk, ref.dv))]
        log(f"  slice ({b},{h}): max-rel dq {errs[0]:.3e} dk {errs[1]:.3e} dv {errs[2]:.3e} (tol {tol})")
        worst = max(worst, *errs)
        assert max(errs) <= tol, errs
    return worst


CASES = [("tiny_f32", None, None, (1, 1)), ("tiny_f32", None, None, (0, 1)), ("tiny_f32", None, None, (1, 0)),
         ("vits_bf16", 2, 2, (1, 1)), ("vits_bf16", 2, 2, (0, 1)), ("vits_bf16", 2, 2, (1, 0)),
         ("vitb_hr_bf16", 1, 2, (1, 1)), ("dense_pred_bf16", 1, 1, (1, 1)), ("long_bf16", 1, 1, (1, 1))]


@pytest.mark.parametrize("name,B,H,flags", CASES, ids=[f"{c[0]}_f{c[3][0]}{c[3][1]}" for c in CASES])
def test_backward_parity(name, B, H, flags):
    inp = _inputs(name, B, H)
    wl = inp.wl
    cfg = mita.Config.from_workload(wl, use_shared=flags[0], use_routed=flags[1])
    log(f"[backward] {name} B={wl.B} H={wl.H} N={wl.N} d={wl.d} M={wl.M} k={wl.k} flags={flags}")
    sl = [(b, h) for b in range(wl.B) for h in range(wl.H)]
    if wl.N > 4096:
        sl = sl[:1]
    _check_backward(cfg, inp, sl[:4])


def test_backward_dense_equivalence_is_attention_backward():
    # route-only, one landmark, k = N: the gradients of dense attention
    wl = synth.WORKLOADS["dense_equiv_bf16"].with_(H=2)
    inp = synth.generate(wl)
    cfg = mita.Config.from_workload(wl)
    q, k, v = (to_dev(x, wl.dtype) for x in (inp.q, inp.k, inp.v))
    dO = to_dev(_upstream(wl), wl.dtype)
    o = mita.forward(cfg, q, k, v)
    dq, dk, dv = mita.backward(cfg, q, k, v, o, dO)
    # the reference in float64 on the CPU (no device library in the reference)
    tq, tk, tv = (x.double().cpu().detach().requires_grad_() for x in (q, k, v))
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv)
    (ref * dO.double().cpu()).sum().backward()
    for name, got, r in (("dq", dq, tq.grad), ("dk", dk, tk.grad), ("dv", dv, tv.grad)):
        g = got.double().cpu()
        assert bool(torch.isfinite(g).all()), f"{name}: {int((~torch.isfinite(g)).sum())} non-finite values"
        err = ((g - r).abs().amax() / r.abs().amax()).item()
        log(f"  dense equivalence {name}: max-rel {err:.3e} vs SDPA autograd (float64, CPU)")
        assert err <= TOL["bf16"]


def test_backward_rejects_s_above_one_and_overlaps():
    inp = _inputs("tiny_f32")
    cfg = mita.Config.from_workload(inp.wl)
    q, k, v = (to_dev(x, "f32") for x in (inp.q, inp.k, inp.v))
    o = mita.forward(cfg, q, k, v)
    with pytest.raises(mita.MitaError) as ex:
        mita.backward(dataclasses.replace(cfg, s=2), q, k, v, o, o)
    assert ex.value.status == mita.MITA_ERR_UNSUPPORTED
    with pytest.raises(mita.MitaError) as ex:
        mita.backward(cfg, q, k, v, o, o, dq=q)
    assert ex.value.status == mita.MITA_ERR_INVALID_ARG


# Shapes whose inverse index splits a head's tokens into ranges that do not
# divide N, with more heads than XCDs, through the fp32 gather pass and the
# bf16 fused finish (d = 64 and 128); M k = 255 entries per head takes the
# inverse index's one-entry loads (M k not a multiple of 4), in both dtypes.
BWD_EDGE = [(36, 36, 6, 6, 36, 64, "bf16", 3, 3), (36, 36, 6, 6, 36, 64, "f32", 1, 3),
            (33, 41, 5, 4, 300, 128, "bf16", 2, 5), (15, 20, 3, 5, 17, 64, "bf16", 2, 3),
            (15, 20, 3, 5, 17, 128, "f32", 1, 2)]


@pytest.mark.parametrize("case", BWD_EDGE, ids=[f"{c[0]}x{c[1]}_m{c[2]*c[3]}_k{c[4]}_d{c[5]}_{c[6]}_b{c[7]}h{c[8]}"
                                                for c in BWD_EDGE])
def test_backward_edge_cases(case):
    gh, gw, lh, lw, kk, d, dtype, B, H = case
    wl = synth.Workload(name="bwd_edge", B=B, H=H, grid_h=gh, grid_w=gw, d=d, lm_h=lh, lm_w=lw, k=kk, dtype=dtype,
                        clusters=4, std=0.5, cluster_map="iid", seed=91 + gh * gw, use_shared=1, use_routed=1)
    inp = synth.generate(wl)
    cfg = mita.Config.from_workload(wl)
    log(f"[backward edge] {case}")
    _check_backward(cfg, inp, [(0, 0), (B - 1, H - 1)])


# Shapes with a partial query tile in every key pass: route-only k = N (most
# experts hold a few queries), the landmark rows as queries with M = 16 < 32
# (bf16, both branches), and the fp32 kernels.
WS_CASES = [("dense_equiv_bf16", 1, 2), ("vits_bf16", 2, 2), ("tiny_f32", None, None)]


@pytest.mark.skipif(shutil.which("g++") is None, reason="the layout helper needs g++")
@pytest.mark.parametrize("name,B,H", WS_CASES, ids=[c[0] for c in WS_CASES])
def test_backward_does_not_read_stale_workspace_or_lds(name, B, H, tmp_path_factory):
    """Regression: rows past a chunk's last query in the key passes once took
    0 * (dP - D) with D from an LDS slot not written for that chunk, which made
    every key's dk NaN when the slot held NaN bits. With the workspace's float
    regions filled with NaN beforehand (integer regions zero), the gradients
    must be finite and equal those from a zeroed workspace (to the rounding of
    the backward's unordered fp32 sums)."""
    inp = _inputs(name, B, H)
    wl = inp.wl
    cfg = mita.Config.from_workload(wl)
    q, k, v = (to_dev(x, wl.dtype) for x in (inp.q, inp.k, inp.v))
    dO = to_dev(_upstream(wl), wl.dtype)
    o = mita.forward(cfg, q, k, v)
    ws = torch.zeros(mita.workspace_size(cfg, mita.WS_BACKWARD), dtype=torch.uint8, device="cuda")
    clean = [g.float().clone() for g in mita.backward(cfg, q, k, v, o, dO, ws=ws)]
    regions = float_regions(cfg, str(tmp_path_factory.mktemp("layout")), forward=False)
    fill_float_regions(ws, regions, q.dtype)
    outs = [torch.full_like(q, float("nan")) for _ in range(3)]
    mita.backward(cfg, q, k, v, o, dO, dq=outs[0], dk=outs[1], dv=outs[2], ws=ws)
    torch.cuda.synchronize()
    for gname, g, ref in zip(("dq", "dk", "dv"), outs, clean):
        g = g.float()
        bad = int((~torch.isfinite(g)).sum())
        err = ((g - ref).abs().amax() / ref.abs().amax()).item() if bad == 0 else float("nan")
        log(f"  {name} {gname}: {bad} non-finite, max-rel {err:.3e} against the zeroed workspace")
        assert bad == 0
        assert err <= 1e-2
