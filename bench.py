#!/usr/bin/env python3
"""Benchmark of the MiTA forward on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--dense]
    python bench.py --sweep            # the paper's operating points, MiTA and dense

One step = one whole forward (landmarks, scores + landmark values, top-k,
[gather], routing, attention) over one batch of synthetic inputs that are
resident in HBM before the timed region starts. Prints ONE JSON line on stdout
(one per run with --sweep): tokens/s (a token is one sequence position across
all heads) over the timed region of plain forwards; per-kernel times from a
second pass of as many forwards with one HIP event behind each launch (on the
launch stream), each kernel priced against its algorithmic bytes and flops;
the roofline of the dominant kernel; and the CPU oracle timed on a bounded
sample of the same workload. Details go to stderr.

--dense runs the dense reference on the same inputs instead: route-only with
one landmark and k = N, so every query attends over every key (full softmax
attention) on the same kernels; PyTorch's flash SDPA is timed beside it as
context.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MiTA fwd tokens/s at N=16384 + % MFMA/HBM roofline on 1 MI355X"
PEAK_HBM_GBS = 8000.0
PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
CSRC = os.path.join(ROOT, "paper_2602_01219_amd", "csrc")
SCORE_NC = 512        # keys per score-pass chunk
ROUTE_TQ = 64         # queries per routing tile
# kernels priced against MFMA whatever their byte count (the attention: its
# algorithmic bytes count every expert's k rows, most of which come from L2)
MFMA_KERNELS = ("attend16_kernel", "attend_kernel", "bwd_attend_kernel", "bwd_landmark_kernel", "bwd_kv_landmark_kernel",
                "bwd_kv_kernel",
                "bwd_kv_shared_kernel")


def eprint(*a):
    print(*a, file=sys.stderr, flush=True)


def source_digest() -> str:
    h = hashlib.sha256()
    for f in sorted(os.listdir(CSRC)):
        if f.endswith((".hip", ".hpp")):
            h.update(f.encode())
            h.update(open(os.path.join(CSRC, f), "rb").read())
    return h.hexdigest()[:16]


def kernel_work(name: str, wl, plan: dict, staged: bool, s: int = 1, launched=()):
    """Algorithmic (bytes, flops) of one launch of kernel `name`: the tensors
    its step must read and write at least (inputs once, outputs once) and its
    multiply-adds x 2. Intermediate buffers of this design (score-pass
    partials, candidate lists) are not counted, except, with s > 1 routed
    experts, the pairs' partial results, which the expert-wise evaluation
    must write and merge."""
    e = 4 if wl.dtype == "f32" else 2
    BH, N, d, M, k = wl.BH, wl.N, wl.d, wl.M, wl.k
    sh, rt = wl.use_shared, wl.use_routed
    s = s if rt else 1
    rows = BH * M
    tens = BH * N * d * e            # one of q, k, v, o
    lmt = BH * M * d * e             # q_lm or v_lm
    nch = -(-N // SCORE_NC)
    G = 2 * M if s > 1 else M        # routing groups
    NP = N * s                       # routing items
    ntiles = -(-NP // ROUTE_TQ)
    pairs = BH * NP * (d + 1) * 4 if s > 1 else 0  # fp32 partials and log-sum-exps
    ns = plan.get("ns") or 0
    stored_s = rt and not plan.get("fused")
    w = {
        "pool_kernel": (tens + lmt, 0),
        "sample_pivot_kernel": (BH * ns * d * e + lmt + 4 * rows + (4 * rows * k if ns == N else 0),
                                2 * M * ns * d * BH),
        "scores_kernel": (tens * (1 + sh) + lmt + 4 * BH * M * N * stored_s, 2 * M * N * d * BH * (1 + sh)),
        "merge_kernel": (BH * nch * M * (d + 2) * 4 + lmt, 0),
        "finalize_kernel": (4 * rows * k + lmt * sh, 0),
        # the routing logits run in the finish launch unless the pivot launch
        # took them (sample_logits_kernel)
        # (with the sample the whole row, N <= 1024, the sample launch writes the
        # sets and the finish launch forms the routing logits only)
        "finalize_logits_kernel": (4 * rows * k + lmt * sh, 0) if "sample_logits_kernel" in launched else
                                  ((tens + lmt + 4 * BH * N, 2 * N * M * d * BH) if ns == N else
                                   (4 * rows * k + lmt * sh + tens + lmt + 4 * BH * N, 2 * N * M * d * BH)),
        "sample_logits_kernel": (BH * ns * d * e + lmt + 4 * rows + tens + lmt + 4 * BH * N,
                                 2 * M * ns * d * BH + 2 * N * M * d * BH),
        "topk_scatter_kernel": (8 * BH * N + 8 * BH * (M + 1), 0),
        "scores_rows_kernel": (0, 0),
        "topk_kernel": (4 * BH * M * N + 4 * rows * k, 0),
        "gather_kernel": (rows * k * (4 + 4 * d * e), 0),
        "route_logits_kernel": (tens + lmt + 4 * BH * N, 2 * N * M * d * BH),
        "route_scan_kernel": (8 * BH * ntiles * G, 0),
        "route_scatter_kernel": (8 * BH * NP + 4 * BH * ntiles * G, 0),
        "route_tops_kernel": (tens + lmt + 8 * BH * NP, 2 * N * M * d * BH),
        "pair_count_kernel": (4 * BH * NP + 4 * BH * ntiles * G, 0),
        "combine_kernel": (pairs + tens, 0),
        "select_landmarks_kernel": (2 * lmt + 4 * rows, 0),
        "worklist_kernel": (8 * BH * (G + 1), 0),
        "zero_kernel": (4 * BH * G, 0),
    }
    att = (2 * tens + 2 * BH * M * k * d * e * rt + 2 * lmt * sh + (pairs - tens if s > 1 else 0),
           4 * N * (M * sh + k * s * rt) * d * BH)
    # backward (s = 1): inputs once (q, o, dO, the keys and values each
    # query attends, landmarks) and each gradient contribution once in fp32;
    # flops of the five products S, dP, dQ, dK, dV (the log-sum-exp pass that
    # recomputes S is this design's overhead and is not counted)
    # (per kernel: the products it forms; S and dP are formed both by the
    # dQ kernel and by the key-owned kernels, so their sum exceeds the
    # backward's minimum of five products)
    nkeys = M * sh + k * rt
    w["bwd_attend_kernel"] = (3 * tens + 2 * BH * M * k * d * e * rt + 2 * lmt * sh + 4 * BH * N * d + 8 * BH * N,
                              6 * N * nkeys * d * BH)
    w["bwd_kv_kernel"] = (2 * BH * M * k * d * e + 2 * tens + 8 * BH * N + 8 * BH * M * k * d, 8 * N * k * d * BH * rt)
    w["bwd_kv_shared_kernel"] = (2 * lmt + 2 * tens + 8 * BH * N + 8 * BH * M * d, 8 * N * M * d * BH * sh)
    # inverse index of the top-k sets: the sets read once, slots and starts written
    w["inv_index_kernel"] = (8 * BH * M * k * rt + 4 * BH * (N + 1) * rt, 0)
    w["inv_gather_kernel"] = (8 * BH * M * k * d + 4 * BH * M * k + 8 * BH * N + 8 * BH * N * d, 0)
    if wl.dtype == "f32":
        w["bwd_landmark_kernel"] = (2 * lmt + 4 * BH * M * d + 2 * tens + 4 * rows + 8 * BH * N * d + 4 * BH * M * d,
                                    10 * M * N * d * BH * sh)
    else:
        # bf16: the landmark queries' gradient (S, dP, dQ~) and, in its own
        # launch, the keys' (S, dP, dK, dV; each token row read and written once)
        w["bwd_landmark_kernel"] = (2 * lmt + 2 * tens + 8 * rows + 4 * BH * M * d, 6 * M * N * d * BH * sh)
        # (with the routed keys' staged rows summed in and dk, dv written)
        w["bwd_kv_landmark_kernel"] = (2 * tens + 2 * lmt + 8 * rows
                                       + (8 * BH * M * k * d + 4 * BH * M * k + 4 * BH * N) * rt + 2 * tens,
                                       8 * M * N * d * BH * sh)
        w["lmv_prep_kernel"] = (4 * BH * M * d + 2 * lmt + 4 * rows, 0)
    # (bf16 with the landmark values: dk, dv come from the landmark-value
    # key pass, the finish forms dq only)
    w["bwd_finish_kernel"] = ((4 * BH * N * d + 4 * BH * M * d + tens, 0) if "bwd_kv_landmark_kernel" in launched
                              else (12 * BH * N * d + 4 * BH * M * d * sh + 3 * tens, 0))
    w["lse_rows_kernel"] = (8 * BH * nch * M + 4 * rows, 0)
    w["scores16_kernel"] = w["scores_kernel"]
    w["pool_small_kernel"] = w["pool_kernel"]
    w["finalize_wave_kernel"] = w["finalize_kernel"]
    w["attend16_kernel"] = att
    w["attend_kernel"] = att
    return w.get(name, (0, 0))


def price(name, us, by, fl, dtype):
    """Roofline of one kernel: achieved rates and fractions of both peaks;
    `bound` is the roof whose ideal time is longer (MFMA for the attention)."""
    t = us * 1e-6
    peak_f = PEAK_TFLOPS[dtype]
    t_hbm = by / (PEAK_HBM_GBS * 1e9)
    t_mfma = fl / (peak_f * 1e12)
    bound = "mfma" if (name in MFMA_KERNELS or t_mfma > t_hbm) else "hbm"
    gbs = by / t / 1e9 if t > 0 else 0.0
    tfs = fl / t / 1e12 if t > 0 else 0.0
    return {"kernel": name, "us": round(us, 2), "bound": bound, "algorithmic_bytes": by, "algorithmic_flops": fl,
            "gb_s": round(gbs, 1), "tflop_s": round(tfs, 2),
            "frac_hbm": round(gbs / PEAK_HBM_GBS, 4), "frac_mfma": round(tfs / peak_f, 4),
            "frac": round((tfs / peak_f) if bound == "mfma" else (gbs / PEAK_HBM_GBS), 4)}


def cpu_info():
    model = platform.processor() or "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    blas, threads = "unknown", 1
    try:
        from threadpoolctl import threadpool_info
        info = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        if info:
            blas = f"{info[0].get('internal_api')} {info[0].get('version')}"
            threads = max(i.get("num_threads", 1) for i in info)
    except Exception:
        pass
    return model, blas, threads


def cpu_baseline(wl, inp, budget_s: float):
    """Time the CPU oracle (as it stands) on whole (b, h) slices until about
    budget_s seconds are spent, once with float32 inputs (the oracle then
    computes in float32) and once in float64 (its parity precision) on half
    the budget; scale to tokens/s of the full workload."""
    import numpy as np
    from oracle import mita_oracle as O
    from paper_2602_01219_amd import synth
    model, blas, threads = cpu_info()
    order = [(b, h) for b in range(wl.B) for h in range(wl.H)]

    def run(dtype, budget):
        done, spent = 0, 0.0
        while done < len(order) and (spent < budget or done == 0):
            b, h = order[done]
            if wl.dtype == "f32":
                q, k, v = (x[b, h].astype(dtype) for x in (inp.q, inp.k, inp.v))
            else:
                q, k, v = (synth.bf16_bits_to_f32(x[b, h]).astype(dtype) for x in (inp.q, inp.k, inp.v))
            t0 = time.perf_counter()
            O.forward_slice(q, k, v, wl.grid_h, wl.grid_w, wl.lm_h, wl.lm_w, wl.k, None, wl.use_shared,
                            wl.use_routed)
            spent += time.perf_counter() - t0
            done += 1
        return wl.tokens / (spent / done * wl.BH), done, spent

    v32, n32, s32 = run(np.float32, budget_s)
    v64, n64, s64 = run(np.float64, budget_s / 2)
    return {"value": v32, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{n32} of {wl.BH} (b,h) slices of the same workload, numpy oracle on float32 inputs, "
                      f"{s32:.1f} s; scaled by {wl.BH}/{n32} slices",
            "value_f64": v64, "sample_f64": f"{n64} slices in float64 (the parity precision), {s64:.1f} s",
            "cpu_model": model, "blas": blas, "affinity_cpus": len(os.sched_getaffinity(0))}


def sdpa_ms(q, k, v, steps, warmup):
    """PyTorch's flash SDPA on the same tensors (context only): the flash
    backend is forced, so no other kernel is timed; None if it is unavailable."""
    import torch
    try:
        from torch.nn.attention import SDPBackend, sdpa_kernel
        with sdpa_kernel(SDPBackend.FLASH_ATTENTION):
            for _ in range(warmup):
                torch.nn.functional.scaled_dot_product_attention(q, k, v)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(steps):
                torch.nn.functional.scaled_dot_product_attention(q, k, v)
            torch.cuda.synchronize()
            return (time.perf_counter() - t0) * 1e3 / steps
    except RuntimeError as ex:
        eprint(f"[bench] flash SDPA unavailable: {str(ex).splitlines()[0][:120]}")
        return None


def run(wl, name, a, dense: bool):
    import numpy as np
    import torch
    from paper_2602_01219_amd import mita, synth

    inp = synth.generate(wl)
    if dense:
        wl = synth.dense_reference(wl)
    eprint(f"[bench] workload {name}{' (dense reference)' if dense else ''}: B={wl.B} H={wl.H} N={wl.N} d={wl.d} "
           f"M={wl.M} k={wl.k} shared={wl.use_shared} routed={wl.use_routed} {wl.dtype}")
    dt = torch.float32 if wl.dtype == "f32" else torch.bfloat16

    def dev(x):
        if wl.dtype == "f32":
            return torch.from_numpy(x).cuda()
        return torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).cuda()

    q, k, v = dev(inp.q), dev(inp.k), dev(inp.v)
    s_exp = a.s if wl.use_routed else 1
    cfg = mita.Config.from_workload(wl, staged_gather=a.staged_gather, full_scores=a.full_scores, s=s_exp)
    plan = mita.select_plan(cfg)
    o = torch.empty_like(q)
    ws = torch.empty(mita.workspace_size(cfg), dtype=torch.uint8, device="cuda")
    eprint(f"[bench] s = {s_exp}, landmarks by {a.landmarks}; workspace {ws.numel() / 2**20:.1f} MiB; "
           f"selection {plan}")
    random_lm = a.landmarks == "random"
    tome_lm = a.landmarks == "tome"
    if random_lm or tome_lm:
        # random selection (the draw is an input) or token merging: a step
        # forms the landmarks, then runs the forward from them
        sel = torch.from_numpy(synth.landmark_draw(wl)).cuda() if random_lm else None
        q_lm = torch.empty((wl.B, wl.H, wl.M, wl.d), dtype=q.dtype, device="cuda")
        ws_t = (torch.empty(mita.workspace_size(cfg, mita.WS_TOME), dtype=torch.uint8, device="cuda")
                if tome_lm else None)

    def make_landmarks():
        if random_lm:
            mita.landmarks_select(cfg, q, sel, q_lm=q_lm)
        else:
            mita.landmarks_tome(cfg, q, q_lm=q_lm, want_assign=False, ws=ws_t)

    if a.backward:
        r = np.random.default_rng(wl.seed + 17)
        dO = dev(synth.f32_to_bf16_bits((r.standard_normal((wl.B, wl.H, wl.N, wl.d)) / np.sqrt(wl.d)).astype(
            np.float32)) if wl.dtype == "bf16" else (r.standard_normal((wl.B, wl.H, wl.N, wl.d)) /
                                                        np.sqrt(wl.d)).astype(np.float32))
        grads = tuple(torch.empty_like(x) for x in (q, k, v))
        ws_b = torch.empty(mita.workspace_size(cfg, mita.WS_BACKWARD), dtype=torch.uint8, device="cuda")
        eprint(f"[bench] backward workspace {ws_b.numel() / 2**20:.1f} MiB")

    def step(timer=None, timer_b=None):
        if a.backward:
            mita.forward(cfg, q, k, v, o=o, ws=ws, timer=timer)
            mita.backward(cfg, q, k, v, o, dO, *grads, ws=ws_b, timer=timer_b)
            return
        if random_lm or tome_lm:
            make_landmarks()
            mita.forward(cfg, q, k, v, o=o, ws=ws, timer=timer, q_lm=q_lm)
        else:
            mita.forward(cfg, q, k, v, o=o, ws=ws, timer=timer)

    for _ in range(a.warmup):
        step()
    torch.cuda.synchronize()

    # timed region: whole steps, as a caller runs them
    t0 = time.perf_counter()
    for _ in range(a.steps):
        step()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    fallbacks = mita.forward_fallbacks(cfg, ws)
    # per-kernel times: the same number of forwards right after, with one HIP
    # event behind each launch on the launch stream (the events add a few
    # microseconds per forward, so they stay out of the timed region above);
    # random selection's landmark copy is timed with events of its own
    timer = mita.Timer(a.steps)
    timer_b = mita.Timer(a.steps) if a.backward else None
    sel_ev = []
    for _ in range(a.steps):
        if a.backward:
            step(timer, timer_b)
        elif random_lm or tome_lm:
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            make_landmarks()
            e1.record()
            sel_ev.append((e0, e1))
            mita.forward(cfg, q, k, v, o=o, ws=ws, timer=timer, q_lm=q_lm)
        else:
            mita.forward(cfg, q, k, v, o=o, ws=ws, timer=timer)
    per_call = timer.launches()
    timer.close()
    if a.backward:
        per_call = [f + b_ for f, b_ in zip(per_call, timer_b.launches())]
        timer_b.close()
    if random_lm or tome_lm:
        torch.cuda.synchronize()
        lm_name = "select_landmarks_kernel" if random_lm else "token merging (all launches)"
        per_call = [call + [(lm_name, 0, e0.elapsed_time(e1))] for call, (e0, e1) in zip(per_call, sel_ev)]
    # cold caches (secondary figure): before each forward, reading 512 MiB
    # evicts the inputs from L2 and the 256 MiB MALL; each forward is timed
    # alone with events on the launch stream and the median is reported
    flush = torch.ones(128 * 2**20, dtype=torch.float32, device="cuda")
    pairs = []
    for _ in range(a.steps):
        flush.sum()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        step()
        e1.record()
        pairs.append((e0, e1))
    torch.cuda.synchronize()
    cold_ms = sorted(e0.elapsed_time(e1) for e0, e1 in pairs)[len(pairs) // 2]
    del flush
    sdpa = None
    if dense:
        sdpa = sdpa_ms(q, k, v, a.steps, a.warmup)
    if a.calib_copy_mib:
        # a plain elementwise kernel that reads and writes calib_copy_mib MiB
        # each (torch's copy_ of contiguous tensors is a runtime blit, whose
        # stores the counters need not see like an ordinary kernel's)
        src = torch.ones(a.calib_copy_mib * 2**18, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()

    # the HBM rate a plain streaming kernel reaches on this machine (context for
    # the fractions, which use the published 8 TB/s): torch.mul by 1 of 1 GiB
    # of fp32 into another 1 GiB, median of 5 event-timed launches
    hbm_src = torch.ones(2**28, dtype=torch.float32, device="cuda")
    hbm_dst = torch.empty_like(hbm_src)
    torch.mul(hbm_src, 1.0, out=hbm_dst)
    hbm_ms = []
    for _ in range(5):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        torch.mul(hbm_src, 1.0, out=hbm_dst)
        e1.record()
        torch.cuda.synchronize()
        hbm_ms.append(e0.elapsed_time(e1))
    measured_hbm = 2 * 2**30 / (sorted(hbm_ms)[2] * 1e-3) / 1e9
    del hbm_src, hbm_dst
    eprint(f"[bench] streaming kernel on this box: {measured_hbm:.0f} GB/s (1 GiB read + 1 GiB written)")

    ms_per_step = wall * 1e3 / a.steps
    value = wl.tokens * a.steps / wall
    # per kernel: average time per forward (launches of one kernel in a forward summed)
    per_kernel, launches, stage_us = {}, {}, [0.0] * mita.NUM_STAGES
    for call in per_call:
        seen = {}
        for kname, stage, ms in call:
            seen[kname] = seen.get(kname, 0.0) + ms * 1e3
            launches[kname] = launches.get(kname, 0) + 1
            stage_us[stage] += ms * 1e3
        for kname, us in seen.items():
            per_kernel[kname] = per_kernel.get(kname, 0.0) + us
    ncalls = max(1, len(per_call))
    kernels = []
    for kname, us in sorted(per_kernel.items(), key=lambda x: -x[1]):
        us /= ncalls
        by, fl = kernel_work(kname, wl, plan, a.staged_gather, s_exp, per_kernel)
        ent = price(kname, us, by, fl, wl.dtype)
        ent["launches_per_forward"] = round(launches[kname] / ncalls, 2)
        kernels.append(ent)
    stage_us = [u / ncalls for u in stage_us]
    eprint(f"[bench] {ms_per_step:.4f} ms/step, {value / 1e6:.2f} M tokens/s; "
           f"cold caches {cold_ms:.4f} ms/forward ({wl.tokens / cold_ms / 1e3:.2f} M tokens/s); "
           f"fallback rows {fallbacks}")
    for ent in kernels:
        eprint(f"[bench]   {ent['kernel']:24s} {ent['us']:9.2f} us  {ent['gb_s']:8.1f} GB/s ({ent['frac_hbm']:.3f})"
               f"  {ent['tflop_s']:8.2f} TFLOP/s ({ent['frac_mfma']:.3f})  bound {ent['bound']}")
    for s, u in zip(mita.STAGES, stage_us):
        eprint(f"[bench]   stage {s:10s} {u:9.2f} us" + ("" if u > 0 else "  (launches nothing)"))

    dom = kernels[0]
    traffic = None
    try:
        tr = json.load(open(TRAFFIC_FILE))
        ent = tr.get(f"{dom['kernel']}@{name}{'@dense' if dense else ''}")
        if ent and ent.get("source_digest") == source_digest():
            traffic = ent["bytes_per_launch"]
    except (OSError, ValueError):
        pass
    bound = dom["bound"]
    roofline = {"bound": bound,
                "achieved": dom["tflop_s"] if bound == "mfma" else dom["gb_s"],
                "peak": PEAK_TFLOPS[wl.dtype] if bound == "mfma" else PEAK_HBM_GBS,
                "unit": "TFLOP/s" if bound == "mfma" else "GB/s",
                "frac": dom["frac"], "traffic": traffic, "kernel": dom["kernel"], "launch_us": dom["us"],
                "algorithmic_bytes": dom["algorithmic_bytes"], "algorithmic_flops": dom["algorithmic_flops"]}

    cpu = None
    if not a.no_cpu_baseline and not dense and s_exp == 1 and a.landmarks == "pool" and not a.backward:
        eprint("[bench] timing the CPU oracle on a sample ...")
        cpu = cpu_baseline(wl, inp, a.cpu_budget)
        eprint(f"[bench] cpu oracle {cpu['value']:.1f} tokens/s fp32, {cpu['value_f64']:.1f} fp64 "
               f"({cpu['cores']} threads, {cpu['cpu_model']}, {cpu['blas']})")

    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": a.steps,
        "warmup": a.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": wl.dtype, "data": "synthetic",
        "config": {"workload": name + (" dense reference" if dense else "") + (" forward+backward" if a.backward
                                                                                  else ""), "B": wl.B, "H": wl.H,
                   "N": wl.N,
                   "d": wl.d, "M": wl.M, "k": wl.k, "grid": [wl.grid_h, wl.grid_w],
                   "use_shared": wl.use_shared, "use_routed": wl.use_routed,
                   "gather": "staged" if a.staged_gather else "in-place",
                   "select": "fused" if plan["fused"] else "full-scores", "s": s_exp, "landmarks": a.landmarks,
                   "parallelism": "none (1 GPU)"},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "kernels": kernels,
        "stages_us": {s: round(u, 2) for s, u in zip(mita.STAGES, stage_us)},
        "fallback_rows": fallbacks,
        "measured_hbm_gb_s": round(measured_hbm, 1),
        "cold": {"ms_per_forward": round(cold_ms, 4), "tokens_per_s": round(wl.tokens / cold_ms * 1e3, 1),
                 "note": "median single forward after reading 512 MiB (L2 and MALL evicted)"},
    }
    if dense:
        out["sdpa_flash_ms"] = None if sdpa is None else round(sdpa, 4)
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=None)
    ap.add_argument("--dense", action="store_true",
                    help="dense reference on the same inputs: route-only, one landmark, k = N")
    ap.add_argument("--sweep", action="store_true",
                    help="the paper's operating points, MiTA then the dense reference, one JSON line each")
    ap.add_argument("--staged-gather", action="store_true", help="materialise expert tiles (flag path)")
    ap.add_argument("--full-scores", action="store_true",
                    help="store the score matrix and select from it (flag path) instead of the fused selection")
    ap.add_argument("--s", type=int, default=1, help="routed experts per query (Eq. mita)")
    ap.add_argument("--backward", action="store_true",
                    help="time forward + backward steps (gradients of q, k, v for a synthetic upstream gradient)")
    ap.add_argument("--landmarks", choices=("pool", "random", "tome"), default="pool",
                    help="landmark extraction: 2-D pooling (default), random selection or token merging (Tab. A1)")
    ap.add_argument("--cpu-budget", type=float, default=12.0,
                    help="seconds of float32 oracle time for cpu_baseline (half as much again in float64)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="after the timed region, run one device copy of this many MiB (counter calibration)")
    a = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if a.gpus != 1 or world != 1:
        print(json.dumps({"error": "this build measures one GPU only: run with --gpus 1",
                          "n_gpus": a.gpus}), flush=True)
        sys.exit(2)

    import torch
    from paper_2602_01219_amd import synth
    torch.cuda.set_device(0)

    if a.sweep:
        a.no_cpu_baseline = True  # the oracle baseline belongs to the headline line
        for name in synth.OPERATING_ORDER:
            for dense in (False, True):
                out = run(synth.WORKLOADS[name], name, a, dense)
                print(json.dumps(out), flush=True)
        return
    name = a.workload or synth.HEADLINE
    print(json.dumps(run(synth.WORKLOADS[name], name, a, a.dense)), flush=True)


if __name__ == "__main__":
    main()
