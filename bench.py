#!/usr/bin/env python3
"""Benchmark of the MiTA forward on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

One step = one whole forward (landmarks, scores + landmark values, top-k,
[gather], routing, attention) over one batch of synthetic inputs that are
resident in HBM before the timed region starts. Prints ONE JSON line on
stdout: tokens/s (a token is one sequence position across all heads) over the
timed region of plain forwards; the roofline of the dominant kernel, its
launch time measured live with HIP events on the launch stream in a second
pass of as many forwards with stage events; and the CPU oracle timed on a
bounded sample of the same workload. Per-stage details go to stderr.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MiTA fwd tokens/s at N=16384 + % MFMA/HBM roofline on 1 MI355X"
PEAK_HBM_GBS = 8000.0
PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
CSRC = os.path.join(ROOT, "paper_2602_01219_amd", "csrc")


def eprint(*a):
    print(*a, file=sys.stderr, flush=True)


def source_digest() -> str:
    h = hashlib.sha256()
    for f in sorted(os.listdir(CSRC)):
        if f.endswith((".hip", ".hpp")):
            h.update(f.encode())
            h.update(open(os.path.join(CSRC, f), "rb").read())
    return h.hexdigest()[:16]


def stage_work(wl, staged: bool, fused: bool):
    """Algorithmic work per stage launch: (bound, bytes, flops).

    bytes: what the stage must read and write at least (inputs once, outputs
    once); flops: its multiply-adds x 2 on the MFMA path. With the fused
    selection the score matrix is neither written nor read back."""
    e = 4 if wl.dtype == "f32" else 2
    BH, N, d, M, k = wl.BH, wl.N, wl.d, wl.M, wl.k
    sh, rt = wl.use_shared, wl.use_routed
    lm = ("hbm", BH * N * d * e + BH * M * d * e, 0)
    s_bytes = 4 * BH * M * N if (rt and not fused) else 0
    sc_bytes = BH * N * d * e * (1 + sh) + s_bytes + BH * M * d * e * (1 + sh)
    sc = ("hbm", sc_bytes, 2 * M * N * d * BH * (1 + sh))
    tk = ("hbm", s_bytes + 4 * BH * M * k, 0) if rt else ("hbm", 0, 0)
    ga = ("hbm", BH * M * k * (4 + 4 * d * e), 0) if (rt and staged) else ("hbm", 0, 0)
    ro = ("mfma", BH * N * d * e + BH * M * d * e + 4 * 3 * BH * N, 2 * N * M * d * BH) if rt else ("hbm", 0, 0)
    keys = M * sh + k * rt
    at = ("mfma", 2 * BH * N * d * e + 2 * BH * M * k * d * e * rt + 2 * BH * M * d * e * sh,
          4 * N * keys * d * BH)
    return dict(landmarks=lm, scores=sc, topk=tk, gather=ga, route=ro, attend=at)


# Kernel names (as rocprofv3 reports them) of the single-kernel stages.
KERNEL_OF_STAGE = {"topk": "topk_kernel", "attend": "attend_kernel", "gather": "gather_kernel",
                   "landmarks": "pool_kernel"}
IDX_LDS_MAX = 8192  # key row lists up to this length are staged in LDS by the attention


def kernel_of(stage, wl):
    """The kernel a single-kernel stage runs for this workload: bf16 attention
    with its key row list in LDS uses the 16-query-per-wave kernel."""
    if stage == "attend" and wl.dtype == "bf16":
        if wl.M * wl.use_shared + wl.k * wl.use_routed <= IDX_LDS_MAX:
            return "attend16_kernel"
    return KERNEL_OF_STAGE.get(stage, stage)


def cpu_baseline(wl, inp, budget_s: float):
    """Time the CPU oracle (as it stands) on whole (b, h) slices until about
    budget_s seconds are spent; scale to tokens/s of the full workload."""
    import numpy as np
    from oracle import mita_oracle as O
    from paper_2602_01219_amd import synth
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = 1
    done, spent = 0, 0.0
    order = [(b, h) for b in range(wl.B) for h in range(wl.H)]
    while done < len(order) and (spent < budget_s or done == 0):
        b, h = order[done]
        if wl.dtype == "f32":
            q, k, v = (x[b, h].astype(np.float64) for x in (inp.q, inp.k, inp.v))
        else:
            q, k, v = (synth.bf16_bits_to_f32(x[b, h]).astype(np.float64) for x in (inp.q, inp.k, inp.v))
        t0 = time.perf_counter()
        O.forward_slice(q, k, v, wl.grid_h, wl.grid_w, wl.lm_h, wl.lm_w, wl.k, None, wl.use_shared, wl.use_routed)
        spent += time.perf_counter() - t0
        done += 1
    per_slice = spent / done
    full_s = per_slice * wl.BH
    return {"value": wl.tokens / full_s, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{done} of {wl.BH} (b,h) slices of the same workload, float64 numpy oracle, "
                      f"{spent:.1f} s; scaled by {wl.BH}/{done} slices"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=None)
    ap.add_argument("--staged-gather", action="store_true", help="materialise expert tiles (flag path)")
    ap.add_argument("--full-scores", action="store_true",
                    help="store the score matrix and select from it (flag path) instead of the fused selection")
    ap.add_argument("--cpu-budget", type=float, default=15.0, help="seconds of oracle time for cpu_baseline")
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
    from paper_2602_01219_amd import mita, synth

    name = a.workload or synth.HEADLINE
    wl = synth.WORKLOADS[name]
    eprint(f"[bench] workload {name}: B={wl.B} H={wl.H} N={wl.N} d={wl.d} M={wl.M} k={wl.k} {wl.dtype}")
    inp = synth.generate(wl)
    torch.cuda.set_device(0)
    dt = torch.float32 if wl.dtype == "f32" else torch.bfloat16

    def dev(x):
        import numpy as np
        if wl.dtype == "f32":
            return torch.from_numpy(x).cuda()
        return torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).cuda()

    q, k, v = dev(inp.q), dev(inp.k), dev(inp.v)
    cfg = mita.Config.from_workload(wl, staged_gather=a.staged_gather, full_scores=a.full_scores)
    fused = (not a.full_scores) and bool(wl.use_routed) and (wl.N <= 1024 or 4 * wl.k <= 4096)
    o = torch.empty_like(q)
    ws = torch.empty(mita.workspace_size(cfg), dtype=torch.uint8, device="cuda")
    eprint(f"[bench] workspace {ws.numel() / 2**20:.1f} MiB")
    for _ in range(a.warmup):
        mita.forward(cfg, q, k, v, o=o, ws=ws)
    torch.cuda.synchronize()

    # timed region: plain forwards, as a caller runs them
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(a.steps):
        mita.forward(cfg, q, k, v, o=o, ws=ws)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    # per-stage times: the same number of forwards right after, with HIP events
    # recorded on the launch stream between the stages (the events add a few
    # microseconds per forward, so they stay out of the timed region above)
    timer = mita.Timer(a.steps)
    for _ in range(a.steps):
        mita.forward(cfg, q, k, v, o=o, ws=ws, timer=timer)
    per_call = timer.read()
    timer.close()
    # cold caches (secondary figure): before each forward, reading 512 MiB
    # evicts the inputs from L2 and the 256 MiB MALL; each forward is timed
    # alone with events on the launch stream and the median is reported
    flush = torch.ones(128 * 2**20, dtype=torch.float32, device="cuda")
    pairs = []
    for _ in range(a.steps):
        flush.sum()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        mita.forward(cfg, q, k, v, o=o, ws=ws)
        e1.record()
        pairs.append((e0, e1))
    torch.cuda.synchronize()
    cold_ms = sorted(e0.elapsed_time(e1) for e0, e1 in pairs)[len(pairs) // 2]
    del flush
    if a.calib_copy_mib:
        src = torch.empty(a.calib_copy_mib * 2**20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()

    ms_per_step = wall * 1e3 / a.steps
    value = wl.tokens * a.steps / wall
    stage_ms = {s: sum(c[i] for c in per_call) / len(per_call) for i, s in enumerate(mita.STAGES)}
    work = stage_work(wl, a.staged_gather, fused)
    eprint(f"[bench] {ms_per_step:.3f} ms/step, {value / 1e6:.2f} M tokens/s; "
           f"cold caches {cold_ms:.3f} ms/forward ({wl.tokens / cold_ms / 1e3:.2f} M tokens/s)")
    for s in mita.STAGES:
        bound, by, fl = work[s]
        t = stage_ms[s] * 1e-3
        extra = ""
        if t > 0 and (by or fl):
            extra = f"  {by / t / 1e9:8.1f} GB/s  {fl / t / 1e12:8.2f} TFLOP/s"
        eprint(f"[bench]   {s:10s} {stage_ms[s] * 1e3:9.1f} us{extra}")

    dom = max(stage_ms, key=stage_ms.get)
    bound, by, fl = work[dom]
    t = stage_ms[dom] * 1e-3
    if bound == "mfma":
        ach, peak, unit = fl / t / 1e12, PEAK_TFLOPS[wl.dtype], "TFLOP/s"
    else:
        ach, peak, unit = by / t / 1e9, PEAK_HBM_GBS, "GB/s"
    traffic = None
    try:
        tr = json.load(open(TRAFFIC_FILE))
        ent = tr.get(f"{kernel_of(dom, wl)}@{name}")
        if ent and ent.get("source_digest") == source_digest():
            traffic = ent["bytes_per_launch"]
    except (OSError, ValueError):
        pass
    roofline = {"bound": bound, "achieved": round(ach, 3), "peak": peak, "unit": unit,
                "frac": round(ach / peak, 5), "traffic": traffic, "kernel": kernel_of(dom, wl),
                "stage": dom, "launch_us": round(stage_ms[dom] * 1e3, 2),
                "algorithmic_bytes": by, "algorithmic_flops": fl}

    cpu = None
    if not a.no_cpu_baseline:
        eprint("[bench] timing the CPU oracle on a sample ...")
        cpu = cpu_baseline(wl, inp, a.cpu_budget)
        eprint(f"[bench] cpu oracle {cpu['value']:.1f} tokens/s ({cpu['sample']})")

    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": a.steps,
        "warmup": a.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": wl.dtype, "data": "synthetic",
        "config": {"workload": name, "B": wl.B, "H": wl.H, "N": wl.N, "d": wl.d, "M": wl.M, "k": wl.k,
                   "grid": [wl.grid_h, wl.grid_w], "use_shared": wl.use_shared, "use_routed": wl.use_routed,
                   "gather": "staged" if a.staged_gather else "in-place",
                   "select": "fused" if fused else "full-scores", "parallelism": "none (1 GPU)"},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "stages_us": {s: round(stage_ms[s] * 1e3, 2) for s in mita.STAGES},
        "cold": {"ms_per_forward": round(cold_ms, 4), "tokens_per_s": round(wl.tokens / cold_ms * 1e3, 1),
                 "note": "median single forward after reading 512 MiB (L2 and MALL evicted)"},
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
