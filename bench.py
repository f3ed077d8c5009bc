"""Benchmark of the MoE expert stage on one MI355X.

One step = one micro-batch through the whole stage (dispatch, grouped GEMM
gate/up + SiLU*up, grouped GEMM down, combine) via
moe_stage_submit_microbatch, inputs already resident in HBM.

Prints ONE JSON line.  `value` is tokens/s of the primary workload
(DeepSeek-V3-shaped EP32 share, T=4096, 8 of 256 experts local, top-8).
The same line carries the same measurement at T=32768 (about 1024 token-slots
per local expert, where the grouped GEMM is compute-bound), per-kernel times
from HIP events recorded by the library on the launch stream, the roofline
of the dominant kernel, and the CPU oracle's throughput on the host.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MoE-stage prefill tokens/s on 1 GPU; grouped-GEMM TFLOP/s vs MFMA peak"
PEAK_BF16_TFLOPS = 2500.0       # MI355X dense bf16 MFMA
PEAK_FP8_TFLOPS = 5000.0
PEAK_HBM_GBS = 8000.0           # MI355X HBM3E


def _log(msg):
    print(msg, file=sys.stderr, flush=True)


def gemm_accounting(cfg, counts_local, T):
    """Algorithmic FLOPs and HBM bytes of one launch of each grouped GEMM.

    gate/up: 4 d f FLOP per row; reads each active expert's [2f, d] weights
    once, the routed rows of X_perm (and x for the shared expert), writes H.
    down:    2 d f FLOP per row; reads [d, f] weights, H; writes Y.
    """
    d, f = cfg.d, cfg.f
    eb = 1 if cfg.dtype == "fp8" else 2
    rows = int(counts_local.sum())
    active = int(np.count_nonzero(counts_local))
    if cfg.has_shared:
        rows += T
        active += 1
    g1_flop = 4.0 * d * f * rows
    g1_bytes = active * 2 * f * d * eb + rows * d * eb + rows * f * eb
    g2_flop = 2.0 * d * f * rows
    g2_bytes = active * d * f * eb + rows * f * eb + rows * d * 2
    return dict(rows=rows, active=active, g1_flop=g1_flop, g1_bytes=g1_bytes,
                g2_flop=g2_flop, g2_bytes=g2_bytes)


def stream_accounting(cfg, counts_local, n_tokens_with_local, T):
    """Algorithmic bytes of the gather and the combine (overwrite mode)."""
    d, k = cfg.d, cfg.k
    n_loc = int(counts_local.sum())
    rb = d * 2
    gather = n_tokens_with_local * rb + n_loc * rb + n_loc * 4
    combine = T * k * 12 + n_loc * rb + T * rb + (T * rb if cfg.has_shared else 0)
    return dict(gather_bytes=gather, combine_bytes=combine)


def run_workload(name, steps, warmup, n_buffers=3):
    import torch
    from paper_2606_22541_amd import inputs
    from paper_2606_22541_amd import moe_stage as C
    from paper_2606_22541_amd.stage import ExpertStage, to_device_routing

    cfg = inputs.CONFIGS[name]
    t0 = time.time()
    w = inputs.make_weights(cfg, "cuda")
    mb = inputs.make_microbatches(cfg, "cuda")[0]
    T = mb.ids.shape[0]
    _log("[bench] %s: inputs ready in %.1fs (T=%d)" % (name, time.time() - t0, T))
    ids, wt = to_device_routing(mb.ids, mb.w)
    # distinct input/output buffers so consecutive steps do not hit cached rows
    bufs = []
    for i in range(n_buffers):
        x = mb.x.clone()
        out = torch.empty((T, cfg.d), dtype=torch.bfloat16, device="cuda")
        bufs.append((x, ids.clone(), wt.clone(), out))
    torch.cuda.synchronize()
    stage = ExpertStage(cfg, w, n_slots=2, max_tokens=T)
    mbs = [stage.microbatch(x, i_, w_, o) for (x, i_, w_, o) in bufs]
    stream = torch.cuda.Stream()
    for s in range(warmup):
        stage.submit(mbs[s % n_buffers], stream)
    stage.sync()
    torch.cuda.synchronize()
    # timed region 1: the step rate, nothing but the stage on the stream
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for s in range(steps):
        stage.submit(mbs[s % n_buffers], stream)
    end.record(stream)
    stage.sync()
    torch.cuda.synchronize()
    ms = start.elapsed_time(end)
    # timed region 2: the same steps with the library's per-kernel HIP events
    C.moe_stage_profile(stage.handle, True)
    for s in range(steps):
        stage.submit(mbs[s % n_buffers], stream)
    stage.sync()
    torch.cuda.synchronize()
    prof = C.moe_stage_profile_read(stage.handle)
    C.moe_stage_profile(stage.handle, False)
    stage.close()

    counts = np.bincount(mb.ids[(mb.ids >= 0)].ravel(), minlength=cfg.E)
    counts_local = counts[cfg.e0:cfg.e0 + cfg.E_loc]
    local = (mb.ids >= cfg.e0) & (mb.ids < cfg.e0 + cfg.E_loc)
    n_tok_local = int(np.count_nonzero(local.any(axis=1)))
    acct = gemm_accounting(cfg, counts_local, T)
    acct.update(stream_accounting(cfg, counts_local, n_tok_local, T))
    kern = {k: (v[0] / v[1] if v[1] else None) for k, v in prof.items()}
    del w, mb, bufs
    torch.cuda.empty_cache()
    return dict(cfg=cfg, T=T, ms=ms, steps=steps, kern=kern, acct=acct,
                n_local_slots=int(counts_local.sum()))


def measured_traffic(workload, kernel):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or
    None when it is missing or the kernel's sources changed since."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        from paper_2606_22541_amd.profiling import sources_digest
        rec = json.load(open(path))["kernels"]["%s:%s" % (workload, kernel)]
        if rec["source_sha256"] != sources_digest(kernel):
            return None
        return rec["bytes_per_dispatch"]
    except Exception:
        return None


def roofline_for(r, kernel="gemm_gate_up_swiglu"):
    a = r["acct"]
    t = r["kern"][kernel] / 1e3
    flop, byts = (a["g1_flop"], a["g1_bytes"]) if kernel == "gemm_gate_up_swiglu" else (
        a["g2_flop"], a["g2_bytes"])
    peak_tf = PEAK_FP8_TFLOPS if r["cfg"].dtype == "fp8" else PEAK_BF16_TFLOPS
    t_mfma = flop / (peak_tf * 1e12)
    t_hbm = byts / (PEAK_HBM_GBS * 1e9)
    if t_mfma >= t_hbm:
        ach = flop / t / 1e12
        return {"kernel": kernel, "bound": "mfma", "achieved": round(ach, 1), "peak": peak_tf,
                "unit": "TFLOP/s", "frac": round(ach / peak_tf, 4),
                "traffic": measured_traffic(r["cfg"].name, kernel),
                "algorithmic_flop": flop, "algorithmic_bytes": byts, "avg_ms": round(t * 1e3, 4)}
    ach = byts / t / 1e9
    return {"kernel": kernel, "bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS,
            "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBS, 4),
            "traffic": measured_traffic(r["cfg"].name, kernel),
            "algorithmic_flop": flop, "algorithmic_bytes": byts, "avg_ms": round(t * 1e3, 4),
            "tflops": round(flop / t / 1e12, 1)}


def stream_rooflines(r):
    a = r["acct"]
    out = {}
    for k, b in (("gather", a["gather_bytes"]), ("combine", a["combine_bytes"])):
        t = r["kern"][k]
        if t:
            gbs = b / (t / 1e3) / 1e9
            out[k] = {"avg_ms": round(t, 4), "algorithmic_bytes": b, "achieved_GBs": round(gbs, 1),
                      "frac_hbm": round(gbs / PEAK_HBM_GBS, 4)}
    g1, g2 = r["kern"]["gemm_gate_up_swiglu"], r["kern"]["gemm_down"]
    out["gemm_gate_up_swiglu"] = {"avg_ms": round(g1, 4),
                                  "tflops": round(a["g1_flop"] / (g1 / 1e3) / 1e12, 1)}
    out["gemm_down"] = {"avg_ms": round(g2, 4),
                        "tflops": round(a["g2_flop"] / (g2 / 1e3) / 1e12, 1)}
    out["grouped_gemm_total"] = {
        "tflops": round((a["g1_flop"] + a["g2_flop"]) / ((g1 + g2) / 1e3) / 1e12, 1),
        "frac_mfma": round((a["g1_flop"] + a["g2_flop"]) / ((g1 + g2) / 1e3) / 1e12
                           / PEAK_BF16_TFLOPS, 4)}
    out["dispatch_index"] = {"avg_ms": round(r["kern"]["dispatch_index"], 4)}
    return out


def cpu_baseline(name="c1", min_seconds=10.0):
    """The CPU oracle on the full T=4096 micro-batch of the primary workload."""
    import oracle
    import torch
    from paper_2606_22541_amd import inputs
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count()
    cfg = inputs.CONFIGS[name]
    dev = "cuda" if torch.cuda.is_available() else "cpu"
    w = inputs.make_weights(cfg, dev)
    mb = inputs.make_microbatches(cfg, dev)[0]
    ow = oracle.OracleWeights(w, cfg.dtype)
    xb = mb.x.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)
    del w
    # repeat the whole micro-batch until about 10 s of CPU work has been timed
    runs, t0 = 0, time.time()
    while True:
        oracle.run_stage(cfg, ow, xb, mb.ids, mb.w)
        runs += 1
        dt = time.time() - t0
        if dt >= min_seconds or runs >= 50:
            break
    T = mb.ids.shape[0]
    return {"value": round(T * runs / dt, 1), "unit": "tokens/s", "cores": int(threads),
            "kind": "oracle",
            "sample": "%d x the full %s micro-batch (T=%d, %d local slots), fp64, %.1f s wall" % (
                runs, name, T,
                int(np.count_nonzero((mb.ids >= cfg.e0) & (mb.ids < cfg.e0 + cfg.E_loc))), dt)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="c1")
    ap.add_argument("--secondary", default="c1p", help="'' to skip")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="only run a plain device copy of this many MiB (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU's expert share; runs on %d GPUs are not part of this "
              "build (the stage shards by expert; see the design notes)." % args.gpus,
              file=sys.stderr)
        sys.exit(2)
    import torch
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.calibrate_copy_mib:
        n = args.calibrate_copy_mib << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibration_copy_bytes": n}))
        return

    prim = run_workload(args.workload, args.steps, args.warmup)
    cfg = prim["cfg"]
    ms_step = prim["ms"] / prim["steps"]
    line = {
        "metric": METRIC,
        "value": round(prim["T"] * prim["steps"] / (prim["ms"] / 1e3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded; DeepSeek-V3 layer shapes, Gaussian bf16 weights, uniform "
                "top-8 routing)",
        "config": {"workload": "%s: DeepSeek-V3 EP32 expert share, T=%d tokens, d=%d, f=%d, "
                               "%d of %d experts local, top-%d, bf16" % (
                                   cfg.name, prim["T"], cfg.d, cfg.f, cfg.E_loc, cfg.E, cfg.k),
                   "tokens_per_step": prim["T"], "local_slots": prim["n_local_slots"]},
        "roofline": roofline_for(prim),
        "kernels": stream_rooflines(prim),
    }
    _log("[bench] primary done: %.3f ms/step" % ms_step)
    if args.secondary:
        sec = run_workload(args.secondary, max(args.steps // 2, 5), args.warmup)
        line[args.secondary] = {
            "workload": "%s: same share at T=%d (about %d token-slots per local expert)" % (
                sec["cfg"].name, sec["T"], sec["n_local_slots"] // sec["cfg"].E_loc),
            "tokens_per_s": round(sec["T"] * sec["steps"] / (sec["ms"] / 1e3), 1),
            "ms_per_step": round(sec["ms"] / sec["steps"], 4),
            "roofline": roofline_for(sec),
            "kernels": stream_rooflines(sec),
        }
        _log("[bench] secondary done")
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(args.workload)
        _log("[bench] cpu baseline done")
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
