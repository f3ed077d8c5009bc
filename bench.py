"""Benchmark of the MoE expert stage on one MI355X.

One step = one micro-batch through the whole stage (dispatch, grouped GEMM
gate/up + SiLU*up, grouped GEMM down, combine) via
moe_stage_submit_microbatch, inputs already resident in HBM.  Workloads with
several micro-batches run each on its own stream, and a step is all of them.

Prints ONE JSON line.  `value` is tokens/s of the primary workload
(DeepSeek-V3-shaped EP32 share, T=4096, 8 of 256 experts local, top-8).
The same line carries the further workloads (T=32768, where the grouped GEMM
is compute-bound; the EP8 share with a shared expert; four skewed ragged
micro-batches on four streams in bf16 and fp8), per-kernel times from HIP
events recorded by the library on the launch streams, the roofline of the
dominant kernel, the spread of the step time over repeated regions, and the
CPU oracle's throughput on the host.
"""
from __future__ import annotations

import argparse
import json
import os
import subprocess
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
    once and every routed row once (the token row of x, found through
    slot_of_row), and the shared expert's rows of x; writes H.
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
    """Algorithmic bytes of the dispatch index (ids read; counts, offsets and
    the two permutation arrays written), the gather and the combine
    (overwrite mode)."""
    d, k = cfg.d, cfg.k
    n_loc = int(counts_local.sum())
    rb = d * 2
    index = T * k * 4 + cfg.E * 4 + (cfg.E_loc + 1) * 4 + (n_loc + T * k) * 4
    # the gather runs in fp8 mode only and moves the token scales (one fp32
    # per 128 channels; the GEMM reads the e4m3 rows of x itself): each
    # token's scales read once, one row of scales written per routed row,
    # plus slot_of_row (and, with a shared expert, every token's scales
    # transposed for it)
    sb = (d // 128) * 4
    gather = n_tokens_with_local * sb + n_loc * sb + n_loc * 4
    if cfg.has_shared:
        gather += 2 * T * sb     # the shared expert's scales, transposed for all T rows
    combine = T * k * 12 + n_loc * rb + T * rb + (T * rb if cfg.has_shared else 0)
    return dict(index_bytes=index, gather_bytes=gather, combine_bytes=combine)


def run_workload(name, steps, warmup, n_buffers=3, repeats=5):
    """Times `steps` steps of workload `name`.  One step is every micro-batch
    of the workload through the stage; micro-batch i runs on its own stream,
    all of them released by one start event and joined at the end (a single
    micro-batch runs on one stream with nothing else on it).  Returns the
    timed region of exactly `steps` steps, the step times of `repeats`
    further regions (spread only), and per-kernel times from the library's
    events in one more region."""
    import torch
    from paper_2606_22541_amd import inputs
    from paper_2606_22541_amd import moe_stage as C
    from paper_2606_22541_amd.stage import ExpertStage, quantize_fp8, to_device_routing

    cfg = inputs.CONFIGS[name]
    t0 = time.time()
    w = inputs.make_weights(cfg, "cuda")
    mbs_in = inputs.make_microbatches(cfg, "cuda")
    n_micro = len(mbs_in)
    Ts = [mb.ids.shape[0] for mb in mbs_in]
    _log("[bench] %s: inputs ready in %.1fs (T=%s)" % (name, time.time() - t0, Ts))
    # distinct input/output buffer sets so consecutive steps do not hit cached rows
    n_sets = n_buffers if n_micro == 1 else 2
    sets = []
    for _ in range(n_sets):
        one = []
        for mb in mbs_in:
            ids, wt = to_device_routing(mb.ids, mb.w)
            x, xs = mb.x.clone(), None
            if cfg.dtype == "fp8":
                x, xs = quantize_fp8(x)        # sender-side, outside the timed region
            out = torch.empty((mb.ids.shape[0], cfg.d), dtype=torch.bfloat16, device="cuda")
            one.append((x, xs, ids, wt, out))
        sets.append(one)
    torch.cuda.synchronize()
    stage = ExpertStage(cfg, w, n_slots=max(2, n_micro), max_tokens=max(Ts))
    mbs = [[stage.microbatch(x, i_, w_, o, xs) for (x, xs, i_, w_, o) in one] for one in sets]
    main = torch.cuda.Stream()
    # micro-batch 0 runs on the launch stream itself, the others on streams
    # of their own: n_micro streams in all
    streams = [main] + [torch.cuda.Stream() for _ in range(n_micro - 1)]

    def step(s):
        group = mbs[s % n_sets]
        if n_micro == 1:
            stage.submit(group[0], main)
            return
        go = torch.cuda.Event()
        go.record(main)
        for i in range(1, n_micro):
            streams[i].wait_event(go)
        for i, m in enumerate(group):
            stage.submit(m, streams[i])
        # the join comes after every submission: the runtime maps streams
        # onto a few hardware queues, and a wait enqueued on the launch
        # stream between two submissions would hold back every later
        # micro-batch whose stream shares that queue
        for i in range(1, n_micro):
            done = torch.cuda.Event()
            done.record(streams[i])
            main.wait_event(done)

    def region(n):
        start = torch.cuda.Event(enable_timing=True)
        end = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        start.record(main)
        for s in range(n):
            step(s)
        end.record(main)
        stage.sync()
        torch.cuda.synchronize()
        return start.elapsed_time(end)

    for s in range(warmup):
        step(s)
    stage.sync()
    torch.cuda.synchronize()
    ms = region(steps)                                  # timed region: exactly `steps` steps
    spread = sorted([ms / steps] + [region(steps) / steps for _ in range(repeats)])
    # per-kernel times: the same steps with the library's HIP events.  With
    # several micro-batches the events of overlapping streams would include
    # each other's kernels, so this pass submits a step's micro-batches one
    # after another on one stream (kernel rates only; the step time above is
    # the overlapped one).
    C.moe_stage_profile(stage.handle, True)
    for s in range(steps):
        if n_micro == 1:
            step(s)
        else:
            for m in mbs[s % n_sets]:
                stage.submit(m, main)
    stage.sync()
    torch.cuda.synchronize()
    prof = C.moe_stage_profile_read(stage.handle)
    C.moe_stage_profile(stage.handle, False)
    stage.close()

    acct = None
    n_local, n_tok_local = 0, 0
    for mb in mbs_in:
        counts = np.bincount(mb.ids[(mb.ids >= 0)].ravel(), minlength=cfg.E)
        counts_local = counts[cfg.e0:cfg.e0 + cfg.E_loc]
        local = (mb.ids >= cfg.e0) & (mb.ids < cfg.e0 + cfg.E_loc)
        a = gemm_accounting(cfg, counts_local, mb.ids.shape[0])
        a.update(stream_accounting(cfg, counts_local, int(np.count_nonzero(local.any(axis=1))),
                                   mb.ids.shape[0]))
        acct = a if acct is None else {k: acct[k] + a[k] for k in acct}
        n_local += int(counts_local.sum())
    # per-step totals (a kernel group runs once per micro-batch)
    kern = {k: (v[0] / steps if v[1] else None) for k, v in prof.items()}
    del w, mbs_in, sets
    torch.cuda.empty_cache()
    return dict(cfg=cfg, T=sum(Ts), Ts=Ts, ms=ms, steps=steps, kern=kern, acct=acct,
                n_local_slots=n_local, n_micro=n_micro,
                spread={"p10": round(float(np.percentile(spread, 10)), 4),
                        "p50": round(float(np.percentile(spread, 50)), 4),
                        "p90": round(float(np.percentile(spread, 90)), 4),
                        "regions": len(spread)})


def measured_traffic(workload, kernel, fp8=False):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or
    None when it is missing or the kernel's sources changed since."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if fp8 and kernel.startswith("gemm_"):
        kernel += "_fp8"
    try:
        from paper_2606_22541_amd.profiling import sources_digest
        rec = json.load(open(path))["kernels"]["%s:%s" % (workload, kernel)]
        if rec["source_sha256"] != sources_digest(kernel):
            return None
        return rec["bytes_per_dispatch"]
    except Exception:
        return None


STEP_GROUPS = ("dispatch_index", "gather", "gemm_gate_up_swiglu", "gemm_down", "combine")


def step_roofline(r):
    """Roofline of a whole step of a multi-micro-batch workload, whose
    micro-batches overlap on their own streams: the step's algorithmic FLOPs
    (both grouped GEMMs) and bytes (every kernel group) over the measured
    step time.  `traffic` sums the counters' bytes per dispatch of each
    kernel group times the micro-batches of a step (null unless every group
    has a current record)."""
    a = r["acct"]
    ms = r["ms"] / r["steps"]
    fp8 = r["cfg"].dtype == "fp8"
    flop = a["g1_flop"] + a["g2_flop"]
    byts = a["g1_bytes"] + a["g2_bytes"] + a["index_bytes"] + a["combine_bytes"] + (
        a["gather_bytes"] if fp8 else 0)
    peak_tf = PEAK_FP8_TFLOPS if fp8 else PEAK_BF16_TFLOPS
    traffic = 0
    for k in STEP_GROUPS:
        if k == "gather" and not fp8:
            continue
        t = measured_traffic(r["cfg"].name, k, fp8)
        if t is None:
            traffic = None
            break
        traffic += t * r["n_micro"]
    base = {"kernel": "step: every kernel of the step's %d micro-batches, overlapped on %d streams"
                      % (r["n_micro"], r["n_micro"]),
            "traffic": traffic, "algorithmic_flop": flop, "algorithmic_bytes": byts,
            "avg_ms": round(ms, 4), "tflops": round(flop / (ms / 1e3) / 1e12, 1),
            "achieved_GBs": round(byts / (ms / 1e3) / 1e9, 1),
            "floor_ms": round(max(flop / (peak_tf * 1e12), byts / (PEAK_HBM_GBS * 1e9)) * 1e3, 4)}
    if flop / (peak_tf * 1e12) >= byts / (PEAK_HBM_GBS * 1e9):
        ach = flop / (ms / 1e3) / 1e12
        base.update(bound="mfma", achieved=round(ach, 1), peak=peak_tf, unit="TFLOP/s",
                    frac=round(ach / peak_tf, 4))
    else:
        ach = byts / (ms / 1e3) / 1e9
        base.update(bound="hbm", achieved=round(ach, 1), peak=PEAK_HBM_GBS, unit="GB/s",
                    frac=round(ach / PEAK_HBM_GBS, 4))
    return base


def roofline_for(r, kernel="gemm_gate_up_swiglu"):
    """Roofline of one launch of `kernel` (per step when the step has one
    micro-batch; summed over the step's micro-batches otherwise)."""
    a = r["acct"]
    t = r["kern"][kernel] / 1e3
    flop, byts = (a["g1_flop"], a["g1_bytes"]) if kernel == "gemm_gate_up_swiglu" else (
        a["g2_flop"], a["g2_bytes"])
    fp8 = r["cfg"].dtype == "fp8"
    peak_tf = PEAK_FP8_TFLOPS if fp8 else PEAK_BF16_TFLOPS
    t_mfma = flop / (peak_tf * 1e12)
    t_hbm = byts / (PEAK_HBM_GBS * 1e9)
    if t_mfma >= t_hbm:
        ach = flop / t / 1e12
        return {"kernel": kernel, "bound": "mfma", "achieved": round(ach, 1), "peak": peak_tf,
                "unit": "TFLOP/s", "frac": round(ach / peak_tf, 4),
                "traffic": measured_traffic(r["cfg"].name, kernel, fp8),
                "algorithmic_flop": flop, "algorithmic_bytes": byts, "avg_ms": round(t * 1e3, 4)}
    ach = byts / t / 1e9
    return {"kernel": kernel, "bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS,
            "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBS, 4),
            "traffic": measured_traffic(r["cfg"].name, kernel, fp8),
            "algorithmic_flop": flop, "algorithmic_bytes": byts, "avg_ms": round(t * 1e3, 4),
            "tflops": round(flop / t / 1e12, 1)}


def stream_rooflines(r):
    """Per-step time of each kernel group (summed over the step's micro-batches,
    which the profiling pass runs one after another on one stream) against its
    algorithmic bytes or FLOPs."""
    a = r["acct"]
    peak_tf = PEAK_FP8_TFLOPS if r["cfg"].dtype == "fp8" else PEAK_BF16_TFLOPS
    g1k, g2k = "gemm_gate_up_swiglu", "gemm_down"
    out = {}
    for k, b in (("gather", a["gather_bytes"]), ("combine", a["combine_bytes"])):
        t = r["kern"].get(k)
        if t:
            gbs = b / (t / 1e3) / 1e9
            out[k] = {"avg_ms": round(t, 4), "algorithmic_bytes": b, "achieved_GBs": round(gbs, 1),
                      "frac_hbm": round(gbs / PEAK_HBM_GBS, 4)}
            if k == "gather":
                # the fp8 token scales only (a few MB): launch and memory latency
                out[k]["bound"] = "latency"
    g1, g2 = r["kern"][g1k], r["kern"][g2k]
    out[g1k] = {"avg_ms": round(g1, 4), "tflops": round(a["g1_flop"] / (g1 / 1e3) / 1e12, 1)}
    out[g2k] = {"avg_ms": round(g2, 4), "tflops": round(a["g2_flop"] / (g2 / 1e3) / 1e12, 1)}
    tot = (a["g1_flop"] + a["g2_flop"]) / ((g1 + g2) / 1e3) / 1e12
    out["grouped_gemm_total"] = {"tflops": round(tot, 1), "frac_mfma": round(tot / peak_tf, 4),
                                 "peak_tflops": peak_tf}
    if r["kern"].get("quantize_h"):
        out["quantize_h"] = {"avg_ms": round(r["kern"]["quantize_h"], 4)}
    t = r["kern"]["dispatch_index"]
    gbs = a["index_bytes"] / (t / 1e3) / 1e9
    # a few hundred KB per micro-batch: launch and memory latency, not bandwidth
    out["dispatch_index"] = {"avg_ms": round(t, 4), "algorithmic_bytes": a["index_bytes"],
                             "achieved_GBs": round(gbs, 1), "frac_hbm": round(gbs / PEAK_HBM_GBS, 4),
                             "bound": "latency"}
    return out


WORKLOAD_TEXT = {
    "c1": "DeepSeek-V3 EP32 expert share, T=%(T)d tokens, d=%(d)d, f=%(f)d, %(El)d of %(E)d "
          "experts local, top-%(k)d, bf16",
    "c1p": "the c1 share at T=%(T)d (about %(per)d token-slots per local expert), bf16",
    "c2": "c1 shapes, %(n)d micro-batches of lognormal lengths %(Ts)s on %(n)d streams, "
          "Zipf(1.2) routing, two dead local experts, bf16",
    "c3": "EP8 share, T=%(T)d, %(El)d of %(E)d experts local plus one shared expert, bf16",
    "c4": "c2 in fp8 (e4m3 with 128-block scales), %(n)d micro-batches %(Ts)s on %(n)d streams",
    "c1p_fp8": "the c1p share in fp8 (e4m3 with 128-block scales), T=%(T)d",
    "c3_fp8": "the c3 share in fp8 (e4m3 with 128-block scales), T=%(T)d, %(El)d of %(E)d experts "
              "local plus one shared expert",
}


def describe(r):
    c = r["cfg"]
    return "%s: " % c.name + WORKLOAD_TEXT.get(c.name, "%(T)d tokens") % dict(
        T=r["T"], d=c.d, f=c.f, El=c.E_loc, E=c.E, k=c.k, n=r["n_micro"], Ts=r["Ts"],
        per=r["n_local_slots"] // c.E_loc)


def secondary_result(name, steps, warmup):
    """One further workload's entry of the JSON line."""
    sec = run_workload(name, steps, warmup)
    out = {
        "workload": describe(sec),
        "tokens_per_step": sec["T"],
        "tokens_per_s": round(sec["T"] * sec["steps"] / (sec["ms"] / 1e3), 1),
        "ms_per_step": round(sec["ms"] / sec["steps"], 4),
        "spread_ms_per_step": sec["spread"],
    }
    if sec["n_micro"] > 1:
        # overlapping streams: the roofline is the step's; kernel rates
        # come from a pass with the micro-batches one after another
        out["roofline"] = step_roofline(sec)
        out["kernels_serialized"] = stream_rooflines(sec)
        out["hw_queues"] = os.environ.get("GPU_MAX_HW_QUEUES", "runtime default")
    else:
        out["roofline"] = roofline_for(sec)
        out["kernels"] = stream_rooflines(sec)
    return out


# The HIP runtime maps a process's streams onto GPU_MAX_HW_QUEUES hardware
# queues (4 unless set), and two streams on one queue run one after the other.
# With 4 queues the four streams of a multi-micro-batch workload (c2, c4) share
# queues in a fresh process (c2 1.31 ms, c4 0.712 ms a step); with 8 they get
# one each (1.10 and 0.615 ms on the same box).  Such workloads are measured
# in a process started with MULTI_STREAM_QUEUES queues; single-stream ones keep
# the environment's setting (with 32 queues, single-stream timings showed
# stalls of a few hundred microseconds).
MULTI_STREAM_QUEUES = 8


def multi_stream(name):
    """True when the workload runs several micro-batches on streams of their own."""
    from paper_2606_22541_amd import inputs
    c = inputs.CONFIGS[name]
    return (len(c.lengths) if c.lengths is not None else c.n_micro) > 1
# GPU_MAX_HW_QUEUES as the process found it
_ENV_HW_QUEUES = os.environ.get("GPU_MAX_HW_QUEUES")


def _env_with_queues(n):
    env = dict(os.environ)
    if n is None:
        env.pop("GPU_MAX_HW_QUEUES", None)
    else:
        env["GPU_MAX_HW_QUEUES"] = str(n)
    return env


def run_secondary_child(name, steps, warmup, queues):
    """A multi-stream workload in a fresh process with `queues` hardware queues."""
    r = subprocess.run([sys.executable, os.path.abspath(__file__), "--workload-child", name,
                        "--steps", str(steps), "--warmup", str(warmup),
                        "--multi-stream-queues", str(queues)],
                       capture_output=True, text=True, timeout=600, env=_env_with_queues(queues))
    if r.returncode != 0:
        raise RuntimeError("workload %s child failed: %s" % (name, r.stderr.strip()[-2000:]))
    return json.loads(r.stdout.strip().splitlines()[-1])


def run_pipelined(name="c1", n_streams=3, steps=40, warmup=30, repeats=3):
    """Throughput of a stream of micro-batches of workload `name` with up to
    n_streams of them in flight: micro-batch i is submitted on stream
    i % n_streams (per-micro-batch streams, section 3.4.1), consecutive ones
    are not joined, and the slot ring's device-side waits are the only
    dependency between them.  Returns the best of `repeats` timed regions."""
    import torch
    from paper_2606_22541_amd import inputs
    from paper_2606_22541_amd.stage import ExpertStage, to_device_routing

    cfg = inputs.CONFIGS[name]
    w = inputs.make_weights(cfg, "cuda")
    mb = inputs.make_microbatches(cfg, "cuda")[0]
    T = mb.ids.shape[0]
    ids, wt = to_device_routing(mb.ids, mb.w)
    nb = n_streams + 1                       # distinct input/output buffer sets
    xs = [mb.x.clone() for _ in range(nb)]
    outs = [torch.empty((T, cfg.d), dtype=torch.bfloat16, device="cuda") for _ in range(nb)]
    stage = ExpertStage(cfg, w, n_slots=nb, max_tokens=T)
    del w
    mbs = [stage.microbatch(xs[i], ids, wt, outs[i]) for i in range(nb)]
    main = torch.cuda.Stream()
    streams = [torch.cuda.Stream() for _ in range(n_streams)]
    torch.cuda.synchronize()

    def run(n):
        go = torch.cuda.Event()
        go.record(main)
        for st_ in streams:
            st_.wait_event(go)
        for i in range(n):
            stage.submit(mbs[i % nb], streams[i % n_streams])
        for st_ in streams:
            e = torch.cuda.Event()
            e.record(st_)
            main.wait_event(e)

    run(warmup)
    stage.sync()
    torch.cuda.synchronize()
    best = None
    for _ in range(repeats):
        start = torch.cuda.Event(enable_timing=True)
        end = torch.cuda.Event(enable_timing=True)
        start.record(main)
        run(steps)
        end.record(main)
        stage.sync()
        torch.cuda.synchronize()
        ms = start.elapsed_time(end) / steps
        best = ms if best is None else min(best, ms)
    stage.close()
    return {"workload": "%s micro-batches (T=%d) submitted round-robin on %d streams, up to %d in "
                        "flight" % (name, T, n_streams, n_streams),
            "streams": n_streams, "ms_per_microbatch": round(best, 4),
            "tokens_per_s": round(T / (best / 1e3), 1)}


def run_triple_stream(name="c1", in_flight=3, steps=40, warmup=30, repeats=3):
    """The paper's three-stream layout on one GPU: dispatch on one stream,
    the grouped GEMMs on a compute stream, the combine on a third, each
    micro-batch's steps chained by events and slot reuse guarded by the
    slot's last combine, so one micro-batch's dispatch and combine run
    beside another's GEMMs.  Returns the best of `repeats` timed regions."""
    import torch
    from paper_2606_22541_amd import inputs
    from paper_2606_22541_amd.stage import ExpertStage, to_device_routing

    cfg = inputs.CONFIGS[name]
    w = inputs.make_weights(cfg, "cuda")
    mb = inputs.make_microbatches(cfg, "cuda")[0]
    T = mb.ids.shape[0]
    ids, wt = to_device_routing(mb.ids, mb.w)
    nb = in_flight + 1
    xs = [mb.x.clone() for _ in range(nb)]
    outs = [torch.empty((T, cfg.d), dtype=torch.bfloat16, device="cuda") for _ in range(nb)]
    stage = ExpertStage(cfg, w, n_slots=nb, max_tokens=T)
    del w
    mbs = [stage.microbatch(xs[i], ids, wt, outs[i]) for i in range(nb)]
    main = torch.cuda.Stream()
    D, G, R = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
    slot_done = [None] * nb

    def run(n):
        go = torch.cuda.Event()
        go.record(main)
        for st_ in (D, G, R):
            st_.wait_event(go)
        for i in range(n):
            k = i % nb
            if slot_done[k] is not None:
                D.wait_event(slot_done[k])
            stage.dispatch(k, mbs[k], D)
            e1 = torch.cuda.Event()
            e1.record(D)
            G.wait_event(e1)
            stage.expert_ffn(k, G)
            e2 = torch.cuda.Event()
            e2.record(G)
            R.wait_event(e2)
            stage.combine(k, R)
            e3 = torch.cuda.Event()
            e3.record(R)
            slot_done[k] = e3
        e = torch.cuda.Event()
        e.record(R)
        main.wait_event(e)

    run(warmup)
    torch.cuda.synchronize()
    best = None
    for _ in range(repeats):
        start = torch.cuda.Event(enable_timing=True)
        end = torch.cuda.Event(enable_timing=True)
        start.record(main)
        run(steps)
        end.record(main)
        torch.cuda.synchronize()
        ms = start.elapsed_time(end) / steps
        best = ms if best is None else min(best, ms)
    stage.sync()
    torch.cuda.synchronize()
    stage.close()
    return {"workload": "%s micro-batches (T=%d), dispatch / grouped GEMMs / combine on three "
                        "streams, up to %d micro-batches in flight" % (name, T, nb),
            "ms_per_microbatch": round(best, 4), "tokens_per_s": round(T / (best / 1e3), 1)}


# CU partitions of the three-stream layout (section 3.4.1 gives compute and
# each communication stream its own share of the cores): name -> per stream
# (first CU, CU count) as a function of the device's CU count.
CU_PARTITIONS = {
    "all_cus": lambda n: {"dispatch": (0, n), "gemm": (0, n), "combine": (0, n)},
    "split16": lambda n: {"dispatch": (0, 16), "combine": (16, 16), "gemm": (32, n - 32)},
    "split32": lambda n: {"dispatch": (0, 32), "combine": (32, 32), "gemm": (64, n - 64)},
    "gemm_all_16": lambda n: {"dispatch": (0, 16), "combine": (16, 16), "gemm": (0, n)},
}


def run_cu_partition_child(partition, name="c1", in_flight=3, steps=40, warmup=30, repeats=3):
    """The three-stream layout of run_triple_stream on CU-masked streams, in
    a process where nothing else created a stream: each masked stream takes
    a hardware queue of its own (the runtime gives a process four), so the
    three are created first, through the library, and torch's work stays on
    the null stream (events reach the masked streams through ExternalStream
    wrappers)."""
    import torch
    from paper_2606_22541_amd import inputs
    from paper_2606_22541_amd import moe_stage as C
    from paper_2606_22541_amd.stage import ExpertStage, to_device_routing

    cus = torch.cuda.get_device_properties(0).multi_processor_count
    C.load_library()
    parts = CU_PARTITIONS[partition](cus)
    hs = {k: C.moe_stream_create_cu_masked(*v) for k, v in parts.items()}
    D, G, R = (torch.cuda.ExternalStream(hs[k]) for k in ("dispatch", "gemm", "combine"))
    main = torch.cuda.current_stream()
    cfg = inputs.CONFIGS[name]
    w = inputs.make_weights(cfg, "cuda")
    mb = inputs.make_microbatches(cfg, "cuda")[0]
    T = mb.ids.shape[0]
    ids, wt = to_device_routing(mb.ids, mb.w)
    nb = in_flight + 1
    xs = [mb.x.clone() for _ in range(nb)]
    outs = [torch.empty((T, cfg.d), dtype=torch.bfloat16, device="cuda") for _ in range(nb)]
    stage = ExpertStage(cfg, w, n_slots=nb, max_tokens=T)
    del w
    mbs = [stage.microbatch(xs[i], ids, wt, outs[i]) for i in range(nb)]
    slot_done = [None] * nb
    torch.cuda.synchronize()

    def run(n):
        go = torch.cuda.Event()
        go.record(main)
        for st_ in (D, G, R):
            st_.wait_event(go)
        for i in range(n):
            k = i % nb
            if slot_done[k] is not None:
                D.wait_event(slot_done[k])
            stage.dispatch(k, mbs[k], hs["dispatch"])
            e1 = torch.cuda.Event()
            e1.record(D)
            G.wait_event(e1)
            stage.expert_ffn(k, hs["gemm"])
            e2 = torch.cuda.Event()
            e2.record(G)
            R.wait_event(e2)
            stage.combine(k, hs["combine"])
            e3 = torch.cuda.Event()
            e3.record(R)
            slot_done[k] = e3
        e = torch.cuda.Event()
        e.record(R)
        main.wait_event(e)

    run(warmup)
    torch.cuda.synchronize()
    best = None
    for _ in range(repeats):
        start = torch.cuda.Event(enable_timing=True)
        end = torch.cuda.Event(enable_timing=True)
        start.record(main)
        run(steps)
        end.record(main)
        torch.cuda.synchronize()
        ms = start.elapsed_time(end) / steps
        best = ms if best is None else min(best, ms)
    stage.sync()
    torch.cuda.synchronize()
    stage.close()
    for h in hs.values():
        C.moe_stream_destroy(h)
    return {"partition": partition,
            "cus": {k: list(v) for k, v in parts.items()},
            "ms_per_microbatch": round(best, 4), "tokens_per_s": round(T / (best / 1e3), 1)}


def run_cu_partition(name="c1", partitions=("all_cus", "split16", "split32", "gemm_all_16")):
    """CU-partitioned three-stream layouts, each measured in a child process
    of its own (a fresh budget of hardware queues)."""
    res = []
    for part in partitions:
        # the children keep the environment's hardware-queue count (each
        # masked stream takes a queue of its own; the layouts were measured so)
        r = subprocess.run([sys.executable, os.path.abspath(__file__), "--cu-partition-child", part,
                            "--workload", name, "--multi-stream-queues", "0"], capture_output=True,
                           text=True, timeout=300, env=_env_with_queues(_ENV_HW_QUEUES))
        if r.returncode != 0:
            res.append({"partition": part, "error": r.stderr.strip().splitlines()[-1:]})
            continue
        res.append(json.loads(r.stdout.strip().splitlines()[-1]))
        _log("[bench] cu partition %s done" % part)
    return {"workload": "%s micro-batches, dispatch / grouped GEMMs / combine on three CU-masked "
                        "streams, up to 4 micro-batches in flight" % name, "layouts": res}


def run_ingest(name="c1", senders=4, rounds=20, warmup=5):
    """Asynchronous ingest (section 3.2.1): each round, `senders` senders copy
    their share of a micro-batch (token rows, ids, weights) into the stage's
    receive buffers and raise their ready words; the stage round waits for
    them, runs, and acknowledges, and the next round's senders wait for that
    acknowledgement before overwriting the buffers.
      device-gated: both waits happen on the device (moe_ingest_wait /
        moe_ingest_signal); the host enqueues every round without blocking;
      host-gated: the host learns of each step's completion by synchronising
        on an event before it enqueues the next.
    Returns ms per round for both and their difference."""
    import torch
    from paper_2606_22541_amd import inputs
    from paper_2606_22541_amd import moe_stage as C
    from paper_2606_22541_amd.stage import ExpertStage, to_device_routing

    cfg = inputs.CONFIGS[name]
    w = inputs.make_weights(cfg, "cuda")
    mb = inputs.make_microbatches(cfg, "cuda")[0]
    T = mb.ids.shape[0]
    per = T // senders
    sids, sw = to_device_routing(mb.ids, mb.w)
    x = torch.empty_like(mb.x)                 # receive buffers
    ids = torch.empty_like(sids)
    wt = torch.empty_like(sw)
    out = torch.empty((T, cfg.d), dtype=torch.bfloat16, device="cuda")
    ready = torch.zeros(senders, dtype=torch.int32, device="cuda")
    consumed = torch.zeros(1, dtype=torch.int32, device="cuda")
    stage = ExpertStage(cfg, w, n_slots=2, max_tokens=T)
    del w
    m = stage.microbatch(x, ids, wt, out)
    prod, cons, main = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    epoch = [0]

    def send(r):
        with torch.cuda.stream(prod):
            for g in range(senders):
                sl = slice(g * per, (g + 1) * per)
                x[sl].copy_(mb.x[sl], non_blocking=True)
                ids[sl].copy_(sids[sl], non_blocking=True)
                wt[sl].copy_(sw[sl], non_blocking=True)
                C.moe_ingest_signal(ready[g:g + 1], r, prod)

    def device_gated(n):
        for _ in range(n):
            r = epoch[0] = epoch[0] + 1
            C.moe_ingest_wait(stage.handle, consumed, 1, r - 1, 0, prod)
            send(r)
            C.moe_ingest_wait(stage.handle, ready, senders, r, 0, cons)
            stage.submit(m, cons)
            C.moe_ingest_signal(consumed, r, cons)

    def host_gated(n):
        for _ in range(n):
            r = epoch[0] = epoch[0] + 1
            send(r)
            e = torch.cuda.Event()
            e.record(prod)
            e.synchronize()                    # the host learns the rows have arrived
            stage.submit(m, cons)
            C.moe_ingest_signal(consumed, r, cons)
            e2 = torch.cuda.Event()
            e2.record(cons)
            e2.synchronize()                   # ... and that the buffers are free again

    res = {}
    for label, fn in (("device_gated", device_gated), ("host_gated", host_gated)):
        fn(warmup)
        stage.sync()
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record(main)
        prod.wait_stream(main)
        cons.wait_stream(main)
        fn(rounds)
        main.wait_stream(cons)
        t1.record(main)
        stage.sync()
        torch.cuda.synchronize()
        res[label] = t0.elapsed_time(t1) / rounds
    stage.sync()
    stage.close()
    return {"workload": "%s micro-batch (T=%d) from %d senders of %d tokens through one set of "
                        "receive buffers, %d rounds" % (name, T, senders, per, rounds),
            "ms_per_round_device_gated": round(res["device_gated"], 4),
            "ms_per_round_host_gated": round(res["host_gated"], 4),
            "host_gating_us_per_round": round((res["host_gated"] - res["device_gated"]) * 1e3, 1)}


def run_grouped(name="c1", steps=40, warmup=20, repeats=3):
    """The pre-grouped input path (moe_expert_ffn_grouped): the micro-batch's
    local (token, expert) rows laid out grouped by expert before the timed
    region (torch ops), the per-expert counts in device memory; each step is
    one moe_expert_ffn_grouped call (tile tables from the counts, then the two
    grouped GEMMs).  Returns ms per call (median of `repeats` regions)."""
    import torch
    from paper_2606_22541_amd import inputs
    from paper_2606_22541_amd.stage import ExpertStage, to_device_routing

    cfg = inputs.CONFIGS[name]
    w = inputs.make_weights(cfg, "cuda")
    mb = inputs.make_microbatches(cfg, "cuda")[0]
    T = mb.ids.shape[0]
    ids, _ = to_device_routing(mb.ids, mb.w)
    flat = ids.reshape(-1).to(torch.int64)
    local = torch.nonzero((flat >= cfg.e0) & (flat < cfg.e0 + cfg.E_loc)).squeeze(1)
    key = flat[local] - cfg.e0
    order = torch.sort(key, stable=True).indices
    rows = mb.x[local[order] // cfg.k].contiguous()
    counts = torch.bincount(key, minlength=cfg.E_loc).to(torch.int32)
    y = torch.empty((rows.shape[0], cfg.d), dtype=torch.bfloat16, device="cuda")
    stage = ExpertStage(cfg, w, n_slots=1, max_tokens=T)
    del w
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    times = []
    for rep in range(repeats + 1):
        n = warmup if rep == 0 else steps
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record(s)
        for _ in range(n):
            stage.expert_ffn_grouped(0, rows, counts, y, stream=s)
        t1.record(s)
        t1.synchronize()
        if rep:
            times.append(t0.elapsed_time(t1) / n)
    stage.sync()
    stage.close()
    times.sort()
    return {"workload": "%s micro-batch (T=%d) as %d pre-grouped rows with device-side per-expert "
                        "counts, one moe_expert_ffn_grouped call per step" % (name, T, rows.shape[0]),
            "ms_per_call": round(times[len(times) // 2], 4),
            "rows_per_s": round(rows.shape[0] / (times[len(times) // 2] / 1e3), 1)}


SWEEP_TOKENS = (512, 1024, 2048, 4096, 8192, 12288, 16384, 24576, 32768)


def sweep_knee(pts, rise=1.5, linear_from=8192):
    """(knee tokens or None, ms per token of the linear regime or None) of a
    latency-vs-tokens sweep [{"T", "ms"}, ...] in increasing T."""
    T = np.array([p["T"] for p in pts], np.float64)
    ms = np.array([p["ms"] for p in pts], np.float64)
    knee = None
    lim = rise * ms[0]
    for i in range(1, len(pts)):
        if ms[i] > lim:
            knee = T[i - 1] + (lim - ms[i - 1]) / (ms[i] - ms[i - 1]) * (T[i] - T[i - 1])
            break
    sel = T >= linear_from
    slope = float(np.polyfit(T[sel], ms[sel], 1)[0]) if np.count_nonzero(sel) >= 2 else None
    return knee, slope


def run_sweep(tokens=SWEEP_TOKENS, steps=10, warmup=5):
    """MoE-stage latency against micro-batch size for the c1 expert share
    (7168 x 2048, 8 of 256 experts local, top-8, uniform routing, bf16): the
    single-GPU analog of the paper's latency-vs-tokens curve under perfect
    balance, which is flat while the weights' HBM stream dominates and turns
    linear once the grouped GEMM is MFMA-bound.  The flat region ends (the
    knee) where the latency first exceeds 1.5 times the smallest batch's,
    interpolated linearly between measured sizes; the marginal cost is the
    least-squares slope over the sizes from 8192 tokens up."""
    import torch
    from paper_2606_22541_amd import inputs
    from paper_2606_22541_amd.stage import ExpertStage, to_device_routing

    cfg = inputs.CONFIGS["c1"]
    w = inputs.make_weights(cfg, "cuda")
    stage = ExpertStage(cfg, w, n_slots=2, max_tokens=max(tokens))
    del w
    main = torch.cuda.Stream()
    pts = []
    for T in tokens:
        c = inputs.scaled(cfg, name="c1_T%d" % T, lengths=(T,))
        mb = inputs.make_microbatches(c, "cuda")[0]
        ids, wt = to_device_routing(mb.ids, mb.w)
        outs = [torch.empty((T, cfg.d), dtype=torch.bfloat16, device="cuda") for _ in range(2)]
        mbs = [stage.microbatch(mb.x, ids, wt, o) for o in outs]
        torch.cuda.synchronize()
        for i in range(warmup):
            stage.submit(mbs[i % 2], main)
        stage.sync()
        torch.cuda.synchronize()
        start = torch.cuda.Event(enable_timing=True)
        end = torch.cuda.Event(enable_timing=True)
        start.record(main)
        for i in range(steps):
            stage.submit(mbs[i % 2], main)
        end.record(main)
        stage.sync()
        torch.cuda.synchronize()
        ms = start.elapsed_time(end) / steps
        local = int(np.count_nonzero((mb.ids >= cfg.e0) & (mb.ids < cfg.e0 + cfg.E_loc)))
        pts.append({"T": T, "ms": round(ms, 4), "us_per_token": round(ms * 1e3 / T, 4),
                    "rows_per_expert": round(local / cfg.E_loc, 1)})
        del mbs, outs
    stage.close()
    knee, slope = sweep_knee(pts)
    return {"workload": "c1 expert share at T tokens (d=7168, f=2048, 8 of 256 experts local, "
                        "top-8, uniform, bf16)",
            "points": pts,
            "knee_tokens": round(knee) if knee else None,
            "knee_rows_per_expert": round(knee * cfg.k / cfg.E) if knee else None,
            "ms_per_1k_tokens_linear": round(slope * 1e3, 4) if slope else None}


def run_layers(n_layers, passes=3):
    """Layer-oblivious submission against host-in-the-loop dispatch, on one
    stage holding n_layers copies of the c1 expert share (7168 x 2048, 8
    local experts).  One pass submits one c1 micro-batch per layer, layers in
    a fixed shuffled order, each naming its layer through a device int32.
      device-resolved: every pass is enqueued ahead; the GEMM kernels pick the
        layer's weights from the on-device address table (no host in the loop);
      host-dispatched: before each layer the host learns which layer comes
        next by reading the id back from the device (which waits for the
        stream), then enqueues it -- the dispatch pattern whose per-layer
        latency the super kernel removes.
    Returns ms per layer for both and the GPU's idle time between one layer's
    end and the next layer's start (events around each submission); their
    difference is the per-layer host dispatch bubble.  (Per-layer times also
    differ through caching: idle gaps let earlier writes drain.)"""
    import torch
    from paper_2606_22541_amd import inputs
    from paper_2606_22541_amd.stage import ExpertStage, to_device_routing

    cfg = inputs.CONFIGS["c1"]
    w = inputs.make_weights(cfg, "cuda")
    mb = inputs.make_microbatches(cfg, "cuda")[0]
    T = mb.ids.shape[0]
    stage = ExpertStage(cfg, [w] * n_layers, n_slots=2, max_tokens=T)   # n_layers packed copies
    del w
    ids, wt = to_device_routing(mb.ids, mb.w)
    x = mb.x.clone()
    outs = [torch.empty((T, cfg.d), dtype=torch.bfloat16, device="cuda") for _ in range(2)]
    order = [int(l) for l in np.random.default_rng(0).permutation(n_layers)]
    lids = [torch.tensor([l], dtype=torch.int32, device="cuda") for l in order]
    mbs = [stage.microbatch(x, ids, wt, outs[i % 2], layer_id=lids[i]) for i in range(n_layers)]
    main = torch.cuda.Stream()
    torch.cuda.synchronize()

    def device_resolved(marks):
        for m in mbs:
            a = torch.cuda.Event(enable_timing=True)
            a.record(main)
            stage.submit(m, main)
            b = torch.cuda.Event(enable_timing=True)
            b.record(main)
            marks.append((a, b))

    def host_dispatched(marks):
        for i, m in enumerate(mbs):
            with torch.cuda.stream(main):
                assert int(lids[i].item()) == order[i]   # synchronising read of the layer id
            a = torch.cuda.Event(enable_timing=True)
            a.record(main)
            stage.submit(m, main)
            b = torch.cuda.Event(enable_timing=True)
            b.record(main)
            marks.append((a, b))

    res, gaps = {}, {}
    for name, fn in (("device_resolved", device_resolved), ("host_dispatched", host_dispatched)):
        fn([])                                         # warm-up pass
        stage.sync()
        torch.cuda.synchronize()
        marks = []
        for _ in range(passes):
            fn(marks)
        stage.sync()
        torch.cuda.synchronize()
        res[name] = (marks[0][0].elapsed_time(marks[-1][1])) / len(marks)
        # GPU idle time between one layer's end and the next layer's start
        g = [marks[i][1].elapsed_time(marks[i + 1][0]) for i in range(len(marks) - 1)]
        gaps[name] = float(np.mean(g)) * 1e3
    stage.close()
    return {
        "layers": n_layers,
        "workload": "c1 expert share (T=4096, d=7168, f=2048, 8 of 256 experts local, top-8, "
                    "bf16) x %d layers resident, layers in shuffled order" % n_layers,
        "ms_per_layer_device_resolved": round(res["device_resolved"], 4),
        "ms_per_layer_host_dispatched": round(res["host_dispatched"], 4),
        "gap_us_between_layers_device_resolved": round(gaps["device_resolved"], 1),
        "gap_us_between_layers_host_dispatched": round(gaps["host_dispatched"], 1),
        "host_bubble_us_per_layer": round(gaps["host_dispatched"] - gaps["device_resolved"], 1),
    }


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_once(name, threads=None):
    """Seconds for one oracle run of workload `name`'s first micro-batch,
    optionally with the BLAS pool limited to `threads`."""
    import oracle
    import torch
    from paper_2606_22541_amd import inputs
    cfg = inputs.CONFIGS[name]
    dev = "cuda" if torch.cuda.is_available() else "cpu"
    w = inputs.make_weights(cfg, dev)
    mb = inputs.make_microbatches(cfg, dev)[0]
    ow = oracle.OracleWeights(w, cfg.dtype)
    xb = mb.x.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)
    del w

    def run():
        t0 = time.time()
        oracle.run_stage(cfg, ow, xb, mb.ids, mb.w)
        return time.time() - t0
    if threads is None:
        return run(), mb.ids.shape[0]
    from threadpoolctl import threadpool_limits
    with threadpool_limits(limits=threads):
        return run(), mb.ids.shape[0]


def cpu_baseline(name="c1", min_seconds=10.0):
    """The CPU oracle on the full T=4096 micro-batch of the primary workload,
    on all of the host's BLAS threads; also c0 and c1 once on one thread."""
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
    res = {"value": round(T * runs / dt, 1), "unit": "tokens/s", "cores": int(threads),
           "kind": "oracle",
           "sample": "%d x the full %s micro-batch (T=%d, %d local slots), fp64, %.1f s wall" % (
               runs, name, T,
               int(np.count_nonzero((mb.ids >= cfg.e0) & (mb.ids < cfg.e0 + cfg.E_loc))), dt),
           "cpu_model": cpu_model(), "nproc": os.cpu_count(),
           "affinity_cpus": len(os.sched_getaffinity(0))}
    del ow, mb
    single = {}
    for wl in ("c0", name):
        try:
            sec, Tw = _oracle_once(wl, threads=1)
            single[wl] = {"tokens_per_s": round(Tw / sec, 1), "seconds": round(sec, 3),
                          "tokens": Tw}
        except Exception as e:          # threadpoolctl missing: report why
            single[wl] = {"error": repr(e)}
    res["single_thread"] = single
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--workload", default="c1")
    ap.add_argument("--secondary", default="c1p,c3,c2,c4",
                    help="comma-separated further workloads ('' for none)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--pipelined-streams", type=int, default=3,
                    help="also time the primary workload with this many micro-batches in flight "
                         "on separate streams (<= 1: skip)")
    ap.add_argument("--triple-stream", type=int, default=1,
                    help="also time the dispatch / GEMM / combine three-stream layout (0: skip)")
    ap.add_argument("--ingest", type=int, default=1,
                    help="also time device-gated against host-gated ingest (0: skip)")
    ap.add_argument("--grouped", type=int, default=1,
                    help="also time the pre-grouped input path on the primary workload (0: skip)")
    ap.add_argument("--no-sweep", action="store_true",
                    help="skip the latency-vs-tokens sweep of the c1 expert share")
    ap.add_argument("--layers", type=int, default=8,
                    help="layers for the layer-oblivious dispatch measurement (0: skip)")
    ap.add_argument("--cu-partition", type=int, default=1,
                    help="also time the three-stream layout on CU-masked streams (0: skip)")
    ap.add_argument("--cu-partition-child", default="",
                    help="internal: measure one CU partition in this (fresh) process and exit")
    ap.add_argument("--multi-stream-queues", type=int, default=MULTI_STREAM_QUEUES,
                    help="hardware queues (GPU_MAX_HW_QUEUES) of the processes that measure "
                         "multi-micro-batch workloads (0: the environment's, in this process)")
    ap.add_argument("--workload-child", default="",
                    help="internal: measure this workload in this (fresh) process and exit")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="only run a plain device copy of this many MiB (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU's expert share and runs on one GPU only (asked for %d); "
              "across GPUs the stage shards by expert, one process per GPU on its own experts."
              % args.gpus, file=sys.stderr)
        sys.exit(2)
    if args.multi_stream_queues > 0 and multi_stream(args.workload_child or args.workload):
        # set before HIP starts (the first CUDA call below)
        os.environ["GPU_MAX_HW_QUEUES"] = str(args.multi_stream_queues)
    import torch
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.workload_child:
        print(json.dumps(secondary_result(args.workload_child, args.steps, args.warmup)), flush=True)
        return
    if args.cu_partition_child:
        print(json.dumps(run_cu_partition_child(args.cu_partition_child, args.workload)), flush=True)
        return
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
        "config": {"workload": describe(prim), "tokens_per_step": prim["T"],
                   "local_slots": prim["n_local_slots"]},
        "spread_ms_per_step": prim["spread"],
        "roofline": roofline_for(prim),
        "kernels": stream_rooflines(prim),
    }
    _log("[bench] primary done: %.3f ms/step" % ms_step)
    # before the multi-stream workloads: their streams would share hardware
    # queues with the ingest measurement's sender and stage streams
    if args.ingest:
        line["%s_ingest" % args.workload] = run_ingest(args.workload)
        _log("[bench] ingest %s done" % args.workload)
    for name in [n for n in args.secondary.split(",") if n]:
        steps = max(args.steps // 2, 5)
        if args.multi_stream_queues > 0 and multi_stream(name):
            line[name] = run_secondary_child(name, steps, args.warmup, args.multi_stream_queues)
        else:
            line[name] = secondary_result(name, steps, args.warmup)
        _log("[bench] %s done" % name)
    if args.pipelined_streams > 1:
        line["%s_pipelined" % args.workload] = run_pipelined(args.workload, args.pipelined_streams)
        _log("[bench] pipelined %s done" % args.workload)
    if args.triple_stream:
        line["%s_triple_stream" % args.workload] = run_triple_stream(args.workload)
        _log("[bench] triple-stream %s done" % args.workload)
    if args.grouped:
        line["%s_grouped" % args.workload] = run_grouped(args.workload)
        _log("[bench] grouped %s done" % args.workload)
    if args.cu_partition:
        line["%s_cu_partition" % args.workload] = run_cu_partition(args.workload)
    if not args.no_sweep:
        line["token_sweep"] = run_sweep()
        _log("[bench] token sweep done")
    if args.layers > 0:
        line["layer_oblivious"] = run_layers(args.layers)
        _log("[bench] layer-oblivious dispatch done")
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(args.workload)
        _log("[bench] cpu baseline done")
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
