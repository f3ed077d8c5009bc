"""Summaries of rocprofv3 output for the stage's kernels.

``kernel_stats``: reduces a ``--kernel-trace --stats`` kernel_stats.csv to
the stage's kernels (calls, average and total duration).

``traffic``: turns two ``--pmc FETCH_SIZE`` / ``--pmc WRITE_SIZE`` runs of a
workload, plus the same two counters read for a plain device copy of known
size, into HBM bytes per dispatch of each kernel.  Each counter is scaled by
(known copy bytes / what the counter reported for the copy), so systematic
under- or over-counting of the counters cancels.

Usage:
  python -m paper_2606_22541_amd.profiling stats <kernel_stats.csv>
  python -m paper_2606_22541_amd.profiling traffic --workload c1 \\
      --fetch <counter_collection.csv> --write <counter_collection.csv> \\
      --copy-fetch <csv> --copy-write <csv> --copy-bytes N --out profiles/traffic.json
"""
from __future__ import annotations

import argparse
import collections
import csv
import glob
import hashlib
import json
import os
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
KERNEL_SOURCES = {
    "gemm_gate_up_swiglu": ["csrc/gemm_bf16.hip", "csrc/gemm_bf16_small.hip", "csrc/common.h",
                            "csrc/kernels.h"],
    "gemm_down": ["csrc/gemm_bf16.hip", "csrc/gemm_bf16_small.hip", "csrc/common.h",
                  "csrc/kernels.h"],
    "gemm_gate_up_swiglu_fp8": ["csrc/gemm_fp8.hip", "csrc/common.h", "csrc/kernels.h"],
    "gemm_down_fp8": ["csrc/gemm_fp8.hip", "csrc/common.h", "csrc/kernels.h"],
    "combine": ["csrc/combine.hip", "csrc/common.h", "csrc/kernels.h"],
    "gather": ["csrc/dispatch.hip", "csrc/common.h", "csrc/kernels.h"],
    "dispatch_index": ["csrc/dispatch.hip", "csrc/common.h", "csrc/kernels.h"],
}
# rocprof kernel-name prefixes of the stage's kernels -> the kernel groups
# bench.py times (a group's kernels each run once per micro-batch, so a
# group's per-step figure is the sum over its kernels)
NAME_MAP = (
    ("void moe::k_gemm_bf16_small<true>", "gemm_gate_up_swiglu"),
    ("void moe::k_gemm_bf16<true>", "gemm_gate_up_swiglu"),
    ("void moe::k_gemm_bf16<false>", "gemm_down"),
    ("void moe::k_gemm_bf16_small<false>", "gemm_down"),
    ("void moe::k_gemm_fp8<true>", "gemm_gate_up_swiglu_fp8"),
    ("void moe::k_gemm_fp8<false>", "gemm_down_fp8"),
    ("moe::k_combine", "combine"),
    ("moe::k_gather_scales", "gather"),
    ("moe::k_transpose_scales", "gather"),
    ("moe::k_hist", "dispatch_index"),
    ("moe::k_place", "dispatch_index"),
    ("moe::k_quantize_fp8", "quantize_fp8"),
)
COPY_NAMES = ("__amd_rocclr_copyBuffer",)


def sources_digest(kind: str) -> str:
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES.get(kind, []):
        with open(os.path.join(PKG, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def kind_of(name: str):
    for prefix, kind in NAME_MAP:
        if name.startswith(prefix):
            return kind
    return None


def _find_csv(path: str, suffix: str) -> str:
    if os.path.isdir(path):
        hits = glob.glob(os.path.join(path, "**", "*" + suffix), recursive=True)
        if not hits:
            raise FileNotFoundError("no *%s under %s" % (suffix, path))
        return hits[0]
    return path


def kernel_stats(path: str):
    """Per kernel group: calls of its first kernel and the summed average
    and total durations of its kernels."""
    rows = list(csv.DictReader(open(_find_csv(path, "kernel_stats.csv"))))
    out = {}
    for r in rows:
        k = kind_of(r["Name"])
        if not k:
            continue
        e = out.setdefault(k, {"calls": int(r["Calls"]), "avg_ms": 0.0, "total_ms": 0.0,
                               "kernels": []})
        e["avg_ms"] += float(r["AverageNs"]) / 1e6
        e["total_ms"] += float(r["TotalDurationNs"]) / 1e6
        e["kernels"].append(r["Name"].split("(")[0])
    return out


def counter_per_dispatch(path: str, counter: str):
    """Mean counter value per dispatch of each kernel, summed over the
    kernels of a group (copy kernels are their own group)."""
    rows = list(csv.DictReader(open(_find_csv(path, "counter_collection.csv"))))
    acc = collections.defaultdict(float)
    disp = collections.defaultdict(set)
    group = {}
    for r in rows:
        if r["Counter_Name"] != counter:
            continue
        name = r["Kernel_Name"]
        k = kind_of(name) or (name if name in COPY_NAMES else None)
        if k is None:
            continue
        key = name.split("(")[0]
        group[key] = k
        acc[key] += float(r["Counter_Value"])
        disp[key].add(r["Dispatch_Id"])
    out = collections.defaultdict(float)
    for key, k in group.items():
        out[k] += acc[key] / len(disp[key])
    return dict(out)


def traffic(args):
    fetch = counter_per_dispatch(args.fetch, "FETCH_SIZE")
    write = counter_per_dispatch(args.write, "WRITE_SIZE")
    cf = counter_per_dispatch(args.copy_fetch, "FETCH_SIZE")
    cw = counter_per_dispatch(args.copy_write, "WRITE_SIZE")
    copy = COPY_NAMES[0]
    # the largest copy dispatch is the calibration copy
    f_scale = args.copy_bytes / (cf[copy] * 1024.0)
    w_scale = args.copy_bytes / (cw[copy] * 1024.0)
    rec = json.load(open(args.out)) if os.path.exists(args.out) else {}
    rec.setdefault("kernels", {})
    rec["calibration"] = {"copy_bytes": args.copy_bytes, "fetch_kib": cf[copy],
                          "write_kib": cw[copy], "fetch_scale": f_scale, "write_scale": w_scale}
    for k in sorted(set(fetch) | set(write)):
        if k == copy:
            continue
        fb = fetch.get(k, 0.0) * 1024.0 * f_scale
        wb = write.get(k, 0.0) * 1024.0 * w_scale
        rec["kernels"]["%s:%s" % (args.workload, k)] = {
            "fetch_bytes_per_dispatch": round(fb), "write_bytes_per_dispatch": round(wb),
            "bytes_per_dispatch": round(fb + wb), "source_sha256": sources_digest(k)}
    rec.setdefault("commands", [])
    if args.command:
        rec["commands"].append(args.command)
    with open(args.out, "w") as f:
        json.dump(rec, f, indent=1, sort_keys=True)
    print(json.dumps(rec, indent=1, sort_keys=True))


def overlap(path: str, steps_skip: int, steps_use: int):
    """Per-step overlap of the stage's kernels in a --kernel-trace of a
    workload whose micro-batches run on their own streams.  The stage's
    dispatches, in issue order, are cut into steps of equal kernel count
    (every step issues the same kernels); of those, `steps_use` steps after
    the first `steps_skip` are reduced.  Per step: the span (first start to
    last end), the sum of kernel durations, the busy time of each stream
    (union of its kernels' intervals) and of the device (union of all), and
    the sum per kernel group.  overlap = sum of durations / device busy time
    (1: nothing ran concurrently)."""
    rows = [r for r in csv.DictReader(open(_find_csv(path, "kernel_trace.csv")))
            if kind_of(r["Kernel_Name"]) not in (None, "quantize_fp8")]
    rows.sort(key=lambda r: int(r["Dispatch_Id"]))
    streams = sorted({r["Stream_Id"] for r in rows})
    # kernels per step: the number of dispatches between consecutive
    # dispatches of the first kernel name seen on the first stream
    first = rows[0]["Kernel_Name"]
    idx = [i for i, r in enumerate(rows) if r["Kernel_Name"] == first and
           r["Stream_Id"] == rows[0]["Stream_Id"]]
    per_step = idx[1] - idx[0]

    def union(iv):
        iv = sorted(iv)
        tot, cur_s, cur_e = 0, None, None
        for s_, e_ in iv:
            if cur_e is None or s_ > cur_e:
                if cur_e is not None:
                    tot += cur_e - cur_s
                cur_s, cur_e = s_, e_
            else:
                cur_e = max(cur_e, e_)
        return tot + (cur_e - cur_s if cur_e is not None else 0)

    acc = collections.defaultdict(float)
    n = 0
    for st in range(steps_skip, steps_skip + steps_use):
        chunk = rows[st * per_step:(st + 1) * per_step]
        if len(chunk) < per_step:
            break
        iv = [(int(r["Start_Timestamp"]), int(r["End_Timestamp"])) for r in chunk]
        acc["span_us"] += (max(e for _, e in iv) - min(s_ for s_, _ in iv)) / 1e3
        acc["sum_kernels_us"] += sum(e - s_ for s_, e in iv) / 1e3
        acc["device_busy_us"] += union(iv) / 1e3
        for sid in streams:
            acc["stream_%s_busy_us" % sid] += union(
                [(int(r["Start_Timestamp"]), int(r["End_Timestamp"])) for r in chunk
                 if r["Stream_Id"] == sid]) / 1e3
        for r in chunk:
            acc["group_%s_us" % kind_of(r["Kernel_Name"])] += (
                int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        n += 1
    out = {k: round(v / n, 2) for k, v in acc.items()}
    out["steps"] = n
    out["kernels_per_step"] = per_step
    out["overlap"] = round(out["sum_kernels_us"] / out["device_busy_us"], 3)
    return out


# gfx950 MFMA accounting (checked against the kernels' own tile counts):
# SQ_INSTS_MFMA counts one per MFMA instruction a wave issues, and a
# v_mfma_f32_32x32x16_bf16 (32768 FLOP) adds 32 to SQ_VALU_MFMA_BUSY_CYCLES;
# both are summed over the 1024 SIMDs, and GRBM_GUI_ACTIVE over the 8 XCDs.
# The fp8 kernel issues v_mfma_scale_f32_16x16x128_f8f6f4 (65536 FLOP).
SIMDS = 1024
XCDS = 8
PEAK_CLOCK_GHZ = 2.4


def flop_per_mfma(kernel: str) -> int:
    return 65536 if "k_gemm_fp8" in kernel else 32768


def mfma_util(path: str):
    """Per GEMM kernel: mean over its dispatches of the duration, the clock
    (GRBM_GUI_ACTIVE per XCD over the duration), the MFMA instructions and
    FLOP executed, and the MFMA pipes' busy fraction at that clock and at
    the nominal 2.4 GHz."""
    rows = list(csv.DictReader(open(_find_csv(path, "counter_collection.csv"))))
    per = collections.defaultdict(dict)
    for r in rows:
        n = r["Kernel_Name"]
        if not n.startswith("void moe::k_gemm"):
            continue
        d = per[(n.split("(")[0], r["Dispatch_Id"])]
        d[r["Counter_Name"]] = float(r["Counter_Value"])
        d["ns"] = float(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
    by_kernel = collections.defaultdict(list)
    for (name, _), d in per.items():
        by_kernel[name].append(d)
    out = {}
    for name, ds in by_kernel.items():
        m = {k: sum(d.get(k, 0.0) for d in ds) / len(ds) for k in ds[0]}
        ns, gui = m["ns"], m["GRBM_GUI_ACTIVE"] / XCDS
        busy, n_mfma = m["SQ_VALU_MFMA_BUSY_CYCLES"], m["SQ_INSTS_MFMA"]
        out[name] = {
            "dispatches": len(ds),
            "avg_us": ns / 1e3,
            "clock_ghz": gui / ns if ns else 0.0,
            "mfma_per_dispatch": n_mfma,
            "busy_cycles_per_mfma": busy / n_mfma if n_mfma else 0.0,
            "executed_tflops": n_mfma * flop_per_mfma(name) / ns / 1e3 if ns else 0.0,
            "mfma_busy_at_clock": busy / (gui * SIMDS) if gui else 0.0,
            "mfma_busy_at_peak_clock": busy / (ns * PEAK_CLOCK_GHZ * SIMDS) if ns else 0.0,
        }
    return out


def main(argv=None):
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("path")
    t = sub.add_parser("traffic")
    t.add_argument("--workload", required=True)
    t.add_argument("--fetch", required=True)
    t.add_argument("--write", required=True)
    t.add_argument("--copy-fetch", required=True)
    t.add_argument("--copy-write", required=True)
    t.add_argument("--copy-bytes", type=int, required=True)
    t.add_argument("--out", required=True)
    t.add_argument("--command", default="")
    m = sub.add_parser("mfma")
    m.add_argument("path")
    o = sub.add_parser("overlap")
    o.add_argument("path")
    o.add_argument("--skip", type=int, default=20)
    o.add_argument("--use", type=int, default=120)
    a = ap.parse_args(argv)
    if a.cmd == "overlap":
        print(json.dumps(overlap(a.path, a.skip, a.use), indent=1, sort_keys=True))
    elif a.cmd == "stats":
        print(json.dumps(kernel_stats(a.path), indent=1, sort_keys=True))
    elif a.cmd == "mfma":
        print(json.dumps(mfma_util(a.path), indent=1, sort_keys=True))
    else:
        traffic(a)


if __name__ == "__main__":
    main()
