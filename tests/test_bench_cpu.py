"""Host logic of the measurement, on the CPU: the token-sweep knee, the
single-GPU guard of bench.py, and the reduction of MFMA counters."""
import csv
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2606_22541_amd import profiling  # noqa: E402


def _pts(f, Ts=(512, 1024, 2048, 4096, 8192, 16384, 32768)):
    return [{"T": T, "ms": f(T)} for T in Ts]


def test_sweep_knee_flat_then_linear():
    # flat at 0.2 ms up to 4096 tokens, then 0.05 ms per 1k tokens
    pts = _pts(lambda T: 0.2 if T <= 4096 else 0.2 + 0.05e-3 * (T - 4096))
    knee, slope = bench.sweep_knee(pts)
    # 1.5 x 0.2 = 0.3 ms is reached at 4096 + 0.1 / 0.05e-3 = 6096 tokens
    assert knee == pytest.approx(6096.0)
    assert slope == pytest.approx(0.05e-3)


def test_sweep_knee_never_rises():
    knee, slope = bench.sweep_knee(_pts(lambda T: 0.2))
    assert knee is None
    assert slope == pytest.approx(0.0, abs=1e-15)


def test_bench_refuses_several_gpus():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def _write_counters(path, kernel, ns, values):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name",
                                          "Counter_Value", "Start_Timestamp", "End_Timestamp"])
        w.writeheader()
        for disp in (1, 2):
            for name, v in values.items():
                w.writerow({"Dispatch_Id": disp, "Kernel_Name": kernel + "(moe::GemmArgs)",
                            "Counter_Name": name, "Counter_Value": v,
                            "Start_Timestamp": 1000, "End_Timestamp": 1000 + ns})


def test_mfma_util_reduction(tmp_path):
    # 1e6 bf16 MFMAs (32 busy cycles each) in 100 us, GRBM summed over 8 XCDs at 2.0 GHz
    ns = 100_000
    n = 1_000_000
    _write_counters(tmp_path / "run_counter_collection.csv", "void moe::k_gemm_bf16<true>", ns,
                    {"SQ_INSTS_MFMA": n, "SQ_VALU_MFMA_BUSY_CYCLES": 32 * n,
                     "GRBM_GUI_ACTIVE": 8 * 2.0 * ns, "SQ_BUSY_CU_CYCLES": 0})
    r = profiling.mfma_util(str(tmp_path))["void moe::k_gemm_bf16<true>"]
    assert r["dispatches"] == 2
    assert r["clock_ghz"] == pytest.approx(2.0)
    assert r["executed_tflops"] == pytest.approx(n * 32768 / ns / 1e3)
    # busy cycles over all 1024 SIMDs at 2.0 GHz for 100 us
    assert r["mfma_busy_at_clock"] == pytest.approx(32 * n / (1024 * 2.0 * ns))
    assert r["mfma_busy_at_peak_clock"] == pytest.approx(32 * n / (1024 * 2.4 * ns))
    assert r["busy_cycles_per_mfma"] == pytest.approx(32.0)


def test_fp8_mfma_counts_double_flop():
    assert profiling.flop_per_mfma("void moe::k_gemm_fp8<true, 8>") == 2 * profiling.flop_per_mfma(
        "void moe::k_gemm_bf16<true>")


def test_stream_accounting_bytes():
    """Algorithmic bytes: the dispatch index moves ids and index arrays; the
    fp8 gather moves the token scales (one fp32 per 128 channels), the e4m3
    rows being read by the gate/up GEMM."""
    import numpy as np
    from paper_2606_22541_amd import inputs
    T, U = 4096, 900
    counts = np.full(8, 132)
    n_loc = int(counts.sum())
    c1 = inputs.CONFIGS["c1"]
    a = bench.stream_accounting(c1, counts, U, T)
    assert a["index_bytes"] == T * 8 * 4 + 256 * 4 + 9 * 4 + (n_loc + T * 8) * 4
    assert a["combine_bytes"] == T * 8 * 12 + n_loc * 7168 * 2 + T * 7168 * 2
    f8 = inputs.CONFIGS["c4"]
    b = bench.stream_accounting(f8, counts, U, T)
    assert b["gather_bytes"] == (U + n_loc) * 56 * 4 + n_loc * 4


def test_step_roofline_of_overlapped_micro_batches():
    """Multi-stream workloads report the whole step: both GEMMs' FLOPs and
    every kernel group's bytes over the measured step time."""
    from paper_2606_22541_amd import inputs
    acct = dict(g1_flop=4e12, g2_flop=2e12, g1_bytes=1e9, g2_bytes=0.5e9, index_bytes=1e6,
                combine_bytes=2e8, gather_bytes=1e8)
    r = dict(cfg=inputs.CONFIGS["c2"], acct=acct, ms=40.0, steps=20, n_micro=4)
    ro = bench.step_roofline(r)
    # 6 TFLOP / 2 ms = 3000 TFLOP/s against bf16; MFMA time 2.4 ms > HBM time 0.21 ms
    assert ro["bound"] == "mfma" and ro["peak"] == bench.PEAK_BF16_TFLOPS
    assert ro["achieved"] == pytest.approx(3000.0)
    assert ro["frac"] == pytest.approx(1.2)
    assert ro["algorithmic_bytes"] == 1e9 + 0.5e9 + 1e6 + 2e8        # bf16: no gather kernel
    assert ro["floor_ms"] == pytest.approx(6e12 / 2.5e15 * 1e3)
    r8 = dict(r, cfg=inputs.CONFIGS["c4"])
    ro8 = bench.step_roofline(r8)
    assert ro8["peak"] == bench.PEAK_FP8_TFLOPS
    assert ro8["algorithmic_bytes"] == 1e9 + 0.5e9 + 1e6 + 2e8 + 1e8  # fp8 gathers the x scales


def test_cu_partitions_fit_the_device():
    """Every CU partition of the three-stream ablation lies inside the
    device's CUs; the split layouts give the three streams disjoint sets."""
    for n in (256, 304, 80):
        for name, f in bench.CU_PARTITIONS.items():
            parts = f(n)
            assert set(parts) == {"dispatch", "gemm", "combine"}
            for first, cnt in parts.values():
                assert 0 <= first and cnt >= 1 and first + cnt <= n
            if name.startswith("split"):
                sets = [set(range(a, a + c)) for a, c in parts.values()]
                assert not (sets[0] & sets[1]) and not (sets[0] & sets[2]) and not (sets[1] & sets[2])
