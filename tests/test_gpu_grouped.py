"""GPU parity of the pre-grouped input path (moe_expert_ffn_grouped): rows
that arrive already grouped by local expert, with the senders' per-expert
counts as metadata (the MoE-side receive region of section 3.2.1, Table 2).

The grouped rows are laid out from the oracle's own dispatch (x[slot_of_row
// k] and the local experts' counts), so every expected value comes from the
oracle.  The rows buffers are larger than the counted rows and the outputs
start as NaN, so a row that the stage computed but should not have, or did
not compute but should have, fails the comparison.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_22541_amd import inputs
from paper_2606_22541_amd import moe_stage as C
from paper_2606_22541_amd.stage import ExpertStage, bf16_bits, quantize_fp8, to_device_routing

from gpu_common import BF16_TOL, FP8_TOL, bits_to_f64, log

pytestmark = pytest.mark.gpu

SPARE = 37          # rows of buffer past the counted rows


def _cfg(dtype, seed, **kw):
    base = dict(d=512, f=256, E=16, e0=3, E_loc=6, k=4, lengths=(780,), dtype=dtype, seed=seed)
    base.update(kw)
    return inputs.MoEConfig("grouped", **base)


def _grouped_inputs(cfg, mb):
    """Oracle dispatch -> grouped rows on the device (bf16 rows, or e4m3 codes
    and scales from the stage's sender-side quantiser), fp64 rows as the
    oracle's FFN sees them, and the local experts' counts."""
    x_bits = bf16_bits(mb.x)
    disp = oracle.dispatch(np.asarray(mb.ids, np.int32), cfg.E, cfg.e0, cfg.E_loc)
    tok = disp["slot_of_row"] // cfg.k
    counts = disp["counts"][cfg.e0:cfg.e0 + cfg.E_loc].astype(np.int32)
    x_all, _, _ = oracle.stage_inputs_x(x_bits, cfg.dtype)
    n = tok.size
    idx = torch.from_numpy(tok.astype(np.int64)).to("cuda")
    x = mb.x.to("cuda")
    scales = None
    if cfg.dtype == "fp8":
        codes, xs = quantize_fp8(x)
        rows = torch.zeros((n + SPARE, cfg.d), dtype=torch.uint8, device="cuda")
        rows[:n] = codes[idx]
        scales = torch.ones((n + SPARE, cfg.d // 128), dtype=torch.float32, device="cuda")
        scales[:n] = xs[idx]
    else:
        rows = torch.full((n + SPARE, cfg.d), float("nan"), dtype=torch.bfloat16, device="cuda")
        rows[:n] = x[idx]
    return rows, scales, x_all[tok], counts


def _y_buffer(cfg, n):
    return torch.full((n, cfg.d), float("nan"), dtype=torch.bfloat16, device="cuda")


def _check_rows(y_bits, ref_y, counts, tol, what):
    """Per-expert rel-L2 of the computed rows; every row past them stays NaN."""
    n = ref_y.shape[0]
    got = bits_to_f64(y_bits[:n])
    assert np.all(np.isfinite(got)), "non-finite grouped output " + what
    lo = 0
    for i, c in enumerate(np.asarray(counts).tolist()):
        if c:
            e = oracle.rel_l2(got[lo:lo + c], ref_y[lo:lo + c])
            assert e <= tol, "expert %d rel-L2 %.3e > %.1e %s" % (i, e, tol, what)
        lo += c
    rest = bits_to_f64(y_bits[n:])
    assert np.all(np.isnan(rest)), "rows past the counted ones were written " + what


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
def test_grouped_rows_match_oracle_and_dispatched_path(dtype):
    cfg = _cfg(dtype, 51)
    wts = inputs.make_weights(cfg, "cuda")
    ow = oracle.OracleWeights(wts, dtype)
    mb = inputs.make_microbatches(cfg, "cuda")[0]
    rows, scales, rows_x, counts = _grouped_inputs(cfg, mb)
    log("grouped %s: counts %s (small and large groups), %d spare rows" % (dtype, counts.tolist(), SPARE))
    assert counts.max() > 192 and counts.min() <= 192, counts
    ref = oracle.run_grouped(cfg, ow, rows_x, counts)
    tol = FP8_TOL if dtype == "fp8" else BF16_TOL
    # counts produced on the device by earlier stream work (the host never passes them)
    dev_counts = torch.from_numpy(counts).to("cuda")
    dev_counts = (dev_counts * 3 - dev_counts * 2).contiguous()
    y = _y_buffer(cfg, rows.shape[0])
    with ExpertStage(cfg, wts, n_slots=2, max_tokens=cfg.lengths[0]) as st:
        st.expert_ffn_grouped(1, rows, dev_counts, y, row_scales=scales)
        # the dispatched path on the other slot computes the same rows
        ids, w = to_device_routing(mb.ids, mb.w)
        x = mb.x.to("cuda")
        xs = None
        if dtype == "fp8":
            x, xs = quantize_fp8(x)
        out = torch.empty((cfg.lengths[0], cfg.d), dtype=torch.bfloat16, device="cuda")
        m = st.microbatch(x, ids, w, out, xs)
        slot = st.submit(m)
        st.sync()
        torch.cuda.synchronize()
        view = st.view(slot)
        with pytest.raises(C.MoEStageError) as e:       # no micro-batch in the grouped slot
            st.combine(1)
        assert e.value.status == C.MOE_EINVAL
    yb = bf16_bits(y)
    _check_rows(yb, ref["y"], counts, tol, dtype)
    n = int(counts.sum())
    assert np.array_equal(yb[:n], view["y_perm"][:n]), "grouped rows differ from the dispatched rows"


def test_bad_counts_are_clamped_and_reported():
    cfg = _cfg("bf16", 52)
    wts = inputs.make_weights(cfg, "cuda")
    ow = oracle.OracleWeights(wts, "bf16")
    rng = np.random.default_rng(52)
    n = 300
    x_bits = rng.standard_normal((n, cfg.d)).astype(np.float32)
    rows = torch.from_numpy(x_bits).to("cuda").to(torch.bfloat16)
    rows_x = bits_to_f64(bf16_bits(rows))
    counts = np.array([40, -7, 0, 200, 90, 5], np.int32)       # 40 + 200 + 60 of 90 fit
    kept = oracle.grouped_counts(counts, n)
    assert kept.tolist() == [40, 0, 0, 200, 60, 0]
    ref = oracle.run_grouped(cfg, ow, rows_x, counts)
    y = _y_buffer(cfg, n)
    with ExpertStage(cfg, wts, n_slots=1, max_tokens=cfg.lengths[0]) as st:
        st.expert_ffn_grouped(0, rows, torch.from_numpy(counts).to("cuda"), y)
        with pytest.raises(C.MoEStageError) as e:
            st.sync()
        assert e.value.status == C.MOE_EBADCOUNT
        st.sync()                                               # cleared
        torch.cuda.synchronize()
    _check_rows(bf16_bits(y), ref["y"], kept, BF16_TOL, "clamped")


def test_grouped_layer_and_empty_and_host_errors():
    cfg = _cfg("bf16", 53, E_loc=4)
    layers = [inputs.make_weights(inputs.scaled(cfg, seed=200 + l), "cuda") for l in range(2)]
    ow1 = oracle.OracleWeights(layers[1], "bf16")
    rng = np.random.default_rng(53)
    n = 150
    rows = torch.from_numpy(rng.standard_normal((n, cfg.d)).astype(np.float32)).to("cuda").to(torch.bfloat16)
    counts = np.array([0, 100, 0, 50], np.int32)
    ref = oracle.run_grouped(cfg, ow1, bits_to_f64(bf16_bits(rows)), counts)
    y = _y_buffer(cfg, n)
    lid = torch.tensor([1], dtype=torch.int32, device="cuda")
    with ExpertStage(cfg, layers, n_slots=1, max_tokens=cfg.lengths[0]) as st:
        dc = torch.from_numpy(counts).to("cuda")
        st.expert_ffn_grouped(0, rows, dc, y, layer_id=lid)
        # all-zero counts: nothing is written
        y0 = _y_buffer(cfg, n)
        st.expert_ffn_grouped(0, rows, torch.zeros(cfg.E_loc, dtype=torch.int32, device="cuda"), y0)
        st.sync()
        torch.cuda.synchronize()
        assert torch.isnan(y0.float()).all()
        # host errors: nothing enqueued
        cap = C.moe_stage_query(st.handle, 0).capacity_rows
        for gb in (C.make_grouped_batch(cap + 1, rows, dc, y), C.make_grouped_batch(n, None, dc, y),
                   C.make_grouped_batch(n, rows, None, y), C.make_grouped_batch(n, rows, dc, None),
                   C.make_grouped_batch(-1, rows, dc, y)):
            with pytest.raises(C.MoEStageError) as e:
                C.moe_expert_ffn_grouped(st.handle, 0, gb)
            assert e.value.status == C.MOE_EINVAL
        with pytest.raises(C.MoEStageError):
            C.moe_expert_ffn_grouped(st.handle, 5, C.make_grouped_batch(n, rows, dc, y))
    _check_rows(bf16_bits(y), ref["y"], counts, BF16_TOL, "layer 1")


def test_counts_across_wave_chunks():
    """80 local experts: the device reads the counts in chunks of 64 with a
    running total, and the clamp to the rows buffer falls in the second
    chunk (expert 70 keeps part of its rows, 71..79 keep none)."""
    cfg = _cfg("bf16", 54, d=256, f=128, E=96, e0=8, E_loc=80, k=2, lengths=(1000,))
    wts = inputs.make_weights(cfg, "cuda")
    ow = oracle.OracleWeights(wts, "bf16")
    rng = np.random.default_rng(54)
    counts = rng.integers(0, 30, cfg.E_loc).astype(np.int32)
    counts[[3, 64, 65]] = [0, 200, 0]                  # a large group opening the second chunk
    counts[10] = -5
    n = int(np.maximum(counts, 0)[:70].sum()) + 7      # expert 70 keeps 7 rows
    kept = oracle.grouped_counts(counts, n)
    assert kept[70] == min(7, counts[70]) and kept[71:].sum() == 0 and kept[10] == 0
    rows = torch.from_numpy(rng.standard_normal((n, cfg.d)).astype(np.float32)).to("cuda").to(torch.bfloat16)
    ref = oracle.run_grouped(cfg, ow, bits_to_f64(bf16_bits(rows)), counts)
    y = _y_buffer(cfg, n + SPARE)
    log("grouped: 80 experts, %d rows, clamp inside the second chunk" % n)
    with ExpertStage(cfg, wts, n_slots=1, max_tokens=cfg.lengths[0]) as st:
        buf = torch.zeros((n + SPARE, cfg.d), dtype=torch.bfloat16, device="cuda")
        buf[:n] = rows
        gb = C.make_grouped_batch(n, buf, torch.from_numpy(counts).to("cuda"), y)
        C.moe_expert_ffn_grouped(st.handle, 0, gb)
        with pytest.raises(C.MoEStageError) as e:
            st.sync()
        assert e.value.status == C.MOE_EBADCOUNT
        torch.cuda.synchronize()
    _check_rows(bf16_bits(y), ref["y"], kept, BF16_TOL, "80 experts")
