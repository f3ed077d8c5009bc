"""GPU parity of the HIP expert stage against the CPU oracle (bf16 path).

Bit-exact: counts, offsets, slot_of_row, row_of_slot (X_perm is not materialised:
the gate/up GEMM gathers the token rows itself, so the gather is checked through the outputs).
Floating point: rel-L2 <= 1e-2 on outputs and per expert on Y_perm rows.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_22541_amd import inputs
from paper_2606_22541_amd import moe_stage as C
from paper_2606_22541_amd.stage import ExpertStage, bf16_bits, to_device_routing

from gpu_common import (BF16_TOL, CachedWeights, band_order_tiles, check_dispatch, check_expert_rows,
                        check_outputs, gpu_run, log, oracle_run, poison_workspace)

pytestmark = pytest.mark.gpu


def _case(cfg, mbs=None, *, n_streams=1, mode=0, tol=BF16_TOL, n_slots=None):
    """Every token and every Y_perm row of every micro-batch against the
    oracle, with the workspace poisoned with NaN before the run."""
    log("case %s: d=%d f=%d E=%d E_loc=%d k=%d lengths=%s shared=%d streams=%d" % (
        cfg.name, cfg.d, cfg.f, cfg.E, cfg.E_loc, cfg.k, cfg.lengths, cfg.has_shared, n_streams))
    w = inputs.make_weights(cfg, "cuda")
    if mbs is None:
        mbs = inputs.make_microbatches(cfg, "cuda")
    ow = CachedWeights(oracle.OracleWeights(w, cfg.dtype))
    streams = [torch.cuda.Stream() for _ in range(n_streams)] if n_streams > 1 else None
    with ExpertStage(cfg, w, n_slots=n_slots or len(mbs),
                     max_tokens=max(max(mb.ids.shape[0] for mb in mbs), 1)) as st:
        poison_workspace(st)
        outs, slots, keep = gpu_run(st, mbs, streams=streams, mode=mode)
        errs = []
        for mb, ob, sl in zip(mbs, outs, slots):
            ref = oracle_run(cfg, ow, mb)
            view = st.view(sl)
            check_dispatch(view, ref, cfg, mb)
            errs.append(check_outputs(ob, ref, tol, cfg.name))
            check_expert_rows(view, ref, cfg, tol, cfg.name)
        log("  rel-L2 per micro-batch: %s" % ["%.2e" % e for e in errs])
    return outs


def test_c0_tiny_full_parity():
    _case(inputs.CONFIGS["c0"])


@pytest.mark.parametrize("T,d,f,E,E_loc,k", [
    (700, 1024, 384, 16, 4, 4),     # several row and column tiles, ragged tails
    (333, 640, 256, 8, 3, 2),       # d = 640: partial 256-column tile in the down GEMM
    (100, 640, 256, 8, 3, 2),       # groups of <= 64 rows: the down GEMM's small-group tiles end
                                    # in a half weight panel (d = 640 = 2.5 panels of 256)
    (1, 256, 128, 8, 4, 2),         # one token
    (257, 256, 128, 1, 1, 1),       # one expert, 257 rows: tile + 1
])
def test_multi_tile_shapes(T, d, f, E, E_loc, k):
    cfg = inputs.MoEConfig("mt", d=d, f=f, E=E, e0=0, E_loc=E_loc, k=k, lengths=(T,), seed=3)
    _case(cfg)


def test_multi_tile_with_shared_expert_and_offset_experts():
    cfg = inputs.MoEConfig("sh", d=512, f=256, E=12, e0=5, E_loc=4, k=3, lengths=(600,),
                           has_shared=True, seed=4)
    _case(cfg)


def test_edge_cases_dispatch_and_outputs():
    cfg = inputs.MoEConfig("edge", d=256, f=128, E=8, e0=0, E_loc=4, k=2, lengths=(0,), seed=5)
    w = inputs.make_weights(cfg, "cuda")
    ow = oracle.OracleWeights(w, "bf16")
    rng = np.random.default_rng(0)
    cases = {
        "empty": np.zeros((0, 2), np.int32),
        "all_masked": np.full((9, 2), -1, np.int32),
        "one_expert": np.full((300, 2), 2, np.int32),            # duplicates count twice
        "tile_minus_one": np.stack([np.full(255, 1), np.full(255, 5)], 1).astype(np.int32),
        "tile_plus_one": np.stack([np.full(257, 3), np.full(257, -1)], 1).astype(np.int32),
        "mixed": rng.integers(-1, 8, size=(513, 2)).astype(np.int32),
    }
    with ExpertStage(cfg, w, n_slots=2, max_tokens=600) as st:
        for name, ids in cases.items():
            log("edge case %s T=%d" % (name, ids.shape[0]))
            T = ids.shape[0]
            x = torch.randn((T, cfg.d), generator=torch.Generator("cuda").manual_seed(1),
                            device="cuda").to(torch.bfloat16)
            mb = inputs.MicroBatch(x=x, ids=ids, w=rng.random((T, 2)).astype(np.float32))
            outs, slots, _ = gpu_run(st, [mb])
            ref = oracle_run(cfg, ow, mb)
            view = st.view(slots[0])
            check_dispatch(view, ref, cfg, mb)
            if T:
                check_outputs(outs[0], ref, BF16_TOL, name)


def test_bad_expert_id_is_reported_and_skipped():
    cfg = inputs.MoEConfig("bad", d=256, f=128, E=8, e0=0, E_loc=4, k=2, lengths=(5,), seed=6)
    w = inputs.make_weights(cfg, "cuda")
    ids = np.array([[0, 1], [9, 2], [-7, 3], [1, -1], [2, 2]], np.int32)
    mb = inputs.MicroBatch(x=torch.ones((5, 256), dtype=torch.bfloat16, device="cuda"), ids=ids,
                           w=np.full((5, 2), 0.5, np.float32))
    with ExpertStage(cfg, w) as st:
        i, wt = to_device_routing(ids, mb.w)
        out = torch.zeros((5, 256), dtype=torch.bfloat16, device="cuda")
        st.submit(st.microbatch(mb.x, i, wt, out))
        assert C.moe_stage_sync_status(st.handle) == C.MOE_EBADID
        assert C.moe_stage_sync_status(st.handle) == C.MOE_OK          # reported once
        view = st.view(0)
        ref = oracle.dispatch(np.where((ids >= -1) & (ids < 8), ids, -1), 8, 0, 4)
        assert np.array_equal(view["row_of_slot"], ref["row_of_slot"])
        assert np.array_equal(view["counts"], ref["counts"])


@pytest.mark.parametrize("T", [1000, 4200])
def test_bad_ids_in_many_dispatch_chunks(T):
    """Bad ids spread over 8 and 33 chunks of 1024 slots (8000 and 33600
    slots): reported once, placed as masked."""
    cfg = inputs.MoEConfig("bad2", d=256, f=128, E=64, e0=8, E_loc=8, k=8, lengths=(T,), seed=14)
    w = inputs.make_weights(cfg, "cuda")
    rng = np.random.default_rng(14)
    ids = rng.integers(-1, 64, size=(T, 8)).astype(np.int32)
    bad = rng.choice(T * 8, size=5, replace=False)
    ids.reshape(-1)[bad] = np.array([64, 100, -2, -50, 1 << 20], np.int32)
    mb = inputs.MicroBatch(x=torch.ones((T, 256), dtype=torch.bfloat16, device="cuda"), ids=ids,
                           w=np.full((T, 8), 0.125, np.float32))
    with ExpertStage(cfg, w, max_tokens=T) as st:
        i, wt = to_device_routing(ids, mb.w)
        out = torch.zeros((T, 256), dtype=torch.bfloat16, device="cuda")
        st.submit(st.microbatch(mb.x, i, wt, out))
        assert C.moe_stage_sync_status(st.handle) == C.MOE_EBADID
        assert C.moe_stage_sync_status(st.handle) == C.MOE_OK
        view = st.view(0)
        ref = oracle.dispatch(np.where((ids >= -1) & (ids < 64), ids, -1), 64, 8, 8)
        assert np.array_equal(view["row_of_slot"], ref["row_of_slot"])
        assert np.array_equal(view["counts"], ref["counts"])
        assert np.array_equal(view["offsets"], ref["offsets"])


@pytest.mark.parametrize("T,k,E,e0,E_loc", [
    (4097, 8, 64, 8, 8),          # 32776 slots: a last chunk of 8 slots
    (16385, 2, 1024, 512, 256),   # 32770 slots over 1024 experts, 256 of them local
])
def test_dispatch_many_chunks_and_largest_tables(T, k, E, e0, E_loc):
    cfg = inputs.MoEConfig("cnt", d=256, f=128, E=E, e0=e0, E_loc=E_loc, k=k, lengths=(T,), seed=13)
    _case(cfg)


def test_host_errors_enqueue_nothing():
    cfg = inputs.MoEConfig("err", d=256, f=128, E=8, e0=0, E_loc=4, k=2, lengths=(4,), seed=7)
    w = inputs.make_weights(cfg, "cuda")
    with ExpertStage(cfg, w, max_tokens=4) as st:
        ids, wt = to_device_routing(np.zeros((8, 2), np.int32), np.ones((8, 2), np.float32))
        x = torch.zeros((8, 256), dtype=torch.bfloat16, device="cuda")
        out = torch.zeros((8, 256), dtype=torch.bfloat16, device="cuda")
        with pytest.raises(C.MoEStageError) as e:             # T > max_tokens
            st.submit(st.microbatch(x, ids, wt, out))
        assert e.value.status == C.MOE_EINVAL
        with pytest.raises(C.MoEStageError):                  # bad slot
            C.moe_dispatch(st.handle, 3, C.make_microbatch(2, x, ids, wt, out))
        with pytest.raises(C.MoEStageError):                  # null pointer
            C.moe_dispatch(st.handle, 0, C.make_microbatch(2, None, ids, wt, out))
        with pytest.raises(C.MoEStageError):                  # ffn before any dispatch
            C.moe_expert_ffn(st.handle, 0)
        with pytest.raises(C.MoEStageError):                  # bad combine mode
            C.moe_dispatch(st.handle, 0, C.make_microbatch(2, x, ids, wt, out, combine_mode=7))
        assert C.moe_stage_sync_status(st.handle) == C.MOE_OK
    for dd, ff in ((200, 128), (256, 192)):                    # d or f not a multiple of 128
        bad = C.make_desc(dd, ff, 8, 0, 4, 2, 4)
        with pytest.raises(C.MoEStageError) as e:
            C.moe_stage_create(bad, C.make_weights(w.w_gate, w.w_up, w.w_down))
        assert e.value.status == C.MOE_EUNSUPPORTED
    bad = C.make_desc(256, 128, 8, 6, 4, 2, 4)                # local experts past n_experts
    with pytest.raises(C.MoEStageError) as e:
        C.moe_stage_create(bad, C.make_weights(w.w_gate, w.w_up, w.w_down))
    assert e.value.status == C.MOE_EINVAL


def test_poll_reports_busy_then_done():
    """moe_stage_poll never waits: a slot is MOE_OK before its first use,
    MOE_OK or MOE_EBUSY while a micro-batch runs, and MOE_OK once it is done."""
    cfg = inputs.CONFIGS["c1"]
    w = inputs.make_weights(cfg, "cuda")
    mbs = inputs.make_microbatches(cfg, "cuda")
    with ExpertStage(cfg, w, n_slots=2) as st:
        assert C.moe_stage_poll(st.handle, 0) == C.MOE_OK
        assert C.moe_stage_poll(st.handle, 1) == C.MOE_OK
        with pytest.raises(C.MoEStageError):
            C.moe_stage_poll(st.handle, 2)
        ids, wt = to_device_routing(mbs[0].ids, mbs[0].w)
        out = torch.empty((4096, cfg.d), dtype=torch.bfloat16, device="cuda")
        torch.cuda.synchronize()
        seen = set()
        for _ in range(4):                       # four micro-batches, ~0.2 ms each
            slot = st.submit(st.microbatch(mbs[0].x, ids, wt, out))
            seen.add(C.moe_stage_poll(st.handle, slot))
        log("  poll right after submit: %s" % sorted(seen))
        st.sync()
        assert C.moe_stage_poll(st.handle, 0) == C.MOE_OK
        assert C.moe_stage_poll(st.handle, 1) == C.MOE_OK


def test_accumulate_mode_and_determinism():
    cfg = inputs.MoEConfig("acc", d=512, f=256, E=16, e0=0, E_loc=4, k=4, lengths=(300,), seed=8)
    w = inputs.make_weights(cfg, "cuda")
    mbs = inputs.make_microbatches(cfg, "cuda")
    ow = oracle.OracleWeights(w, "bf16")
    base = torch.randn((300, 512), device="cuda").to(torch.bfloat16)
    with ExpertStage(cfg, w, n_slots=2) as st:
        o1, s1, _ = gpu_run(st, mbs, mode=C.MOE_COMBINE_ACCUMULATE, out_init=[base])
        o2, _, _ = gpu_run(st, mbs, mode=C.MOE_COMBINE_ACCUMULATE, out_init=[base])
        assert np.array_equal(o1[0], o2[0]), "not bit-identical run to run"
        ref = oracle_run(cfg, ow, mbs[0], mode=1, base=oracle.bf16_bits_to_f64(bf16_bits(base)))
        check_outputs(o1[0], ref, BF16_TOL, "accumulate")
        untouched = np.all(ref["row_of_slot"].reshape(300, 4) < 0, axis=1)
        assert np.array_equal(o1[0][untouched], bf16_bits(base)[untouched])


def test_down_weight_scaling_is_exact():
    """Doubling W_down doubles Y and the output exactly (power-of-two scale)."""
    cfg = inputs.MoEConfig("x2", d=512, f=256, E=8, e0=0, E_loc=4, k=2, lengths=(200,), seed=9)
    w = inputs.make_weights(cfg, "cuda")
    mbs = inputs.make_microbatches(cfg, "cuda")
    with ExpertStage(cfg, w) as st:
        o1, _, _ = gpu_run(st, mbs)
    w.w_down = (w.w_down.float() * 2).to(torch.bfloat16)
    with ExpertStage(cfg, w) as st:
        o2, _, _ = gpu_run(st, mbs)
    a = oracle.bf16_bits_to_f64(o1[0])
    b = oracle.bf16_bits_to_f64(o2[0])
    assert np.array_equal(b, 2 * a)


def test_empty_experts_poisoned_with_nan_contribute_nothing():
    cfg = inputs.MoEConfig("nan", d=256, f=128, E=8, e0=0, E_loc=4, k=2, lengths=(100,), seed=10)
    w = inputs.make_weights(cfg, "cuda")
    rng = np.random.default_rng(1)
    ids = np.stack([rng.choice([0, 2, 4, 6, 7], size=2, replace=False) for _ in range(100)]).astype(np.int32)
    for m in (w.w_gate, w.w_up, w.w_down):
        m[1].fill_(float("nan"))
        m[3].fill_(float("nan"))
    mb = inputs.MicroBatch(x=torch.randn((100, 256), device="cuda").to(torch.bfloat16), ids=ids,
                           w=rng.random((100, 2)).astype(np.float32))
    with ExpertStage(cfg, w) as st:
        outs, _, _ = gpu_run(st, [mb])
    assert np.all(np.isfinite(oracle.bf16_bits_to_f64(outs[0])))


def test_streams_match_single_stream_bitwise():
    cfg = inputs.scaled(inputs.CONFIGS["c2"], d=512, f=256, name="c2s")
    w = inputs.make_weights(cfg, "cuda")
    mbs = inputs.make_microbatches(cfg, "cuda")
    with ExpertStage(cfg, w, n_slots=4, max_tokens=cfg.max_tokens) as st:
        one, _, _ = gpu_run(st, mbs)
        four, _, _ = gpu_run(st, mbs, streams=[torch.cuda.Stream() for _ in range(4)])
        two_slots = ExpertStage(cfg, w, n_slots=2, max_tokens=cfg.max_tokens)
        ring, _, _ = gpu_run(two_slots, mbs, streams=[torch.cuda.Stream() for _ in range(4)])
        two_slots.close()
    for a, b, c in zip(one, four, ring):
        assert np.array_equal(a, b) and np.array_equal(a, c)


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
def test_three_stream_layout_matches_single_stream_bitwise(dtype):
    """The three-stream layout bench.py times: dispatch, expert FFN and
    combine of each micro-batch on three streams chained by events, six
    micro-batches through three slots (a slot is reused once its last
    combine has run), bit-identical to one stream with whole submissions."""
    cfg = inputs.scaled(inputs.CONFIGS["c2"], d=512, f=256, n_micro=6, dtype=dtype,
                        name="tri_" + dtype)
    w = inputs.make_weights(cfg, "cuda")
    mbs = inputs.make_microbatches(cfg, "cuda")
    with ExpertStage(cfg, w, n_slots=3, max_tokens=cfg.max_tokens) as st:
        ref, _, keep = gpu_run(st, mbs)
        outs = []
        for (x, xs, ids, wt, out, _) in keep:
            o = torch.full_like(out, float("nan"))
            outs.append((st.microbatch(x, ids, wt, o, xs), o))
        D, G, R = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
        torch.cuda.synchronize()
        slot_done = [None] * 3
        for i, (m, _) in enumerate(outs):
            k = i % 3
            if slot_done[k] is not None:
                D.wait_event(slot_done[k])
            st.dispatch(k, m, D)
            e1 = torch.cuda.Event()
            e1.record(D)
            G.wait_event(e1)
            st.expert_ffn(k, G)
            e2 = torch.cuda.Event()
            e2.record(G)
            R.wait_event(e2)
            st.combine(k, R)
            slot_done[k] = torch.cuda.Event()
            slot_done[k].record(R)
        st.sync()
        torch.cuda.synchronize()
    for i, ((_, o), r) in enumerate(zip(outs, ref)):
        assert np.array_equal(bf16_bits(o), r), "micro-batch %d differs" % i


# ---------------------------------------------------------------------------
# Full-size configurations (every token and every routed row checked)
# ---------------------------------------------------------------------------
def test_c1_deepseek_ep32_share():
    _case(inputs.CONFIGS["c1"])


def test_c1p_deepseek_ep32_share_32k_tokens():
    _case(inputs.CONFIGS["c1p"])


def test_c2_skewed_four_streams():
    _case(inputs.CONFIGS["c2"], n_streams=4)


def test_c3_ep8_share_with_shared_expert():
    _case(inputs.CONFIGS["c3"])


def test_band_order_with_more_tiles_than_cus():
    """More 256x256 tiles than CUs with a last round more than half full: the
    256-row GEMMs keep the band order (row tiles rastered in bands of 4 per
    column block, partial tiles beside their full ones) in both products.
    d = 1024, f = 512 and about 26k routed rows over 8 experts (13-14 row
    tiles each); every row is checked."""
    cfg = inputs.MoEConfig("band", d=1024, f=512, E=16, e0=0, E_loc=8, k=8, lengths=(6500,), seed=21)
    mbs = inputs.make_microbatches(cfg, "cuda")
    disp = oracle.dispatch(mbs[0].ids, cfg.E, cfg.e0, cfg.E_loc)
    for N, small in ((2 * cfg.f, 192), (cfg.d, 0)):       # gate/up, down (every group)
        total, cus, by_size = band_order_tiles(disp["counts"][:cfg.E_loc], N, small)
        log("  N=%d: %d tiles on %d CUs, size order %s" % (N, total, cus, by_size))
        assert not by_size, "the case no longer exercises the band order"
    _case(cfg, mbs)


def test_max_local_experts_and_group_size_boundaries():
    """256 local experts of 1024 (the largest tables the dispatch kernels
    size for, a shared expert making 257 groups) with crafted group sizes
    around the small/large GEMM boundaries (gate/up at 192 rows, down at 64):
    1, 33, 64, 65, 160, 192 and 193 rows, and many empty experts."""
    cfg = inputs.MoEConfig("maxE", d=256, f=128, E=1024, e0=512, E_loc=256, k=2, lengths=(0,),
                           has_shared=True, seed=8)
    rng = np.random.default_rng(8)
    sizes = {512 + 0: 192, 512 + 1: 193, 512 + 2: 160, 512 + 3: 33, 512 + 4: 1, 512 + 5: 64,
             512 + 6: 65}
    first = np.concatenate([np.full(n, e, np.int32) for e, n in sizes.items()])
    T = first.size                                       # 708 tokens
    rng.shuffle(first)
    # second choice: a non-local expert or a sparse spread over the other local experts
    second = np.where(rng.random(T) < 0.7, rng.integers(0, 512, T),
                      rng.integers(512 + 7, 512 + 256, T)).astype(np.int32)
    ids = np.stack([first, second], 1)
    x = torch.randn((T, cfg.d), generator=torch.Generator("cuda").manual_seed(2),
                    device="cuda").to(torch.bfloat16)
    mb = inputs.MicroBatch(x=x, ids=ids, w=rng.random((T, 2)).astype(np.float32))
    _case(cfg, [mb])


def test_partial_row_tiles_in_size_order():
    """The 256-row GEMM runs every group's full row tiles first and then the
    partial ones by decreasing size.  Group sizes around every tile boundary
    (0, 1, 31..33, 63..65, 128/129, 192/193, 255..257, 511..513), two groups with the
    same partial size (300 and 44 rows), a group with several full tiles
    (700) and a shared expert over all 4579 tokens; outputs start as NaN, so a
    tile that no workgroup ran fails the comparison."""
    sizes = [0, 1, 31, 32, 33, 63, 64, 65, 128, 129, 192, 193, 255, 256, 257, 300, 511, 512, 513,
             700, 44]
    cfg = inputs.MoEConfig("tile_order", d=256, f=128, E=24, e0=0, E_loc=len(sizes), k=1,
                           lengths=(0,), has_shared=True, seed=12)
    rng = np.random.default_rng(12)
    first = np.concatenate([np.full(n, e, np.int32) for e, n in enumerate(sizes)] +
                           [rng.integers(len(sizes), cfg.E, 300).astype(np.int32)])
    rng.shuffle(first)
    T = first.size
    x = torch.randn((T, cfg.d), generator=torch.Generator("cuda").manual_seed(3),
                    device="cuda").to(torch.bfloat16)
    mb = inputs.MicroBatch(x=x, ids=first[:, None].copy(), w=rng.random((T, 1)).astype(np.float32))
    _case(cfg, [mb])
