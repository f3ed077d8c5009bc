"""GPU tests of the asynchronous ingest (section 3.2.1): senders write their
token rows into the stage's receive buffers and raise ready words; the stage's
work waits on the device until every word has reached the round's epoch.

The receive buffers start poisoned (NaN rows, masked ids), so a stage that
ran before its senders finished would produce NaN or zero outputs and fail
the oracle comparison.  Work is always enqueued in dependency order (each
sender round before the stage round that waits for it), so a wait can never
be stuck behind its own producer in a shared hardware queue; the timeout test
forces the give-up path from the host with a word that is never raised and a
tiny spin limit, so every kernel still exits normally.  The late-producer test
is the one exception: it enqueues the late senders after the wait that waits
for them (on another stream, once the other micro-batches are seen done); the
wait's spin limit bounds it, so streams sharing a hardware queue would make
that test fail, never hang.
"""
import time

import numpy as np
import pytest
import torch

import oracle
from paper_2606_22541_amd import inputs
from paper_2606_22541_amd import moe_stage as C
from paper_2606_22541_amd.stage import ExpertStage, bf16_bits, to_device_routing

from gpu_common import BF16_TOL, check_outputs, log, oracle_run

pytestmark = pytest.mark.gpu

D = 4          # senders (attention DP groups) per micro-batch
T = 300


def _cfg(seed):
    return inputs.MoEConfig("ingest", d=512, f=256, E=12, e0=2, E_loc=4, k=3, lengths=(T,),
                            dtype="bf16", seed=seed)


def _recv(cfg):
    """Receive buffers of one micro-batch, poisoned."""
    x = torch.full((T, cfg.d), float("nan"), dtype=torch.bfloat16, device="cuda")
    ids = torch.full((T, cfg.k), -1, dtype=torch.int32, device="cuda")
    w = torch.zeros((T, cfg.k), dtype=torch.float32, device="cuda")
    return x, ids, w


def _delay(stream, n=6):
    """Device work that keeps `stream` busy for a while."""
    with torch.cuda.stream(stream):
        a = torch.randn((2048, 2048), device="cuda")
        for _ in range(n):
            a = a @ a
            a = a / a.abs().max()
    return a


def _send(stream, mb, recv, ready, epoch, routing=None):
    """Sender g copies its T/D tokens, then raises ready[g] to `epoch`.
    `routing`: the micro-batch's device ids and weights, made beforehand
    (else made here, with a synchronous copy from the host)."""
    x, ids, w = recv
    sids, sw = routing if routing is not None else to_device_routing(mb.ids, mb.w)
    per = T // D
    with torch.cuda.stream(stream):
        for g in range(D):
            sl = slice(g * per, (g + 1) * per)
            x[sl].copy_(mb.x[sl], non_blocking=True)
            ids[sl].copy_(sids[sl], non_blocking=True)
            w[sl].copy_(sw[sl], non_blocking=True)
            C.moe_ingest_signal(ready[g:g + 1], epoch, stream)
    return sids, sw


def test_stage_waits_for_its_senders():
    cfg = _cfg(31)
    wts = inputs.make_weights(cfg, "cuda")
    mb = inputs.make_microbatches(cfg, "cuda")[0]
    ref = oracle_run(cfg, oracle.OracleWeights(wts, "bf16"), mb)
    recv = _recv(cfg)
    ready = torch.zeros(D, dtype=torch.int32, device="cuda")
    out = torch.full((T, cfg.d), float("nan"), dtype=torch.bfloat16, device="cuda")
    prod, cons = torch.cuda.Stream(), torch.cuda.Stream()
    with ExpertStage(cfg, wts, n_slots=1, max_tokens=T) as st:
        torch.cuda.synchronize()
        log("ingest: %d senders behind a delay, stage waits for epoch 1" % D)
        keep = _delay(prod), _send(prod, mb, recv, ready, 1)
        m = st.microbatch(recv[0], recv[1], recv[2], out)
        C.moe_ingest_wait(st.handle, ready, D, 1, 0, cons)
        st.submit(m, cons)
        st.sync()
        torch.cuda.synchronize()
        del keep
    check_outputs(bf16_bits(out), ref, BF16_TOL, "after ingest")


def test_rounds_with_backpressure():
    """Three rounds through one set of receive buffers: round r's senders
    wait until the stage has acknowledged round r-1, the stage's round r
    waits for epoch r; every round's output matches its own oracle."""
    cfgs = [_cfg(40 + r) for r in range(3)]
    wts = inputs.make_weights(cfgs[0], "cuda")
    ow = oracle.OracleWeights(wts, "bf16")
    mbs = [inputs.make_microbatches(c, "cuda")[0] for c in cfgs]
    refs = [oracle_run(cfgs[0], ow, mb) for mb in mbs]
    recv = _recv(cfgs[0])
    ready = torch.zeros(D, dtype=torch.int32, device="cuda")
    consumed = torch.zeros(1, dtype=torch.int32, device="cuda")
    outs = [torch.full((T, cfgs[0].d), float("nan"), dtype=torch.bfloat16, device="cuda")
            for _ in mbs]
    prod, cons = torch.cuda.Stream(), torch.cuda.Stream()
    keep = []
    with ExpertStage(cfgs[0], wts, n_slots=2, max_tokens=T) as st:
        torch.cuda.synchronize()
        for r, mb in enumerate(mbs, start=1):
            # senders of round r: wait until round r-1 is consumed, then write
            C.moe_ingest_wait(st.handle, consumed, 1, r - 1, 0, prod)
            keep.append(_delay(prod, 2))
            keep.append(_send(prod, mb, recv, ready, r))
            # the stage's round r, then its acknowledgement
            m = st.microbatch(recv[0], recv[1], recv[2], outs[r - 1])
            keep.append(m)
            C.moe_ingest_wait(st.handle, ready, D, r, 0, cons)
            st.submit(m, cons)
            C.moe_ingest_signal(consumed, r, cons)
        st.sync()
        torch.cuda.synchronize()
    assert int(consumed.item()) == 3 and ready.cpu().tolist() == [3] * D
    for r in range(3):
        check_outputs(bf16_bits(outs[r]), refs[r], BF16_TOL, "round %d" % (r + 1))


def test_wait_gives_up_and_reports_timeout():
    cfg = _cfg(33)
    wts = inputs.make_weights(cfg, "cuda")
    recv = _recv(cfg)
    never = torch.zeros(2, dtype=torch.int32, device="cuda")
    out = torch.zeros((T, cfg.d), dtype=torch.bfloat16, device="cuda")
    with ExpertStage(cfg, wts, n_slots=1, max_tokens=T) as st:
        m = st.microbatch(recv[0], recv[1], recv[2], out)
        C.moe_ingest_wait(st.handle, never, 2, 5, 64)     # a word nobody raises, 64 polls
        st.submit(m)
        with pytest.raises(C.MoEStageError) as e:
            st.sync()
        assert e.value.status == C.MOE_ETIMEOUT
        # all ids were masked: every token is written as +0.0
        assert torch.count_nonzero(out).item() == 0
        st.sync()                                           # the error was cleared


def test_wrapping_epochs():
    """Epoch comparison wraps: a word at 2 has reached 0xFFFFFFFF + 3."""
    cfg = _cfg(34)
    wts = inputs.make_weights(cfg, "cuda")
    ready = torch.tensor([2, 7], dtype=torch.int32, device="cuda")
    with ExpertStage(cfg, wts, n_slots=1, max_tokens=T) as st:
        C.moe_ingest_wait(st.handle, ready, 2, 0xFFFFFFFF, 64)   # 2 - (2^32 - 1) = 3 >= 0
        C.moe_ingest_wait(st.handle, ready, 2, 2, 64)
        torch.cuda.synchronize()
        st.sync()
        C.moe_ingest_wait(st.handle, ready, 2, 3, 64)             # word 0 is behind
        torch.cuda.synchronize()
        with pytest.raises(C.MoEStageError) as e:
            st.sync()
        assert e.value.status == C.MOE_ETIMEOUT


def test_late_producer_does_not_hold_back_the_others():
    """A micro-batch whose senders are late holds back only itself (section
    3.2.1: a batch is taken when it is ready, in whatever order).  Micro-batch
    A is submitted first, on its own stream, behind a wait on its ready words
    whose senders are not enqueued yet; B and C are then sent and submitted on
    a second stream.  B's and C's slots complete while A's is still busy --
    a certainty, not a race: nothing can release A yet -- and only then are
    A's senders enqueued.  All three match the oracle.  Every device wait is
    bounded, so if A's wait held back B and C it would give up after its spin
    limit and the test would fail with MOE_ETIMEOUT, every kernel exited."""
    cfgs = [_cfg(50 + i) for i in range(3)]
    wts = inputs.make_weights(cfgs[0], "cuda")
    ow = oracle.OracleWeights(wts, "bf16")
    mbs = [inputs.make_microbatches(c, "cuda")[0] for c in cfgs]
    refs = [oracle_run(cfgs[0], ow, mb) for mb in mbs]
    # everything is allocated and copied before the first wait is enqueued:
    # no later host-side copy may queue behind a wait on another stream
    routing = [to_device_routing(mb.ids, mb.w) for mb in mbs]
    recv = [_recv(cfgs[0]) for _ in mbs]
    ready = [torch.zeros(D, dtype=torch.int32, device="cuda") for _ in mbs]
    outs = [torch.full((T, cfgs[0].d), float("nan"), dtype=torch.bfloat16, device="cuda")
            for _ in mbs]
    s_late, s_rest = torch.cuda.Stream(), torch.cuda.Stream()
    with ExpertStage(cfgs[0], wts, n_slots=3, max_tokens=T) as st:
        ms = [st.microbatch(r[0], r[1], r[2], o) for r, o in zip(recv, outs)]
        warm = torch.empty_like(outs[0])                  # first launches out of the way
        st.submit(st.microbatch(mbs[0].x, routing[0][0], routing[0][1], warm), s_rest)
        st.sync()
        torch.cuda.synchronize()
        log("late producer: A waits for senders not yet enqueued, B and C ready")
        C.moe_ingest_wait(st.handle, ready[0], D, 1, 1 << 22, s_late)   # about 8 s at most
        slot_a = st.submit(ms[0], s_late)
        slots = []
        for i in (1, 2):
            _send(s_rest, mbs[i], recv[i], ready[i], 1, routing[i])
            C.moe_ingest_wait(st.handle, ready[i], D, 1, 0, s_rest)
            slots.append(st.submit(ms[i], s_rest))
        assert len({slot_a, *slots}) == 3
        t0 = time.time()
        others_done = False
        while time.time() - t0 < 4.0:
            if all(C.moe_stage_poll(st.handle, s) == C.MOE_OK for s in slots):
                others_done = True
                break
            time.sleep(0.001)
        a_busy = C.moe_stage_poll(st.handle, slot_a) == C.MOE_EBUSY
        log("  B, C done after %.1f ms: %s; A still busy: %s"
            % ((time.time() - t0) * 1e3, others_done, a_busy))
        _send(s_rest, mbs[0], recv[0], ready[0], 1, routing[0])  # A's senders, late
        st.sync()
        torch.cuda.synchronize()
        assert C.moe_stage_poll(st.handle, slot_a) == C.MOE_OK
    assert others_done, "B and C did not complete while A's senders were held back"
    assert a_busy, "A completed before its senders were enqueued"
    for i, name in enumerate("ABC"):
        check_outputs(bf16_bits(outs[i]), refs[i], BF16_TOL, "micro-batch %s" % name)
