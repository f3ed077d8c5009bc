"""moe_dispatch_index_noalloc (no allocation, scratch in a static device
array) against moe_dispatch on a stage, bit for bit: two calls in a row, the
second with a smaller input, then the edge cases."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_22541_amd import inputs
from paper_2606_22541_amd import moe_stage as C
from paper_2606_22541_amd.stage import ExpertStage, to_device_routing

from gpu_common import log

pytestmark = pytest.mark.gpu


def _noalloc(ids_dev, T, k, E, e0, E_loc, err=None):
    counts = torch.full((E,), -7, dtype=torch.int32, device="cuda")
    offsets = torch.full((E_loc + 1,), -7, dtype=torch.int32, device="cuda")
    sor = torch.full((max(T * k, 1),), -7, dtype=torch.int32, device="cuda")
    ros = torch.full((max(T * k, 1),), -7, dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()
    C.moe_dispatch_index_noalloc(ids_dev, T, k, E, e0, E_loc, counts, offsets, sor, ros, err)
    torch.cuda.synchronize()
    n = int(offsets[-1].item())
    return dict(counts=counts.cpu().numpy(), offsets=offsets.cpu().numpy(),
                slot_of_row=sor[:n].cpu().numpy(), row_of_slot=ros[:T * k].cpu().numpy())


def _stage_dispatch(cfg, mb):
    """The existing entry point: moe_dispatch on a stage's slot."""
    w = inputs.make_weights(cfg, "cuda")
    T = mb.ids.shape[0]
    with ExpertStage(cfg, w, n_slots=1, max_tokens=max(T, 1)) as st:
        ids, wt = to_device_routing(mb.ids, mb.w)
        out = torch.empty((max(T, 1), cfg.d), dtype=torch.bfloat16, device="cuda")
        torch.cuda.synchronize()
        st.dispatch(0, st.microbatch(mb.x, ids, wt, out))
        status = C.moe_stage_sync_status(st.handle)
        v = st.view(0, rows=False)
    return v, status


def _same(a, b, what):
    for key in ("counts", "offsets", "slot_of_row", "row_of_slot"):
        assert np.array_equal(a[key], b[key]), "%s: %s differs" % (what, key)


def test_noalloc_matches_moe_dispatch_twice_second_smaller():
    big = inputs.MoEConfig("na_big", d=256, f=128, E=256, e0=0, E_loc=8, k=8, lengths=(32768,),
                           seed=31)
    small = inputs.MoEConfig("na_small", d=256, f=128, E=64, e0=5, E_loc=6, k=4, lengths=(333,),
                             seed=32)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    for cfg, bad in ((big, False), (small, True)):
        mb = inputs.make_microbatches(cfg, "cuda")[0]
        if bad:                                     # masked slots and one invalid id
            mb.ids[::7, 1] = -1
            mb.ids[5, 2] = cfg.E + 3
        T, k = mb.ids.shape
        log("noalloc %s: T=%d k=%d E=%d e0=%d E_loc=%d" % (cfg.name, T, k, cfg.E, cfg.e0, cfg.E_loc))
        ids_dev, _ = to_device_routing(mb.ids, mb.w)
        got = _noalloc(ids_dev, T, k, cfg.E, cfg.e0, cfg.E_loc, err)
        ref, status = _stage_dispatch(cfg, mb)
        _same(got, ref, cfg.name)
        clean = np.where((mb.ids >= -1) & (mb.ids < cfg.E), mb.ids, -1)
        _same(got, oracle.dispatch(clean, cfg.E, cfg.e0, cfg.E_loc), cfg.name + " vs oracle")
        assert int(err.item()) == (1 if bad else 0)
        assert status == (C.MOE_EBADID if bad else C.MOE_OK)
        log("  %d local rows, bit-exact with moe_dispatch and the oracle" % got["offsets"][-1])


def test_noalloc_edge_cases():
    # no tokens: zero counts and offsets, nothing else written
    ids = torch.zeros((1, 2), dtype=torch.int32, device="cuda")
    got = _noalloc(ids, 0, 2, 8, 0, 4)
    assert not got["counts"].any() and not got["offsets"].any()
    # every slot masked, then a single expert holding every slot
    for ids_np in (np.full((9, 2), -1, np.int32), np.full((300, 2), 2, np.int32)):
        ids_dev = torch.from_numpy(ids_np).cuda()
        got = _noalloc(ids_dev, ids_np.shape[0], 2, 8, 0, 4)
        _same(got, oracle.dispatch(ids_np, 8, 0, 4), "edge")
    # past the scratch's histogram rows: refused on the host, nothing enqueued
    with pytest.raises(C.MoEStageError) as e:
        C.moe_dispatch_index_noalloc(ids, 1 << 20, 8, 256, 0, 8, ids, ids, ids, ids)
    assert e.value.status == C.MOE_EUNSUPPORTED
    with pytest.raises(C.MoEStageError) as e:
        C.moe_dispatch_index_noalloc(ids, 4, 2, 8, 6, 4, ids, ids, ids, ids)
    assert e.value.status == C.MOE_EINVAL
