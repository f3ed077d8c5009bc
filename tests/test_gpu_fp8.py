"""GPU parity of the fp8 (e4m3, 128-block scales) expert stage and of the
sender-side quantiser against the CPU oracle.

Bit-exact: quantiser codes and scales, counts, permutation, the gathered x
scales (the e4m3 rows themselves are read by the gate/up GEMM through
slot_of_row and checked through H and Y_perm).  Floating point: rel-L2 <= 3e-2
on outputs and per expert on Y_perm.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_22541_amd import inputs
from paper_2606_22541_amd.stage import ExpertStage, bf16_bits, quantize_fp8

from gpu_common import (FP8_TOL, CachedWeights, check_dispatch, check_expert_rows, check_outputs,
                        gpu_run, log, oracle_run, poison_workspace)

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("T,d,scale", [(1, 128, 1.0), (333, 512, 1.0), (1000, 7168, 1.0),
                                       (64, 256, 1e-3), (64, 256, 300.0)])
def test_quantizer_bit_exact(T, d, scale):
    log("quantizer T=%d d=%d scale=%g" % (T, d, scale))
    g = torch.Generator("cuda").manual_seed(T + d)
    x = (torch.randn((T, d), generator=g, device="cuda") * scale).to(torch.bfloat16)
    if T > 1:
        x[0, :128] = 0                    # an all-zero group: scale 1, codes 0
        x[T - 1, 5] = -x[T - 1, 5]
    xq, xs = quantize_fp8(x)
    torch.cuda.synchronize()
    codes, scales = oracle.quantize_groups(oracle.bf16_bits_to_f32(bf16_bits(x)))
    got_q = xq.cpu().numpy()
    got_s = xs.cpu().numpy()
    assert np.array_equal(got_s.view(np.uint32), scales.view(np.uint32)), "scales differ"
    bad = np.nonzero(got_q != codes)
    assert bad[0].size == 0, "codes differ at %s: gpu %s oracle %s" % (
        list(zip(*bad))[:5], got_q[bad][:5], codes[bad][:5])


def _case(cfg, mbs=None, *, n_streams=1):
    """Every token and every Y_perm row against the oracle, with the
    workspace poisoned with NaN before the run."""
    log("fp8 case %s: d=%d f=%d E=%d E_loc=%d k=%d lengths=%s shared=%d streams=%d" % (
        cfg.name, cfg.d, cfg.f, cfg.E, cfg.E_loc, cfg.k, cfg.lengths, cfg.has_shared, n_streams))
    w = inputs.make_weights(cfg, "cuda")
    if mbs is None:
        mbs = inputs.make_microbatches(cfg, "cuda")
    ow = CachedWeights(oracle.OracleWeights(w, "fp8"))
    streams = [torch.cuda.Stream() for _ in range(n_streams)] if n_streams > 1 else None
    Tmax = max(max(mb.ids.shape[0] for mb in mbs), 1)
    with ExpertStage(cfg, w, n_slots=len(mbs), max_tokens=Tmax) as st:
        poison_workspace(st)
        outs, slots, _ = gpu_run(st, mbs, streams=streams)
        errs = []
        for mb, ob, sl in zip(mbs, outs, slots):
            ref = oracle_run(cfg, ow, mb)
            view = st.view(sl)
            check_dispatch(view, ref, cfg, mb)
            errs.append(check_outputs(ob, ref, FP8_TOL, cfg.name))
            check_expert_rows(view, ref, cfg, FP8_TOL, cfg.name)
        log("  rel-L2 per micro-batch: %s" % ["%.2e" % e for e in errs])


def test_fp8_tiny():
    _case(inputs.scaled(inputs.CONFIGS["c0"], dtype="fp8", name="c0f8"))


@pytest.mark.parametrize("T,d,f,E,E_loc,k", [
    (700, 1024, 384, 16, 4, 4),
    (333, 640, 256, 8, 3, 2),
    (257, 256, 128, 1, 1, 1),
])
def test_fp8_multi_tile(T, d, f, E, E_loc, k):
    _case(inputs.MoEConfig("f8mt", d=d, f=f, E=E, e0=0, E_loc=E_loc, k=k, lengths=(T,),
                           dtype="fp8", seed=11))


def test_fp8_shared_expert():
    _case(inputs.MoEConfig("f8sh", d=512, f=256, E=12, e0=2, E_loc=4, k=3, lengths=(300,),
                           has_shared=True, dtype="fp8", seed=12))


def test_c4_fp8_skewed_four_streams():
    _case(inputs.CONFIGS["c4"], n_streams=4)


def test_fp8_many_row_tiles_per_group():
    """fp8 with 13-14 row tiles per expert (bands of 4 row tiles, several
    bands per group) and more tiles than CUs; d = 1024, f = 512, about 26k
    routed rows; every row is checked."""
    _case(inputs.MoEConfig("f8band", d=1024, f=512, E=16, e0=0, E_loc=8, k=8, lengths=(6500,),
                           dtype="fp8", seed=21))


def test_fp8_edge_cases():
    """Crafted routings around the fp8 kernel's 128-token tiles: one token,
    all slots masked, one expert taking both slots of 300 tokens (600 rows),
    127 / 128 / 129 rows on one expert, and a mixed routing with masks."""
    cfg = inputs.MoEConfig("f8edge", d=256, f=128, E=8, e0=0, E_loc=4, k=2, lengths=(0,),
                           dtype="fp8", seed=15)
    rng = np.random.default_rng(15)

    def rows_on(e, n, T):
        ids = np.full((T, 2), -1, np.int32)
        ids[:n, 0] = e
        ids[n:, 0] = rng.integers(4, 8, T - n)          # the rest go to non-local experts
        return ids

    cases = {
        "one_token": np.array([[1, 3]], np.int32),
        "all_masked": np.full((9, 2), -1, np.int32),
        "one_expert_both_slots": np.full((300, 2), 2, np.int32),
        "tile_minus_one": rows_on(1, 127, 200),
        "tile": rows_on(1, 128, 200),
        "tile_plus_one": rows_on(3, 129, 200),
        "mixed": rng.integers(-1, 8, size=(513, 2)).astype(np.int32),
    }
    for name, ids in cases.items():
        T = ids.shape[0]
        log("fp8 edge case %s T=%d" % (name, T))
        x = (torch.randn((T, cfg.d), generator=torch.Generator("cuda").manual_seed(T),
                         device="cuda")).to(torch.bfloat16)
        mb = inputs.MicroBatch(x=x, ids=ids, w=rng.random((T, 2)).astype(np.float32))
        _case(inputs.scaled(cfg, name="f8edge_" + name, lengths=(T,)), [mb])


def test_c1p_fp8_full_size():
    """The fp8 gate/up and down launches as bench.py times them at T = 32768
    (8 local experts of about 1015 rows); every row is checked."""
    _case(inputs.CONFIGS["c1p_fp8"])


def test_c3_fp8_full_size_with_shared_expert():
    """The fp8 launches as bench.py times them at T = 16384 with 32 local
    experts and the shared expert over all tokens; every row is checked."""
    _case(inputs.CONFIGS["c3_fp8"])
