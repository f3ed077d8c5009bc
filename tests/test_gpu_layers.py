"""GPU parity of the layer-oblivious weights (the MoE Super Kernel idea of
section 3.4.2): one stage holds the experts of L layers, a micro-batch names
its layer through an int32 in device memory, and the GEMM kernels resolve the
weights from the stage's on-device address table when they run.

Each output is compared with the oracle run on that layer's weights; the
layers' weights differ, so a wrong table entry fails the comparison.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_22541_amd import inputs
from paper_2606_22541_amd import moe_stage as C
from paper_2606_22541_amd.stage import ExpertStage, bf16_bits, quantize_fp8, to_device_routing

from gpu_common import BF16_TOL, FP8_TOL, check_outputs, log, oracle_run

pytestmark = pytest.mark.gpu

L = 3


def _setup(dtype, seed):
    cfg = inputs.MoEConfig("layers", d=512, f=256, E=12, e0=2, E_loc=4, k=3, lengths=(300,),
                           has_shared=True, dtype=dtype, seed=seed)
    ws = [inputs.make_weights(inputs.scaled(cfg, seed=100 + l), "cuda") for l in range(L)]
    mb = inputs.make_microbatches(cfg, "cuda")[0]
    refs = [oracle_run(cfg, oracle.OracleWeights(ws[l], dtype), mb) for l in range(L)]
    ids, w = to_device_routing(mb.ids, mb.w)
    x, xs = mb.x.to("cuda"), None
    if dtype == "fp8":
        x, xs = quantize_fp8(x)
    torch.cuda.synchronize()
    return cfg, ws, mb, refs, (x, xs, ids, w)


def _run(st, cfg, tensors, layer_ids):
    """Submits one micro-batch per entry of layer_ids (a device int32 tensor
    or None) and returns the output tensors."""
    x, xs, ids, w = tensors
    outs = []
    keep = []
    for lid in layer_ids:
        out = torch.full((ids.shape[0], cfg.d), float("nan"), dtype=torch.bfloat16, device="cuda")
        m = st.microbatch(x, ids, w, out, xs, layer_id=lid)
        keep.append(m)
        st.submit(m)
        outs.append(out)
    return outs


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
def test_layers_out_of_order(dtype):
    tol = FP8_TOL if dtype == "fp8" else BF16_TOL
    log("layer table %s: L=%d, layers submitted 2 0 1 2 0 then NULL" % (dtype, L))
    cfg, ws, mb, refs, tensors = _setup(dtype, 21)
    # the layers' results really differ
    assert oracle.rel_l2(refs[0]["out"], refs[1]["out"]) > 0.5
    order = [2, 0, 1, 2, 0]
    lids = [torch.tensor([l], dtype=torch.int32, device="cuda") for l in order]
    with ExpertStage(cfg, ws, n_slots=2, max_tokens=300) as st:
        assert st.n_layers == L
        outs = _run(st, cfg, tensors, lids + [None])
        st.sync()
        torch.cuda.synchronize()
        for l, out in zip(order + [0], outs):
            check_outputs(bf16_bits(out), refs[l], tol, "layer %d" % l)


def test_layer_id_computed_on_device():
    """The host never reads the id: it is derived from the routing on the
    stream, after which the host compares with the oracle of that layer."""
    cfg, ws, mb, refs, tensors = _setup("bf16", 22)
    x, xs, ids, w = tensors
    lid = (ids.to(torch.int64).sum() % L).to(torch.int32).reshape(1)
    with ExpertStage(cfg, ws, n_slots=1, max_tokens=300) as st:
        (out,) = _run(st, cfg, tensors, [lid])
        st.sync()
        torch.cuda.synchronize()
    want = int(np.asarray(mb.ids, dtype=np.int64).sum() % L)
    log("device-computed layer id %d" % want)
    check_outputs(bf16_bits(out), refs[want], BF16_TOL, "layer %d" % want)


def test_bad_layer_id_is_clamped_and_reported():
    cfg, ws, mb, refs, tensors = _setup("bf16", 23)
    lids = [torch.tensor([v], dtype=torch.int32, device="cuda") for v in (7, -4)]
    with ExpertStage(cfg, ws, n_slots=2, max_tokens=300) as st:
        outs = _run(st, cfg, tensors, lids)
        with pytest.raises(C.MoEStageError) as e:
            st.sync()
        assert e.value.status == C.MOE_EBADLAYER
        torch.cuda.synchronize()
        check_outputs(bf16_bits(outs[0]), refs[L - 1], BF16_TOL, "id 7 -> layer %d" % (L - 1))
        check_outputs(bf16_bits(outs[1]), refs[0], BF16_TOL, "id -4 -> layer 0")
        # the error is cleared by the sync that reported it
        good = torch.tensor([1], dtype=torch.int32, device="cuda")
        (out,) = _run(st, cfg, tensors, [good])
        st.sync()
        torch.cuda.synchronize()
        check_outputs(bf16_bits(out), refs[1], BF16_TOL, "layer 1 after the error")
