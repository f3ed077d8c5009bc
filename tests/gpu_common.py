"""Helpers shared by the GPU parity tests: run the HIP stage and the oracle on
the same seeded inputs and compare them."""
import numpy as np
import torch

import oracle
from paper_2606_22541_amd import inputs
from paper_2606_22541_amd import moe_stage as C
from paper_2606_22541_amd.stage import ExpertStage, bf16_bits, quantize_fp8, to_device_routing

BF16_TOL = 1e-2     # rel-L2 bound for the bf16 path
FP8_TOL = 3e-2      # rel-L2 bound for the fp8 path


def log(msg):
    print(msg, flush=True)


def bits_to_f64(u16):
    return oracle.bf16_bits_to_f64(u16)


def gpu_run(stage, mbs, *, streams=None, mode=C.MOE_COMBINE_OVERWRITE, out_init=None):
    """Submits every micro-batch (round-robin over `streams`) and returns the
    outputs as bf16 bit arrays plus the slot each used."""
    dev = "cuda"
    prepared = []
    for i, mb in enumerate(mbs):
        T = mb.ids.shape[0]
        ids, w = to_device_routing(mb.ids, mb.w)
        if out_init is not None:
            out = out_init[i].clone()
        else:
            out = torch.full((T, stage.cfg.d), float("nan"), dtype=torch.bfloat16, device=dev)
        x = mb.x.to(dev)
        xs = None
        if stage.fp8:
            x, xs = quantize_fp8(x)
        prepared.append((x, xs, ids, w, out))
    torch.cuda.synchronize()          # inputs ready before other streams read them
    outs, slots, keep = [], [], []
    for i, (x, xs, ids, w, out) in enumerate(prepared):
        s = streams[i % len(streams)] if streams else None
        m = stage.microbatch(x, ids, w, out, xs, mode)
        keep.append((x, xs, ids, w, out, m))
        slots.append(stage.submit(m, s))
        outs.append(out)
    stage.sync()
    torch.cuda.synchronize()
    return [bf16_bits(o) for o in outs], slots, keep


def oracle_run(cfg, ow, mb, tokens=None, mode=0, base=None):
    return oracle.run_stage(cfg, ow, bf16_bits(mb.x), mb.ids, mb.w, combine_mode=mode,
                            base=base, tokens=tokens)


def check_dispatch(view, ref, cfg, mb=None):
    assert np.array_equal(view["counts"], ref["counts"]), "counts differ"
    assert np.array_equal(view["offsets"], ref["offsets"]), "offsets differ"
    assert np.array_equal(view["slot_of_row"], ref["slot_of_row"]), "slot_of_row differs"
    assert np.array_equal(view["row_of_slot"], ref["row_of_slot"]), "row_of_slot differs"
    if mb is not None and "x_perm" in view and cfg.dtype == "bf16":
        src = bf16_bits(mb.x)[ref["slot_of_row"] // cfg.k]
        assert np.array_equal(view["x_perm"], src), "X_perm is not an exact row gather"
    if mb is not None and "x_perm" in view and cfg.dtype == "fp8":
        tok = ref["slot_of_row"] // cfg.k
        assert np.array_equal(view["x_perm"], ref["x_codes"][tok]), "fp8 X_perm codes differ"
        assert np.array_equal(view["x_perm_scales"], ref["x_scales"][tok]), "fp8 X_perm scales differ"


def check_outputs(out_bits, ref, tol, what=""):
    """Compares the GPU output rows of the oracle's tokens."""
    tok = ref["tok"]
    got = bits_to_f64(out_bits[tok])
    want = ref["out"]
    assert np.all(np.isfinite(got)), "non-finite output " + what
    zero = np.all(want == 0, axis=1)
    if np.any(zero):
        assert np.all(out_bits[tok][zero] == 0), "tokens without local slots must be +0.0 " + what
    err = oracle.rel_l2(got, want)
    assert err <= tol, "rel-L2 %.3e > %.1e %s" % (err, tol, what)
    return err


def check_expert_rows(view, ref, cfg, tol, what=""):
    """Per-expert rel-L2 of the GPU's Y_perm rows against the oracle's y."""
    return _check_expert_rows(view, ref, cfg, tol, what)


def _check_expert_rows(view, ref, cfg, tol, what=""):
    """Per-expert rel-L2 of the GPU's Y_perm rows against the oracle's y."""
    rows = ref["rows"]
    if rows.size == 0:
        return {}
    got = bits_to_f64(view["y_perm"][rows])
    errs = {}
    offs = ref["offsets"]
    for i in range(cfg.E_loc):
        m = (rows >= offs[i]) & (rows < offs[i + 1])
        if np.any(m):
            e = oracle.rel_l2(got[m], ref["y"][m])
            errs[i] = e
            assert e <= tol, "expert %d rel-L2 %.3e > %.1e %s" % (i, e, tol, what)
    return errs


def sample_tokens(T, n, seed=0):
    if T <= n:
        return np.arange(T)
    rng = np.random.default_rng(seed)
    s = set(rng.choice(T, size=n - 2, replace=False).tolist()) | {0, T - 1}
    return np.array(sorted(s))
