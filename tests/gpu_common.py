"""Helpers shared by the GPU parity tests: run the HIP stage and the oracle on
the same seeded inputs and compare them."""
import ctypes

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
    if mb is not None and "x_perm_scales" in view and cfg.dtype == "fp8":
        # the e4m3 rows are read by the gate/up GEMM through slot_of_row (checked
        # through H and Y_perm); their scales are gathered, bit-exact
        tok = ref["slot_of_row"] // cfg.k
        assert np.array_equal(view["x_perm_scales"], ref["x_scales"][tok]), "fp8 gathered x scales differ"


def row_rel_l2(got, want):
    """Per-row ||got - want|| / ||want|| (fp64); rows whose reference is zero
    give 0 when the row is zero too, else inf."""
    num = np.sqrt(np.sum((got - want) ** 2, axis=1))
    den = np.sqrt(np.sum(want ** 2, axis=1))
    out = np.zeros(num.shape)
    nz = den > 0
    out[nz] = num[nz] / den[nz]
    out[~nz & (num > 0)] = np.inf
    return out


def _check_rows(got, want, tol, label, what):
    """Every row within `tol` (relative L2 of the row); logs the worst row."""
    if got.shape[0] == 0:
        return 0.0
    errs = row_rel_l2(got, want)
    worst = int(np.argmax(errs))
    log("  %s: %d rows, worst row %d rel-L2 %.3e (whole %.3e)" % (
        label, got.shape[0], worst, errs[worst], oracle.rel_l2(got, want)))
    bad = np.nonzero(errs > tol)[0]
    assert bad.size == 0, "%s: %d rows above %.1e, e.g. row %d at %.3e %s" % (
        label, bad.size, tol, bad[0], errs[bad[0]], what)
    return float(errs[worst])


def check_outputs(out_bits, ref, tol, what=""):
    """Compares the GPU output rows of the oracle's tokens: the whole output
    and every token row within `tol`, no NaN or Inf, and tokens without a
    local slot (overwrite mode) exactly +0.0."""
    tok = ref["tok"]
    got = bits_to_f64(out_bits[tok])
    want = ref["out"]
    assert np.all(np.isfinite(got)), "non-finite output " + what
    zero = np.all(want == 0, axis=1)
    if np.any(zero):
        assert np.all(out_bits[tok][zero] == 0), "tokens without local slots must be +0.0 " + what
    err = oracle.rel_l2(got, want)
    assert err <= tol, "rel-L2 %.3e > %.1e %s" % (err, tol, what)
    _check_rows(got, want, tol, "out rows", what)
    return err


def check_expert_rows(view, ref, cfg, tol, what=""):
    """Per-expert rel-L2 of the GPU's Y_perm rows against the oracle's y."""
    return _check_expert_rows(view, ref, cfg, tol, what)


def _check_expert_rows(view, ref, cfg, tol, what=""):
    """Per-expert rel-L2 of the GPU's Y_perm rows against the oracle's y, and
    every row on its own; every row of Y_perm (and H) below the local row
    count must be finite, which catches a tile that no workgroup wrote when
    the workspace was poisoned with NaN before the run."""
    n = int(ref["offsets"][-1])
    if "y_perm" in view and n:
        assert np.all(np.isfinite(bits_to_f64(view["y_perm"][:n]))), "non-finite Y_perm row " + what
    if "h" in view and n:
        h = view["h"][:n]
        if h.dtype == np.uint16:
            assert np.all(np.isfinite(bits_to_f64(h))), "non-finite H row " + what
        else:     # e4m3 codes: 0x7f / 0xff are NaN
            assert not np.any((h & 0x7F) == 0x7F), "NaN code in H " + what
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
    _check_rows(got, ref["y"], tol, "Y_perm rows", what)
    return errs


def poison_workspace(stage):
    """Fills every slot's H, Y_perm (and shared-expert) rows with NaN bytes
    (0xff: NaN in bf16 and in e4m3), so that a row the GPU never writes
    fails the finiteness checks."""
    hip = _hip()
    cfg = stage.cfg
    eb = 1 if stage.fp8 else 2
    for sl in range(stage.n_slots):
        v = C.moe_stage_query(stage.handle, sl)
        cap = v.capacity_rows
        for ptr, nbytes in ((v.h, cap * cfg.f * eb), (v.y_perm, cap * cfg.d * 2)):
            if ptr and nbytes:
                assert hip.hipMemset(ctypes.c_void_p(ptr), 0xFF, ctypes.c_size_t(nbytes)) == 0
    assert hip.hipDeviceSynchronize() == 0


_hip_handle = None


def _hip():
    global _hip_handle
    if _hip_handle is None:
        _hip_handle = ctypes.CDLL("libamdhip64.so")
        _hip_handle.hipMemset.restype = ctypes.c_int
        _hip_handle.hipMemset.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t]
        _hip_handle.hipDeviceSynchronize.restype = ctypes.c_int
    return _hip_handle


class CachedWeights:
    """OracleWeights whose decoded experts are kept after first use (fp8
    decoding of a DeepSeek-sized expert takes about a second; micro-batches
    of one stage reuse them)."""

    def __init__(self, ow):
        self.ow = ow
        self.dtype = ow.dtype
        self._cache = {}

    def expert(self, i):
        if i not in self._cache:
            self._cache[i] = self.ow.expert(i)
        return self._cache[i]

    def shared(self):
        if "sh" not in self._cache:
            self._cache["sh"] = self.ow.shared()
        return self._cache["sh"]


def band_order_tiles(rows_per_group, N, small_rows=192, tile=256):
    """Tiles of the 256-row GEMM over groups of more than `small_rows` rows
    with N output columns, the persistent grid it runs on (one workgroup per
    CU, a multiple of 8), and whether it takes the size order: a single round,
    or a last round at most half full.  Mirrors the launch's documented rule
    so a test can assert which order a case exercises."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    nt = -(-N // tile)
    total = sum(-(-int(r) // tile) for r in rows_per_group if r > small_rows) * nt
    P = min(cus, total)
    if P >= 8:
        P &= ~7
    tail = total % P if P else 0
    by_size = total <= P or (tail != 0 and 2 * tail <= P)
    return total, P, by_size
