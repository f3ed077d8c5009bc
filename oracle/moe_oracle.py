"""CPU oracle of the MoE expert stage, in fp64.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import this module.  It shares no
code with the HIP path; the only common module is the seeded input generator.

What the stage computes (one device's share of the experts of a MoE layer):

* Sparse experts replace the dense FFN and each token activates its top-k
  routed experts plus, in DeepSeek-V3, one shared expert (background on MoE
  architectures; evaluation methodology).
* The MoE device groups the tokens it receives by expert, using per-expert
  token counts as metadata (section "Asynchronous Dispatch", Table 2).
* The expert computation is a grouped matrix multiplication with the hidden
  states on the left and each expert's weights on the right (section
  "Bubble-Free Kernel Dispatching").
* The results return as k rows per token and are reduced with the routing
  weights at the receiver (section "Asynchronous Combine", Table 2).

The paper does not write the expert FFN or the combine formula.  This oracle
takes SwiGLU experts, y = W_down (SiLU(W_gate x) * W_up x), applies the
routing weights to the expert outputs, and sums a token's results in
ascending j.  For rows that arrive already grouped by expert (the receive
region with sender-supplied counts), a negative count is read as 0 and rows
past the buffer are dropped in expert order.

Arithmetic: every operand is an exact bf16 (or dequantised e4m3) value held in
fp64, products and sums are fp64, nothing is rounded except where the fp8
variant quantises the intermediate activation h: per row and 128 channels,
scale = amax / 448 and code = e4m3(h / scale), both in fp32, the rule the
activations are quantised by.  The counting sort is plain C
(``dispatch.c``); the dense products use numpy's float64 matmul as a library
primitive.
"""
from __future__ import annotations

import ctypes
import math
from typing import Dict, Iterable, Optional

import numpy as np

from . import build as _build

# ---------------------------------------------------------------------------
# Counting-sort dispatch (C)
# ---------------------------------------------------------------------------
_lib = None


def _load():
    global _lib
    if _lib is None:
        _lib = ctypes.CDLL(_build.ensure_built())
        p = ctypes.POINTER(ctypes.c_int32)
        _lib.oracle_dispatch.restype = ctypes.c_int32
        _lib.oracle_dispatch.argtypes = [ctypes.c_int32] * 5 + [p] * 6
    return _lib


def _i32p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def dispatch(ids: np.ndarray, E: int, e0: int, E_loc: int) -> Dict[str, np.ndarray]:
    """Histogram, offsets and stable counting-sort permutation of the slots.

    ``ids`` is [T, k] int32 with -1 for masked slots.  Returns counts [E],
    offsets [E_loc+1], slot_of_row [N_loc], row_of_slot [T*k], n_loc, n_bad.
    """
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    T, k = ids.shape
    counts = np.zeros(E, np.int32)
    offsets = np.zeros(E_loc + 1, np.int32)
    slot_of_row = np.zeros(max(T * k, 1), np.int32)       # repeated ids: every slot may be local
    row_of_slot = np.zeros(max(T * k, 1), np.int32)
    n_bad = np.zeros(1, np.int32)
    n_loc = _load().oracle_dispatch(T, k, E, e0, E_loc, _i32p(ids), _i32p(counts),
                                    _i32p(offsets), _i32p(slot_of_row),
                                    _i32p(row_of_slot), _i32p(n_bad))
    if n_loc < 0:
        raise MemoryError("oracle_dispatch")
    return dict(counts=counts, offsets=offsets, slot_of_row=slot_of_row[:n_loc].copy(),
                row_of_slot=row_of_slot[:T * k].copy(), n_loc=int(n_loc), n_bad=int(n_bad[0]))


# ---------------------------------------------------------------------------
# Number formats
# ---------------------------------------------------------------------------
def bf16_bits_to_f64(u16: np.ndarray) -> np.ndarray:
    """bf16 is the top half of an IEEE fp32; widening is exact."""
    return (np.asarray(u16, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def bf16_bits_to_f32(u16: np.ndarray) -> np.ndarray:
    return (np.asarray(u16, np.uint16).astype(np.uint32) << 16).view(np.float32)


def round_f32_to_bf16(v: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (nearest, ties to even on the 16 dropped
    bits) and return them as fp32.  Inputs are finite."""
    u = np.asarray(v, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def _e4m3_value(code: int) -> float:
    """OCP 8-bit float E4M3FN: sign bit 7, 4 exponent bits (bias 7), 3
    mantissa bits; exponent field 0 encodes subnormals m/8 * 2^-6; the
    all-ones exponent with all-ones mantissa is NaN and there is no infinity,
    so the largest finite magnitude is 1.75 * 2^8 = 448."""
    sign = -1.0 if code & 0x80 else 1.0
    e = (code >> 3) & 0xF
    m = code & 0x7
    if e == 0xF and m == 0x7:
        return math.nan
    if e == 0:
        return sign * (m / 8.0) * 2.0 ** -6
    return sign * (1.0 + m / 8.0) * 2.0 ** (e - 7)


E4M3_TABLE = np.array([_e4m3_value(c) for c in range(256)], dtype=np.float64)
E4M3_MAX = 448.0
# Positive finite magnitudes in code order 0x00..0x7E (monotone increasing).
_E4M3_POS = E4M3_TABLE[:0x7F].copy()


def e4m3_decode(codes: np.ndarray) -> np.ndarray:
    return E4M3_TABLE[np.asarray(codes, np.uint8)]


def e4m3_encode(v: np.ndarray) -> np.ndarray:
    """Round fp32 values to E4M3FN, nearest with ties to even, saturating to +-448.

    For |v| in binade [2^e, 2^(e+1)) with e >= -6 the spacing of E4M3 values
    is 2^(e-3); below 2^-6 the spacing is the subnormal step 2^-9.  Rounding
    |v| / spacing to the nearest integer, ties to even, gives the nearest
    representable value; its code follows from the monotone code order.
    The sign bit is copied from v (so -0.0 encodes as 0x80).
    """
    v = np.asarray(v, dtype=np.float32).astype(np.float64)
    a = np.abs(v)
    _, ex = np.frexp(a)                 # a = mant * 2^ex, mant in [0.5, 1)
    e = np.maximum(ex - 1, -6)          # floor(log2 a), clamped to the subnormal binade
    spacing = np.ldexp(1.0, e - 3)
    mag = np.rint(a / spacing) * spacing
    mag = np.minimum(mag, E4M3_MAX)
    code = np.searchsorted(_E4M3_POS, mag).astype(np.uint8)
    assert np.array_equal(_E4M3_POS[code], mag), "value not representable"
    code = code | np.where(np.signbit(v), 0x80, 0).astype(np.uint8)
    return code


def quantize_groups(v: np.ndarray, group: int = 128):
    """Per-row, per-``group``-channel e4m3 quantisation with fp32 scales.

    For each group: amax = max |v| (fp32), scale = amax / 448 in fp32 (1 when
    amax is 0), code = e4m3(v / scale) with the quotient rounded to fp32.
    Returns codes [R, C] uint8 and scales [R, C/group] float32.
    """
    v = np.asarray(v, dtype=np.float32)
    R, C = v.shape
    assert C % group == 0
    g = v.reshape(R, C // group, group)
    amax = np.abs(g).max(axis=2) if R else np.zeros((0, C // group), np.float32)
    scale = np.where(amax > 0, amax / np.float32(E4M3_MAX), np.float32(1.0)).astype(np.float32)
    q = (g / scale[:, :, None]).astype(np.float32)
    codes = e4m3_encode(q).reshape(R, C)
    return codes, scale


def dequantize_groups(codes: np.ndarray, scales: np.ndarray, group: int = 128) -> np.ndarray:
    R, C = codes.shape
    vals = e4m3_decode(codes).reshape(R, C // group, group)
    return (vals * scales.astype(np.float64)[:, :, None]).reshape(R, C)


def dequantize_blocks(codes: np.ndarray, scales: np.ndarray, block: int = 128) -> np.ndarray:
    """[R, C] codes with one fp32 scale per block x block tile -> fp64."""
    R, C = codes.shape
    vals = e4m3_decode(codes).reshape(R // block, block, C // block, block)
    return (vals * scales.astype(np.float64)[:, None, :, None]).reshape(R, C)


# ---------------------------------------------------------------------------
# Expert FFN
# ---------------------------------------------------------------------------
def silu(z: np.ndarray) -> np.ndarray:
    """SiLU(z) = z / (1 + e^-z) in fp64."""
    with np.errstate(over="ignore"):
        return z / (1.0 + np.exp(-z))


def swiglu_ffn(X: np.ndarray, Wg: np.ndarray, Wu: np.ndarray, Wd: np.ndarray,
               quantize_h: bool = False):
    """y = W_down (SiLU(W_gate x) * W_up x) for each row x of X, in fp64.

    X [n, d]; Wg, Wu [f, d]; Wd [d, f].  With ``quantize_h`` (the fp8 variant)
    the intermediate h is quantised per row and 128 channels to e4m3 before
    the down projection, by the same rule as the activations: the scale and
    the quotient are fp32 quantities, so h enters the quantiser as its fp32
    value (one rounding of the fp64 h) and nothing else is rounded.
    Returns (y [n, d], h [n, f]).
    """
    g = X @ Wg.T
    u = X @ Wu.T
    h = silu(g) * u
    if quantize_h:
        codes, scales = quantize_groups(h.astype(np.float32))
        h = dequantize_groups(codes, scales)
    y = h @ Wd.T
    return y, h


# ---------------------------------------------------------------------------
# Whole stage
# ---------------------------------------------------------------------------
def _np_bits(t, dtype=None):
    """A torch tensor or numpy array of raw bf16 bits / e4m3 codes / fp32 -> numpy."""
    if hasattr(t, "detach"):
        import torch  # only for moving generator tensors to numpy
        t = t.detach().cpu().contiguous()
        if t.dtype == torch.bfloat16:
            return t.view(torch.int16).numpy().view(np.uint16)
        if t.dtype == torch.float8_e4m3fn:
            return t.view(torch.uint8).numpy()
        return t.numpy()
    return np.asarray(t)


class OracleWeights:
    """Host copies of the local (and shared) expert weights, decoded to fp64
    one expert at a time."""

    def __init__(self, w, dtype: str):
        self.dtype = dtype
        if dtype == "bf16":
            self.gate = _np_bits(w.w_gate, np.uint16)
            self.up = _np_bits(w.w_up, np.uint16)
            self.down = _np_bits(w.w_down, np.uint16)
            if w.sh_gate is not None:
                self.sh = (_np_bits(w.sh_gate, np.uint16)[0], _np_bits(w.sh_up, np.uint16)[0],
                           _np_bits(w.sh_down, np.uint16)[0])
            else:
                self.sh = None
        else:
            self.gate = (_np_bits(w.w_gate, np.uint8), _np_bits(w.s_gate, np.float32))
            self.up = (_np_bits(w.w_up, np.uint8), _np_bits(w.s_up, np.float32))
            self.down = (_np_bits(w.w_down, np.uint8), _np_bits(w.s_down, np.float32))
            if w.sh_gate is not None:
                self.sh = ((_np_bits(w.sh_gate, np.uint8)[0], _np_bits(w.sh_s_gate, np.float32)[0]),
                           (_np_bits(w.sh_up, np.uint8)[0], _np_bits(w.sh_s_up, np.float32)[0]),
                           (_np_bits(w.sh_down, np.uint8)[0], _np_bits(w.sh_s_down, np.float32)[0]))
            else:
                self.sh = None

    def _dec(self, m):
        if self.dtype == "bf16":
            return bf16_bits_to_f64(m)
        return dequantize_blocks(m[0], m[1])

    def expert(self, i: int):
        if self.dtype == "bf16":
            return (bf16_bits_to_f64(self.gate[i]), bf16_bits_to_f64(self.up[i]),
                    bf16_bits_to_f64(self.down[i]))
        return tuple(dequantize_blocks(m[0][i], m[1][i]) for m in (self.gate, self.up, self.down))

    def shared(self):
        return tuple(self._dec(m) for m in self.sh)


def stage_inputs_x(x_bits: np.ndarray, dtype: str):
    """The activations the expert FFN sees, in fp64.

    bf16: the bf16 values themselves.  fp8: the sender-side quantiser
    (per token, per 128 channels) followed by dequantisation; also returns
    the codes and scales so tests can compare them with the stage's."""
    if dtype == "bf16":
        return bf16_bits_to_f64(x_bits), None, None
    codes, scales = quantize_groups(bf16_bits_to_f32(x_bits))
    return dequantize_groups(codes, scales), codes, scales


def run_stage(cfg, weights: OracleWeights, x_bits: np.ndarray, ids: np.ndarray,
              w: np.ndarray, *, combine_mode: int = 0, base: Optional[np.ndarray] = None,
              tokens: Optional[Iterable[int]] = None) -> Dict[str, object]:
    """The expert stage on one micro-batch.

    cfg supplies d, f, E, e0, E_loc, k, has_shared and dtype.  ``base`` is the
    previous content of ``out`` as fp64 [T, d] (accumulate mode).  When
    ``tokens`` is given, FFN rows and outputs are computed only for those
    tokens (dispatch is always complete).

    Returns dispatch results, ``rows`` (row indices whose y was computed),
    ``y`` [len(rows), d], ``tok`` (token indices) and ``out`` [len(tok), d].
    """
    ids = np.ascontiguousarray(ids, np.int32)
    T, k = ids.shape
    d = cfg.d
    quant = cfg.dtype == "fp8"
    disp = dispatch(ids, cfg.E, cfg.e0, cfg.E_loc)
    sor, ros, offs = disp["slot_of_row"], disp["row_of_slot"], disp["offsets"]
    tok = np.arange(T) if tokens is None else np.unique(np.asarray(list(tokens), np.int64))
    x_all, x_codes, x_scales = stage_inputs_x(x_bits, cfg.dtype)

    # Rows needed: every local slot of a selected token.
    sel_slots = (tok[:, None] * k + np.arange(k)[None, :]).ravel()
    rows = np.sort(ros[sel_slots][ros[sel_slots] >= 0]) if T else np.zeros(0, np.int64)
    y = np.zeros((rows.size, d), np.float64)
    for i in range(cfg.E_loc):
        lo, hi = offs[i], offs[i + 1]
        mine = np.nonzero((rows >= lo) & (rows < hi))[0]
        if mine.size == 0:
            continue
        Wg, Wu, Wd = weights.expert(i)
        Xe = x_all[sor[rows[mine]] // k]
        y[mine], _ = swiglu_ffn(Xe, Wg, Wu, Wd, quantize_h=quant)

    out = np.zeros((tok.size, d), np.float64)
    if combine_mode == 1:
        assert base is not None
        out += base[tok]
    if cfg.has_shared and tok.size:
        Sg, Su, Sd = weights.shared()
        ysh, _ = swiglu_ffn(x_all[tok], Sg, Su, Sd, quantize_h=quant)
        out += ysh
    pos = {int(r): p for p, r in enumerate(rows)}
    for j in range(k):                          # ascending j
        r = ros[tok * k + j] if T else np.zeros(0, np.int32)
        has = np.nonzero(r >= 0)[0]
        if has.size:
            idx = np.array([pos[int(v)] for v in r[has]], np.int64)
            out[has] += w[tok[has], j].astype(np.float64)[:, None] * y[idx]
    res = dict(disp)
    res.update(rows=rows, y=y, tok=tok, out=out, x_codes=x_codes, x_scales=x_scales)
    return res


def grouped_counts(counts, n_rows: int) -> np.ndarray:
    """The per-expert counts a pre-grouped batch is read with: in expert
    order, a negative count is taken as 0 and an expert keeps only the rows
    that still fit in the n_rows-row buffer (the stage reports either
    change as an error; this is the reading the results are defined by)."""
    kept = []
    used = 0
    for c in np.asarray(counts, np.int64).tolist():
        c = max(c, 0)
        keep = min(c, max(0, n_rows - used))
        kept.append(keep)
        used += keep
    return np.array(kept, np.int64)


def run_grouped(cfg, weights: OracleWeights, rows_x: np.ndarray, counts) -> Dict[str, object]:
    """Expert FFN of rows that arrive grouped by local expert (the MoE-side
    receive region of section 3.2.1 and Table 2: the senders supply the
    per-expert token counts and one payload row per (token, local expert)
    pair).  Rows [c_0 + ... + c_{i-1}, + c_i) belong to local expert i.

    rows_x: fp64 [n, d], the activations as the FFN sees them (bf16 values,
    or dequantised e4m3 codes in fp8 mode).  Returns the counts actually
    used (``grouped_counts``) and ``y`` [sum of them, d]; no routing weight
    is applied (the weighted sum of a token's results is formed where they
    return to, section 3.2.2)."""
    rows_x = np.asarray(rows_x, np.float64)
    kept = grouped_counts(counts, rows_x.shape[0])
    quant = cfg.dtype == "fp8"
    y = np.zeros((int(kept.sum()), cfg.d), np.float64)
    lo = 0
    for i, c in enumerate(kept.tolist()):
        if c:
            Wg, Wu, Wd = weights.expert(i)
            y[lo:lo + c], _ = swiglu_ffn(rows_x[lo:lo + c], Wg, Wu, Wd, quantize_h=quant)
        lo += c
    return dict(counts=kept, y=y)


def rel_l2(a: np.ndarray, ref: np.ndarray) -> float:
    """||a - ref||_2 / ||ref||_2 in fp64 (0 if both are zero)."""
    a = np.asarray(a, np.float64)
    ref = np.asarray(ref, np.float64)
    num = float(np.sqrt(np.sum((a - ref) ** 2)))
    den = float(np.sqrt(np.sum(ref ** 2)))
    if den == 0.0:
        return 0.0 if num == 0.0 else math.inf
    return num / den
