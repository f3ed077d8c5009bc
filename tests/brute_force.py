"""Pure-Python brute force of the expert stage for tiny inputs.

Written independently of the oracle (no numpy in the arithmetic, no shared
helpers): nested loops, ``math.exp`` and Python's stable ``sorted``.  It is
used to pin the oracle on inputs small enough to enumerate.
"""
import math
import struct


def bf_dispatch(ids, E, e0, E_loc):
    """ids: list of T lists of k ints.  Returns counts, offsets, slot_of_row,
    row_of_slot following the definition (stable order by (expert, slot))."""
    T = len(ids)
    k = len(ids[0]) if T else 0
    counts = [0] * E
    local = []
    for t in range(T):
        for j in range(k):
            e = ids[t][j]
            if 0 <= e < E:
                counts[e] += 1
                if e0 <= e < e0 + E_loc:
                    local.append(t * k + j)
    order = sorted(local, key=lambda s: (ids[s // k][s % k], s))
    offsets = [0]
    for i in range(E_loc):
        offsets.append(offsets[-1] + counts[e0 + i])
    row_of_slot = [-1] * (T * k)
    for r, s in enumerate(order):
        row_of_slot[s] = r
    return counts, offsets, order, row_of_slot


def bf_swiglu(x, Wg, Wu, Wd):
    """One token through one expert with explicit loops.
    x: [d]; Wg, Wu: [f][d]; Wd: [d][f]."""
    d = len(x)
    f = len(Wg)
    h = []
    for i in range(f):
        g = 0.0
        u = 0.0
        for c in range(d):
            g += Wg[i][c] * x[c]
            u += Wu[i][c] * x[c]
        sig = 1.0 / (1.0 + math.exp(-g)) if g > -700 else 0.0
        h.append(g * sig * u)
    y = []
    for c in range(d):
        acc = 0.0
        for i in range(f):
            acc += Wd[c][i] * h[i]
        y.append(acc)
    return y


def bf_stage(x, ids, w, experts, E, e0, E_loc, shared=None, base=None):
    """out[t] = base[t] + shared(x_t) + sum_j w[t][j] * expert_{ids[t][j]}(x_t)
    over local ids, j ascending.  ``experts[i]`` = (Wg, Wu, Wd) for local id
    e0 + i."""
    T = len(x)
    k = len(ids[0]) if T else 0
    d = len(x[0]) if T else 0
    out = []
    for t in range(T):
        acc = list(base[t]) if base is not None else [0.0] * d
        if shared is not None:
            ys = bf_swiglu(x[t], *shared)
            acc = [a + b for a, b in zip(acc, ys)]
        for j in range(k):
            e = ids[t][j]
            if e0 <= e < e0 + E_loc and 0 <= e < E:
                y = bf_swiglu(x[t], *experts[e - e0])
                acc = [a + w[t][j] * b for a, b in zip(acc, y)]
        out.append(acc)
    return out


# ---------------------------------------------------------------------------
# fp8 (OCP E4M3FN) by enumeration
# ---------------------------------------------------------------------------
def _f32(v):
    """Nearest fp32 value of a Python float (IEEE round to nearest even)."""
    return struct.unpack("<f", struct.pack("<f", v))[0]


def bf_e4m3_values():
    """The 127 non-negative finite E4M3FN values, code 0x00..0x7E: exponent
    field e (bias 7) and mantissa m give (1 + m/8) 2^(e-7), or m/8 2^-6 when
    e = 0; code 0x7F is NaN."""
    vals = []
    for code in range(0x7F):
        e, m = code >> 3, code & 7
        vals.append(m / 8.0 * 2.0 ** -6 if e == 0 else (1 + m / 8.0) * 2.0 ** (e - 7))
    return vals


_E4M3 = bf_e4m3_values()


def bf_e4m3_round(v):
    """Nearest E4M3FN value to v (magnitudes above 448 saturate), ties to the
    even code, found by scanning every code."""
    a = min(abs(v), 448.0)
    best = 0
    for c in range(len(_E4M3)):
        db, dc = abs(_E4M3[best] - a), abs(_E4M3[c] - a)
        if dc < db or (dc == db and c % 2 == 0 and best % 2 == 1):
            best = c
    return math.copysign(_E4M3[best], v)


def bf_quantize_dequantize(row, group=128):
    """Quantise a row per group of 128 channels as the fp8 variant does --
    scale = fp32(amax / 448) (1 if amax = 0), code = e4m3(fp32(v / scale)),
    on fp32 inputs -- and return the dequantised values code * scale."""
    row = [_f32(v) for v in row]
    out = []
    for g0 in range(0, len(row), group):
        grp = row[g0:g0 + group]
        amax = max(abs(v) for v in grp)
        s = _f32(amax / 448.0) if amax > 0 else 1.0
        out.extend(bf_e4m3_round(_f32(v / s)) * s for v in grp)
    return out


def bf_swiglu_fp8(x, Wg, Wu, Wd):
    """One token through one expert with h quantised (fp32 value of h, per 128
    channels) before the down projection.  x, W: dequantised fp64 values."""
    d = len(x)
    f = len(Wg)
    h = []
    for i in range(f):
        g = sum(Wg[i][c] * x[c] for c in range(d))
        u = sum(Wu[i][c] * x[c] for c in range(d))
        h.append(g / (1.0 + math.exp(-g)) * u if g > -700 else 0.0)
    hq = bf_quantize_dequantize(h)
    return [sum(Wd[c][i] * hq[i] for i in range(f)) for c in range(d)]
