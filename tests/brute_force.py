"""Pure-Python brute force of the expert stage for tiny inputs.

Written independently of the oracle (no numpy in the arithmetic, no shared
helpers): nested loops, ``math.exp`` and Python's stable ``sorted``.  It is
used to pin the oracle on inputs small enough to enumerate.
"""
import math


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
