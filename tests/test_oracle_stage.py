"""Pins for the oracle's expert FFN and combine (CPU only): a hand-worked
closed form, pure-Python brute force, and invariants of the definition."""
import json
import os
from types import SimpleNamespace

import numpy as np
import pytest
import torch

import oracle
from brute_force import bf_stage, bf_swiglu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _cfg(**kw):
    base = dict(d=8, f=4, E=6, e0=0, E_loc=3, k=2, has_shared=False, dtype="bf16")
    base.update(kw)
    return SimpleNamespace(**base)


class _W:
    """Oracle weights held directly in fp64 (already exact values)."""
    def __init__(self, experts, shared=None):
        self.experts = experts
        self.sh = shared

    def expert(self, i):
        return self.experts[i]

    def shared(self):
        return self.sh


def _bf16_round(a):
    """Round fp64 -> bf16 values (test inputs only)."""
    f = np.asarray(a, np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    return u


def _rand_problem(rng, T, d, f, E, e0, E_loc, k, mask_p=0.1):
    x_bits = _bf16_round(rng.standard_normal((T, d)))
    ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32) if T else np.zeros((0, k), np.int32)
    ids[rng.random(ids.shape) < mask_p] = -1
    w = rng.random((T, k)).astype(np.float32)
    experts = []
    for _ in range(E_loc):
        experts.append(tuple(oracle.bf16_bits_to_f64(_bf16_round(rng.standard_normal(s) * 0.3))
                             for s in ((f, d), (f, d), (d, f))))
    return x_bits, ids, w, experts


def test_hand_example():
    g = json.load(open(os.path.join(GOLDEN, "swiglu_hand_example.json")))
    x = np.array(g["x"])
    exps = [tuple(np.array(e[n], np.float64) for n in ("w_gate", "w_up", "w_down")) for e in g["experts"]]
    for t in range(2):
        for e in range(2):
            y, _ = oracle.swiglu_ffn(x[t:t + 1], *exps[e])
            np.testing.assert_allclose(y[0], g["y_expected"]["t%d_e%d" % (t, e)], rtol=1e-14)
    cfg = _cfg(d=2, f=1, E=2, e0=0, E_loc=2, k=2)
    res = oracle.run_stage(cfg, _W(exps), _bf16_round(x), np.array(g["ids"], np.int32),
                           np.array(g["w"], np.float32))
    np.testing.assert_allclose(res["out"], g["out_expected"], rtol=1e-14)


@pytest.mark.parametrize("seed", range(4))
def test_ffn_brute_force(seed):
    rng = np.random.default_rng(seed)
    n, d, f = 3, 8, 5                       # d != f catches a transposed operand
    X = rng.standard_normal((n, d))
    Wg, Wu, Wd = rng.standard_normal((f, d)), rng.standard_normal((f, d)), rng.standard_normal((d, f))
    y, _ = oracle.swiglu_ffn(X, Wg, Wu, Wd)
    for r in range(n):
        np.testing.assert_allclose(y[r], bf_swiglu(X[r].tolist(), Wg.tolist(), Wu.tolist(), Wd.tolist()),
                                   rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("seed", range(6))
def test_stage_brute_force(seed):
    rng = np.random.default_rng(100 + seed)
    T, d, f, E, k = int(rng.integers(0, 12)), 8, 4, 6, 2
    e0, E_loc = int(rng.integers(0, 3)), int(rng.integers(1, 4))
    shared = bool(seed % 2)
    x_bits, ids, w, experts = _rand_problem(rng, T, d, f, E, e0, E_loc, k)
    sh = tuple(rng.standard_normal(s) * 0.3 for s in ((f, d), (f, d), (d, f))) if shared else None
    cfg = _cfg(d=d, f=f, E=E, e0=e0, E_loc=E_loc, k=k, has_shared=shared)
    mode = seed % 3 == 2
    base = rng.standard_normal((T, d)) if mode else None
    res = oracle.run_stage(cfg, _W(experts, sh), x_bits, ids, w, combine_mode=int(mode), base=base)
    x = oracle.bf16_bits_to_f64(x_bits)
    want = bf_stage(x.tolist(), ids.tolist(), w.astype(np.float64).tolist(),
                    [tuple(m.tolist() for m in e) for e in experts], E, e0, E_loc,
                    shared=tuple(m.tolist() for m in sh) if sh else None,
                    base=base.tolist() if mode else None)
    if T:
        np.testing.assert_allclose(res["out"], np.array(want), rtol=1e-12, atol=1e-12)
    # token sampling gives the same rows as the full run
    if T > 2:
        sub = oracle.run_stage(cfg, _W(experts, sh), x_bits, ids, w, combine_mode=int(mode), base=base,
                               tokens=[T - 1, 0])
        np.testing.assert_allclose(sub["out"], res["out"][[0, T - 1]], rtol=1e-13, atol=1e-14)


def test_single_expert_equals_dense_ffn():
    """One local expert, k=1, weight 1: the stage is the dense SwiGLU FFN."""
    rng = np.random.default_rng(7)
    T, d, f = 16, 24, 12
    x_bits, _, _, experts = _rand_problem(rng, T, d, f, 1, 0, 1, 1, mask_p=0)
    ids = np.zeros((T, 1), np.int32)
    w = np.ones((T, 1), np.float32)
    res = oracle.run_stage(_cfg(d=d, f=f, E=1, E_loc=1, k=1), _W(experts), x_bits, ids, w)
    x = oracle.bf16_bits_to_f64(x_bits)
    Wg, Wu, Wd = experts[0]
    g = x @ Wg.T
    dense = ((g / (1 + np.exp(-g))) * (x @ Wu.T)) @ Wd.T
    np.testing.assert_allclose(res["out"], dense, rtol=1e-13, atol=1e-13)
    assert res["counts"].tolist() == [T] and res["slot_of_row"].tolist() == list(range(T))


def test_closed_forms_and_linearity():
    rng = np.random.default_rng(8)
    T, d, f, E, k = 10, 16, 8, 4, 2
    x_bits, ids, w, experts = _rand_problem(rng, T, d, f, E, 0, E, k, mask_p=0)
    cfg = _cfg(d=d, f=f, E=E, E_loc=E, k=k)
    # W_up = 0 -> exactly zero output
    zero_up = [(g, np.zeros_like(u), dn) for g, u, dn in experts]
    assert np.all(oracle.run_stage(cfg, _W(zero_up), x_bits, ids, w)["out"] == 0)
    # x = 0 -> exactly zero (SiLU(0) = 0)
    assert np.all(oracle.run_stage(cfg, _W(experts), np.zeros_like(x_bits), ids, w)["out"] == 0)
    # scaling W_down by 2 scales the output exactly by 2
    two = [(g, u, 2 * dn) for g, u, dn in experts]
    a = oracle.run_stage(cfg, _W(experts), x_bits, ids, w)["out"]
    b = oracle.run_stage(cfg, _W(two), x_bits, ids, w)["out"]
    assert np.array_equal(b, 2 * a)
    # routing weights enter linearly, per slot
    c = oracle.run_stage(cfg, _W(experts), x_bits, ids, (w * 0.5).astype(np.float32))["out"]
    np.testing.assert_allclose(c, a * 0.5, rtol=1e-13, atol=1e-15)


def test_identical_experts_and_unit_weights_reproduce_expert_output():
    """All experts local and identical, weights sum to 1: out = y(x)."""
    rng = np.random.default_rng(9)
    T, d, f, E, k = 12, 16, 8, 4, 4
    x_bits, ids, _, experts = _rand_problem(rng, T, d, f, E, 0, E, k, mask_p=0)
    same = [experts[0]] * E
    w = np.full((T, k), 0.25, np.float32)
    res = oracle.run_stage(_cfg(d=d, f=f, E=E, E_loc=E, k=k), _W(same), x_bits, ids, w)
    y, _ = oracle.swiglu_ffn(oracle.bf16_bits_to_f64(x_bits), *experts[0])
    np.testing.assert_allclose(res["out"], y, rtol=1e-13, atol=1e-14)


def test_empty_experts_contribute_nothing():
    rng = np.random.default_rng(10)
    T, d, f, E, k = 9, 16, 8, 8, 2
    x_bits, _, w, experts = _rand_problem(rng, T, d, f, E, 0, 4, k, mask_p=0)
    ids = rng.choice([0, 2, 5, 7], size=(T, k)).astype(np.int32)     # locals 1 and 3 unused
    nan = tuple(np.full_like(m, np.nan) for m in experts[1])
    poisoned = [experts[0], nan, experts[2], nan]
    res = oracle.run_stage(_cfg(d=d, f=f, E=E, E_loc=4, k=k), _W(poisoned), x_bits, ids, w)
    assert np.all(np.isfinite(res["out"]))
    assert res["counts"][1] == 0 and res["counts"][3] == 0


def test_token_permutation_equivariance():
    rng = np.random.default_rng(11)
    T, d, f, E, k = 14, 16, 8, 6, 3
    x_bits, ids, w, experts = _rand_problem(rng, T, d, f, E, 1, 3, k)
    cfg = _cfg(d=d, f=f, E=E, e0=1, E_loc=3, k=k)
    perm = rng.permutation(T)
    a = oracle.run_stage(cfg, _W(experts), x_bits, ids, w)["out"]
    b = oracle.run_stage(cfg, _W(experts), x_bits[perm], ids[perm], w[perm])["out"]
    assert np.array_equal(b, a[perm])


def test_fp8_stage_brute_force():
    """fp8: x and W enter through their e4m3 values times scales, and h is
    quantised per row and 128 channels from its fp32 value before the down
    projection.  Checked against a pure-Python rebuild whose quantiser scans
    every e4m3 code (no oracle helper), with two 128-blocks along d so that a
    transposed block scale fails.  A bf16 rounding of h before quantising
    flips about one code in 60 here and fails too."""
    from brute_force import bf_quantize_dequantize, bf_swiglu_fp8
    rng = np.random.default_rng(12)
    T, d, f, E, k, E_loc = 4, 256, 128, 3, 2, 2
    x_bits = _bf16_round(rng.standard_normal((T, d)))
    ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    w = rng.random((T, k)).astype(np.float32)
    codes = [rng.integers(0, 0x7E, size=s).astype(np.uint8) | (rng.integers(0, 2, size=s).astype(np.uint8) << 7)
             for s in ((E_loc, f, d), (E_loc, f, d), (E_loc, d, f))]
    scales = [np.abs(rng.standard_normal(s)).astype(np.float32) * 1e-3 + 1e-4
              for s in ((E_loc, f // 128, d // 128), (E_loc, f // 128, d // 128), (E_loc, d // 128, f // 128))]
    wts = SimpleNamespace(w_gate=codes[0], w_up=codes[1], w_down=codes[2],
                          s_gate=scales[0], s_up=scales[1], s_down=scales[2], sh_gate=None)
    ow = oracle.OracleWeights(wts, "fp8")
    cfg = _cfg(d=d, f=f, E=E, e0=0, E_loc=E_loc, k=k, dtype="fp8")
    res = oracle.run_stage(cfg, ow, x_bits, ids, w)

    vals = bf_e4m3_table()

    def deq(c, s, e):
        R, Cn = c.shape[1], c.shape[2]
        return [[vals[int(c[e, i, j])] * float(s[e, i // 128, j // 128]) for j in range(Cn)] for i in range(R)]

    xf = [[float(v) for v in row] for row in oracle.bf16_bits_to_f32(x_bits)]
    xd = [bf_quantize_dequantize(row) for row in xf]
    W = [tuple(deq(codes[m], scales[m], e) for m in range(3)) for e in range(E_loc)]
    for t in range(T):
        want = [0.0] * d
        for j in range(k):
            e = int(ids[t, j])
            if e < E_loc:
                y = bf_swiglu_fp8(xd[t], *W[e])
                want = [a + float(w[t, j]) * b for a, b in zip(want, y)]
        np.testing.assert_allclose(res["out"][t], want, rtol=1e-12, atol=1e-12)


def bf_e4m3_table():
    """All 256 E4M3FN codes decoded from sign, exponent and mantissa fields."""
    from brute_force import bf_e4m3_values
    pos = bf_e4m3_values() + [float("nan")]
    return pos + [-v for v in pos]


def test_grouped_counts_reading():
    """Negative counts read as 0; rows past the buffer are dropped in expert order."""
    assert oracle.grouped_counts([3, -2, 5], 6).tolist() == [3, 0, 3]
    assert oracle.grouped_counts([0, 0, 0], 4).tolist() == [0, 0, 0]
    assert oracle.grouped_counts([2, 2], 10).tolist() == [2, 2]
    assert oracle.grouped_counts([7, 1], 5).tolist() == [5, 0]
    assert oracle.grouped_counts([], 3).tolist() == []


@pytest.mark.parametrize("seed", range(3))
def test_grouped_rows_brute_force(seed):
    """Each grouped row is its own expert's FFN, checked row by row against
    the pure-Python SwiGLU; the counts are clamped as read."""
    rng = np.random.default_rng(300 + seed)
    d, f, E_loc = 8, 5, 3
    experts = [tuple(rng.standard_normal(s) * 0.3 for s in ((f, d), (f, d), (d, f)))
               for _ in range(E_loc)]
    counts = [int(c) for c in rng.integers(-1, 5, E_loc)]
    n = int(rng.integers(0, 10))
    X = rng.standard_normal((n, d))
    res = oracle.run_grouped(_cfg(d=d, f=f, E_loc=E_loc), _W(experts), X, counts)
    kept = oracle.grouped_counts(counts, n)
    assert res["y"].shape == (int(kept.sum()), d)
    r = 0
    for e, c in enumerate(kept.tolist()):
        for _ in range(c):
            want = bf_swiglu(X[r].tolist(), *[m.tolist() for m in experts[e]])
            np.testing.assert_allclose(res["y"][r], want, rtol=1e-12, atol=1e-12)
            r += 1


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
def test_grouped_rows_equal_the_dispatched_rows(dtype):
    """Rows laid out as the dispatch groups them (x[slot_of_row // k], the
    local experts' counts) give exactly the stage's per-row results."""
    rng = np.random.default_rng(41)
    T, d, f, E, e0, E_loc, k = 24, 128, 128, 8, 2, 4, 3
    x_bits, ids, w, experts = _rand_problem(rng, T, d, f, E, e0, E_loc, k)
    cfg = _cfg(d=d, f=f, E=E, e0=e0, E_loc=E_loc, k=k, dtype=dtype)
    res = oracle.run_stage(cfg, _W(experts), x_bits, ids, w)
    x_all, _, _ = oracle.stage_inputs_x(x_bits, dtype)
    rows = x_all[res["slot_of_row"] // k]
    counts = res["counts"][e0:e0 + E_loc]
    g = oracle.run_grouped(cfg, _W(experts), rows, counts)
    assert g["counts"].tolist() == counts.tolist()
    np.testing.assert_array_equal(g["y"], res["y"])


def test_rel_l2_hand_values():
    """rel_l2 = ||a - ref||_2 / ||ref||_2 over all elements, worked by hand."""
    assert oracle.rel_l2(np.array([1.1, 0.0]), np.array([1.0, 0.0])) == pytest.approx(0.1, rel=1e-12)
    # |a - ref| = 2, |ref| = 1: 2 (dividing by |a| = 3 would give 2/3; no sqrt gives 4)
    assert oracle.rel_l2(np.array([3.0, 0.0]), np.array([1.0, 0.0])) == pytest.approx(2.0, rel=1e-15)
    # a 3-4-5 triangle: |a - ref| = 5, |ref| = sqrt(4 + 4 + 1) = 3
    assert oracle.rel_l2(np.array([5.0, 6.0, 1.0]), np.array([2.0, 2.0, 1.0])) == pytest.approx(5 / 3, rel=1e-15)
    # the norm runs over every element of a matrix, not per row
    a = np.array([[1.0, 0.0], [0.0, 1.0]])
    ref = np.array([[1.0, 0.0], [0.0, 0.0]])
    assert oracle.rel_l2(a, ref) == pytest.approx(1.0, rel=1e-15)
    assert oracle.rel_l2(2 * ref, ref) == pytest.approx(1.0, rel=1e-15)
    # a zero reference: exact zeros pass, anything else is infinitely wrong
    z = np.zeros((3, 4))
    assert oracle.rel_l2(z, z) == 0.0
    assert oracle.rel_l2(z + 1e-30, z) == float("inf")
    # symmetric in the sign of the error, scale-invariant
    r = np.random.default_rng(0).standard_normal(50)
    e = np.random.default_rng(1).standard_normal(50) * 1e-3
    assert oracle.rel_l2(r + e, r) == pytest.approx(oracle.rel_l2(r - e, r), rel=1e-12)
    assert oracle.rel_l2(8 * (r + e), 8 * r) == pytest.approx(oracle.rel_l2(r + e, r), rel=1e-12)


def _bf16_tensor(vals):
    return torch.tensor(vals, dtype=torch.float32).to(torch.bfloat16)


def test_oracle_weights_bf16_values_and_orientation():
    """OracleWeights built from the checkpoint layout (torch bf16 tensors,
    gate/up [E_loc][f][d], down [E_loc][d][f], shared with a leading 1):
    every matrix keeps its own values and orientation, and the whole stage
    with these weights equals the brute force on the same values."""
    E_loc, f, d = 2, 3, 5
    gate = [[[e * 16 + i * 5 + j + 1 for j in range(d)] for i in range(f)] for e in range(E_loc)]
    up = [[[-(e * 16 + i * 5 + j + 1) / 4 for j in range(d)] for i in range(f)] for e in range(E_loc)]
    down = [[[(e * 16 + i * 3 + j + 1) / 8 for j in range(f)] for i in range(d)] for e in range(E_loc)]
    shg = [[[(i * 5 + j + 1) / 16 for j in range(d)] for i in range(f)]]
    shu = [[[(i * 5 + j + 2) / 32 for j in range(d)] for i in range(f)]]
    shd = [[[-(i * 3 + j + 1) / 64 for j in range(f)] for i in range(d)]]
    w = SimpleNamespace(w_gate=_bf16_tensor(gate), w_up=_bf16_tensor(up), w_down=_bf16_tensor(down),
                        sh_gate=_bf16_tensor(shg), sh_up=_bf16_tensor(shu), sh_down=_bf16_tensor(shd))
    ow = oracle.OracleWeights(w, "bf16")
    for e in range(E_loc):
        g, u, dn = ow.expert(e)
        assert g.shape == (f, d) and u.shape == (f, d) and dn.shape == (d, f)
        assert g.dtype == np.float64
        assert np.array_equal(g, np.array(gate[e])) and np.array_equal(u, np.array(up[e]))
        assert np.array_equal(dn, np.array(down[e]))
    sg, su, sd = ow.shared()
    assert np.array_equal(sg, np.array(shg[0])) and np.array_equal(su, np.array(shu[0]))
    assert np.array_equal(sd, np.array(shd[0])) and sd.shape == (d, f)
    # end to end: a swapped gate/up or a transposed matrix changes these outputs
    rng = np.random.default_rng(5)
    T, E, k = 5, 3, 2
    x_bits = _bf16_round(rng.standard_normal((T, d)) * 0.1)
    ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    wt = rng.random((T, k)).astype(np.float32)
    cfg = _cfg(d=d, f=f, E=E, e0=1, E_loc=E_loc, k=k, has_shared=True)
    res = oracle.run_stage(cfg, ow, x_bits, ids, wt)
    want = bf_stage(oracle.bf16_bits_to_f64(x_bits).tolist(), ids.tolist(),
                    wt.astype(np.float64).tolist(),
                    [(gate[e], up[e], down[e]) for e in range(E_loc)], E, 1, E_loc,
                    shared=(shg[0], shu[0], shd[0]))
    np.testing.assert_allclose(res["out"], np.array(want), rtol=1e-12, atol=1e-12)


def test_oracle_weights_fp8_block_scales():
    """fp8 weights: code values times the scale of their 128x128 block,
    scales indexed [E_loc][rows/128][cols/128] (distinct powers of two, so a
    transposed or shifted block index gives other values)."""
    E_loc, f, d = 2, 128, 256
    rng = np.random.default_rng(6)
    mk = lambda s: (rng.integers(0, 0x7E, size=s).astype(np.uint8) |
                    (rng.integers(0, 2, size=s).astype(np.uint8) << 7))
    cg, cu, cd = mk((E_loc, f, d)), mk((E_loc, f, d)), mk((E_loc, d, f))
    sg = np.array([[[2.0 ** -(e * 8 + bj + 1) for bj in range(2)]] for e in range(E_loc)], np.float32)
    su = np.array([[[2.0 ** -(e * 8 + bj + 3) for bj in range(2)]] for e in range(E_loc)], np.float32)
    sd = np.array([[[2.0 ** -(e * 8 + bi + 5)] for bi in range(2)] for e in range(E_loc)], np.float32)
    shc = [mk((1, f, d)), mk((1, f, d)), mk((1, d, f))]
    shs = [np.array([[[0.5, 0.25]]], np.float32), np.array([[[0.125, 0.0625]]], np.float32),
           np.array([[[3.0], [5.0]]], np.float32)]
    w = SimpleNamespace(w_gate=torch.from_numpy(cg), w_up=torch.from_numpy(cu), w_down=torch.from_numpy(cd),
                        s_gate=torch.from_numpy(sg), s_up=torch.from_numpy(su), s_down=torch.from_numpy(sd),
                        sh_gate=shc[0], sh_up=shc[1], sh_down=shc[2],
                        sh_s_gate=shs[0], sh_s_up=shs[1], sh_s_down=shs[2])
    ow = oracle.OracleWeights(w, "fp8")
    vals = bf_e4m3_table()
    for e in range(E_loc):
        g, u, dn = ow.expert(e)
        assert g.shape == (f, d) and dn.shape == (d, f)
        for (i, j) in [(0, 0), (5, 130), (127, 255), (64, 127)]:
            assert g[i, j] == vals[cg[e, i, j]] * 2.0 ** -(e * 8 + j // 128 + 1)
            assert u[i, j] == vals[cu[e, i, j]] * 2.0 ** -(e * 8 + j // 128 + 3)
            assert dn[j, i] == vals[cd[e, j, i]] * 2.0 ** -(e * 8 + j // 128 + 5)
    g, u, dn = ow.shared()
    assert g[3, 200] == vals[shc[0][0, 3, 200]] * 0.25 and u[3, 7] == vals[shc[1][0, 3, 7]] * 0.125
    assert dn[200, 3] == vals[shc[2][0, 200, 3]] * 5.0 and dn[7, 3] == vals[shc[2][0, 7, 3]] * 3.0
