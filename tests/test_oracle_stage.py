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


def test_fp8_stage_is_bf16_stage_on_dequantised_operands():
    """fp8: x and W enter through their e4m3 values times scales, and h is
    quantised per 128 channels before the down projection."""
    rng = np.random.default_rng(12)
    T, d, f, E, k = 6, 256, 128, 4, 2
    x_bits = _bf16_round(rng.standard_normal((T, d)))
    ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    w = rng.random((T, k)).astype(np.float32)
    codes = [rng.integers(0, 0x7E, size=s).astype(np.uint8) | (rng.integers(0, 2, size=s).astype(np.uint8) << 7)
             for s in ((2, f, d), (2, f, d), (2, d, f))]
    scales = [np.abs(rng.standard_normal(s)).astype(np.float32) * 1e-3 + 1e-4
              for s in ((2, f // 128, d // 128), (2, f // 128, d // 128), (2, d // 128, f // 128))]

    class Wt:
        gate, up, down = (codes[0], scales[0]), (codes[1], scales[1]), (codes[2], scales[2])

    ow = oracle.OracleWeights.__new__(oracle.OracleWeights)
    ow.dtype, ow.gate, ow.up, ow.down, ow.sh = "fp8", Wt.gate, Wt.up, Wt.down, None
    cfg = _cfg(d=d, f=f, E=E, e0=0, E_loc=2, k=k, dtype="fp8")
    res = oracle.run_stage(cfg, ow, x_bits, ids, w)
    # rebuild by hand: dequantised x, dequantised W, quantised h
    xq, xs = oracle.quantize_groups(oracle.bf16_bits_to_f32(x_bits))
    x = oracle.e4m3_decode(xq) * np.repeat(xs, 128, axis=1)
    out = np.zeros((T, d))
    for t in range(T):
        for j in range(k):
            e = ids[t, j]
            if e >= 2:
                continue
            Wg = oracle.e4m3_decode(codes[0][e]) * np.kron(scales[0][e], np.ones((128, 128)))
            Wu = oracle.e4m3_decode(codes[1][e]) * np.kron(scales[1][e], np.ones((128, 128)))
            Wd = oracle.e4m3_decode(codes[2][e]) * np.kron(scales[2][e], np.ones((128, 128)))
            g = Wg @ x[t]
            h = (g / (1 + np.exp(-g))) * (Wu @ x[t])
            hb = torch.from_numpy(h[None, :].astype(np.float32)).to(torch.bfloat16).float().numpy()
            hq, hs = oracle.quantize_groups(hb)
            hd = oracle.e4m3_decode(hq[0]) * np.repeat(hs[0], 128)
            out[t] += w[t, j] * (Wd @ hd)
    np.testing.assert_allclose(res["out"], out, rtol=1e-12, atol=1e-12)
    assert np.array_equal(res["x_codes"], xq)


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
