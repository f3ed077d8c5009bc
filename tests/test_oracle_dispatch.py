"""Pins for the oracle's counting-sort dispatch (CPU only): numpy's bincount,
Python's stable sort and the bijection invariants."""
import numpy as np
import pytest

import oracle
from brute_force import bf_dispatch
from paper_2606_22541_amd import inputs


def _check(ids, E, e0, E_loc):
    T, k = ids.shape
    got = oracle.dispatch(ids, E, e0, E_loc)
    flat = ids.ravel()
    valid = flat[(flat >= 0) & (flat < E)]
    assert np.array_equal(got["counts"], np.bincount(valid, minlength=E))
    local = [s for s in range(T * k) if e0 <= flat[s] < e0 + E_loc]
    order = sorted(local, key=lambda s: (int(flat[s]), s))
    assert got["slot_of_row"].tolist() == order
    assert got["n_loc"] == len(order)
    ros = got["row_of_slot"]
    assert np.all(ros[got["slot_of_row"]] == np.arange(len(order)))       # inverse
    assert np.sum(ros >= 0) == len(order)                                  # bijection
    offs = got["offsets"]
    assert offs[0] == 0 and np.all(np.diff(offs) >= 0) and offs[-1] == len(order)
    for i in range(E_loc):
        seg = flat[got["slot_of_row"][offs[i]:offs[i + 1]]]
        assert np.all(seg == e0 + i)
    bc, bo, bs, br = bf_dispatch(ids.tolist(), E, e0, E_loc)
    assert got["counts"].tolist() == bc and got["offsets"].tolist() == bo
    assert got["slot_of_row"].tolist() == bs and got["row_of_slot"].tolist() == br
    return got


@pytest.mark.parametrize("seed", range(5))
def test_dispatch_random_tiny(seed):
    rng = np.random.default_rng(seed)
    T, k, E = int(rng.integers(1, 40)), int(rng.integers(1, 5)), int(rng.integers(2, 12))
    ids = rng.integers(-1, E, size=(T, k)).astype(np.int32)      # duplicates and masks allowed
    e0 = int(rng.integers(0, E))
    E_loc = int(rng.integers(1, E - e0 + 1))
    _check(ids, E, e0, E_loc)


def test_dispatch_c0_sum_invariant():
    cfg = inputs.CONFIGS["c0"]
    mb = inputs.make_microbatches(cfg)[0]
    got = _check(mb.ids, cfg.E, cfg.e0, cfg.E_loc)
    assert got["counts"].sum() == mb.ids.size                    # sum counts = T*k


def test_dispatch_c1_shape_sum_invariant():
    cfg = inputs.CONFIGS["c1"]
    rng = np.random.default_rng(0)
    ids, w = inputs.draw_routing(cfg, 4096, rng, np.random.default_rng(1), None)
    got = oracle.dispatch(ids, cfg.E, cfg.e0, cfg.E_loc)
    assert got["counts"].sum() == 4096 * 8
    assert np.array_equal(got["counts"], np.bincount(ids.ravel(), minlength=256))
    srt = np.sort(ids, axis=1)
    assert np.all(srt[:, 1:] != srt[:, :-1])                       # k distinct experts
    ros = got["row_of_slot"]
    assert np.array_equal(np.sort(ros[ros >= 0]), np.arange(got["n_loc"]))


def test_dispatch_edge_cases():
    E, e0, E_loc = 8, 0, 4
    # T = 0
    got = oracle.dispatch(np.zeros((0, 2), np.int32), E, e0, E_loc)
    assert got["n_loc"] == 0 and got["counts"].sum() == 0 and got["offsets"].tolist() == [0] * 5
    # all slots masked
    got = _check(np.full((5, 2), -1, np.int32), E, e0, E_loc)
    assert got["n_loc"] == 0
    # all slots to one expert, duplicates within a token count twice
    got = _check(np.full((6, 3), 2, np.int32), E, e0, E_loc)
    assert got["counts"][2] == 18 and got["offsets"].tolist() == [0, 0, 0, 18, 18]
    # E_loc = 1 with a non-zero first local expert
    _check(np.array([[5, 1], [5, 5], [0, 7]], np.int32), E, 5, 1)
    # invalid ids are skipped and counted
    got = oracle.dispatch(np.array([[0, 9], [-5, 1]], np.int32), E, e0, E_loc)
    assert got["n_bad"] == 2 and got["n_loc"] == 2 and got["row_of_slot"].tolist() == [0, -1, -1, 1]


def test_zipf_routing_properties():
    cfg = inputs.CONFIGS["c2"]
    mbs = inputs.make_microbatches(inputs.scaled(cfg, d=128, f=128))
    assert len(mbs) == 4
    for mb in mbs:
        T = mb.ids.shape[0]
        assert 16 <= T <= 8192
        cnt = np.bincount(mb.ids.ravel(), minlength=256)[:8]
        assert cnt[6] == 0 and cnt[7] == 0
        assert cnt.max() > 4 * cnt.mean()
        # k distinct experts per token, weights sorted and normalised
        s = np.sort(mb.ids, axis=1)
        assert np.all(s[:, 1:] != s[:, :-1])
        assert np.all(np.diff(mb.w, axis=1) <= 0)
        assert np.allclose(mb.w.sum(axis=1), 1.0, atol=1e-6)
