"""Pins for the oracle's e4m3 codec and the per-128 quantiser (CPU only)."""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_decode_matches_ocp_points():
    pts = json.load(open(os.path.join(GOLDEN, "e4m3_points.json")))["points"]
    for p in pts:
        v = oracle.e4m3_decode(np.array([p["code"]], np.uint8))[0]
        if p["value"] == "nan":
            assert math.isnan(v), p
        else:
            assert v == p["value"] and math.copysign(1, v) == math.copysign(1, p["value"]), p


def test_decode_all_codes_match_torch():
    codes = torch.arange(256, dtype=torch.int32).to(torch.uint8)
    ref = codes.view(torch.float8_e4m3fn).to(torch.float64).numpy()
    mine = oracle.e4m3_decode(np.arange(256, dtype=np.uint8))
    nan = np.isnan(ref)
    assert np.array_equal(nan, np.isnan(mine))
    assert np.array_equal(ref[~nan], mine[~nan])
    assert np.sum(nan) == 2                       # 0x7F and 0xFF only: no infinities


def _brute_nearest(v):
    """Nearest finite e4m3 value, ties to the even code, saturating."""
    vals = [(c, oracle.E4M3_TABLE[c]) for c in range(256) if not math.isnan(oracle.E4M3_TABLE[c])]
    best = None
    for c, x in vals:
        dist = abs(float(v) - x)
        key = (dist, c & 1)
        # keep the sign of v for zeros
        if x == 0 and (math.copysign(1, x) != math.copysign(1, float(v))):
            continue
        if best is None or key < best[0]:
            best = (key, c)
    c = best[1]
    if abs(float(v)) > 448:
        c = 0x7E | (0x80 if v < 0 else 0)
    return c


def test_encode_brute_force_random_and_midpoints():
    rng = np.random.default_rng(1)
    v = np.concatenate([
        rng.standard_normal(300) * 100,
        rng.standard_normal(200) * 0.01,
        np.array([0.0, -0.0, 448.0, -448.0, 455.0, 464.0, 1000.0, -1e30, 2.0 ** -10, 2.0 ** -11]),
    ]).astype(np.float32)
    # exact midpoints between neighbouring positive codes exercise ties-to-even
    pos = oracle.E4M3_TABLE[:0x7F]
    mids = ((pos[:-1] + pos[1:]) / 2).astype(np.float32)
    v = np.concatenate([v, mids, -mids])
    got = oracle.e4m3_encode(v)
    want = np.array([_brute_nearest(x) for x in v], np.uint8)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, [(float(v[i]), int(got[i]), int(want[i])) for i in bad[:10]]


def test_encode_matches_torch_cast_in_range():
    rng = np.random.default_rng(2)
    v = (rng.standard_normal(20000) * 60).astype(np.float32)
    v = np.clip(v, -448, 448)
    ref = torch.from_numpy(v).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(oracle.e4m3_encode(v), ref)


def test_quantize_groups_properties():
    rng = np.random.default_rng(3)
    x = (rng.standard_normal((7, 384)) * np.array([1e-3, 1.0, 300.0]).repeat(128)[None, :]).astype(np.float32)
    x[2, 128:256] = 0.0                       # an all-zero group
    codes, scales = oracle.quantize_groups(x)
    assert codes.shape == x.shape and scales.shape == (7, 3)
    g = x.reshape(7, 3, 128)
    amax = np.abs(g).max(axis=2)
    for r in range(7):
        for b in range(3):
            if amax[r, b] == 0:
                assert scales[r, b] == np.float32(1.0)
                assert np.all(codes[r, b * 128:(b + 1) * 128] & 0x7F == 0)
                continue
            assert scales[r, b] == np.float32(amax[r, b]) / np.float32(448.0)
            i = int(np.argmax(np.abs(g[r, b])))
            c = codes[r, b * 128 + i]
            assert c & 0x7F == 0x7E                  # the amax element maps to +-448
    # dequantised values are within half a step of e4m3 at their magnitude
    deq = oracle.dequantize_groups(codes, scales)
    step = np.ldexp(1.0, np.maximum(np.frexp(np.abs(x / scales.repeat(128, axis=1)))[1] - 1, -6) - 3)
    err = np.abs(deq - x) / scales.repeat(128, axis=1).astype(np.float64)
    assert np.all(err <= step / 2 * (1 + 1e-6) + 1e-30)


def test_quantize_matches_elementwise_definition():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((3, 256)).astype(np.float32)
    codes, scales = oracle.quantize_groups(x)
    for r in range(3):
        for c in range(256):
            s = scales[r, c // 128]
            q = np.float32(x[r, c]) / s                 # fp32 division
            assert codes[r, c] == _brute_nearest(np.float32(q))


def test_bf16_widening_matches_torch_all_patterns():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    mine = oracle.bf16_bits_to_f64(bits)
    nan = np.isnan(ref)
    assert np.array_equal(nan, np.isnan(mine))
    assert np.array_equal(ref[~nan], mine[~nan])


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(5)
    v = (rng.standard_normal(100000) * 10.0 ** rng.integers(-6, 6, 100000)).astype(np.float32)
    # exact ties between two neighbouring bf16 values, both parities of the kept bits
    ties = ((np.arange(0, 4096, dtype=np.uint32) << 16) | 0x8000).view(np.float32)
    v = np.concatenate([v, ties[np.isfinite(ties)]])
    ref = torch.from_numpy(v).to(torch.bfloat16).to(torch.float32).numpy()
    got = oracle.round_f32_to_bf16(v)
    assert np.array_equal(ref.view(np.uint32), got.view(np.uint32))
