"""The oracle's C dispatch under AddressSanitizer and UndefinedBehaviorSanitizer.

`oracle/dispatch.c` is compiled with gcc together with a small driver
(`tests/sanitize_dispatch_main.c`) that sizes every buffer exactly, with
`-fsanitize=address,undefined -fno-sanitize-recover=all`, so an out-of-bounds
access, a leak or undefined behaviour ends the run with an error.  Each case's
outputs are compared bit for bit with the pure-Python brute force (the
definition: a stable sort by (expert id, slot)).  CPU only.
"""
import os
import shutil
import struct
import subprocess

import numpy as np
import pytest

from brute_force import bf_dispatch

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)

pytestmark = pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    exe = str(tmp_path_factory.mktemp("san") / "dispatch_san")
    cmd = ["gcc", "-O1", "-g", "-std=c11", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           os.path.join(ROOT, "oracle", "dispatch.c"), os.path.join(HERE, "sanitize_dispatch_main.c"),
           "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0 and "sanitize" in r.stderr:
        pytest.skip("sanitizer runtime not available: " + r.stderr[-300:])
    assert r.returncode == 0, r.stderr
    return exe


def _run(exe, ids, E, e0, E_loc):
    ids = np.asarray(ids, np.int32).reshape(len(ids), -1) if len(ids) else np.zeros((0, 1), np.int32)
    T, k = ids.shape
    data = struct.pack("<5i", T, k, E, e0, E_loc) + ids.astype("<i4").tobytes()
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:exitcode=86",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([exe], input=data, capture_output=True, env=env)
    assert r.returncode == 0, "sanitizer or driver error %d:\n%s" % (r.returncode,
                                                                      r.stderr.decode()[-3000:])
    out = np.frombuffer(r.stdout, "<i4")
    n_loc, n_bad = int(out[0]), int(out[1])
    p = 2
    counts = out[p:p + E]; p += E
    offsets = out[p:p + E_loc + 1]; p += E_loc + 1
    slot_of_row = out[p:p + n_loc]; p += n_loc
    row_of_slot = out[p:p + T * k]; p += T * k
    assert p == out.size
    return ids, n_loc, n_bad, counts, offsets, slot_of_row, row_of_slot


def _check(exe, ids, E, e0, E_loc):
    ids, n_loc, n_bad, counts, offsets, sor, ros = _run(exe, ids, E, e0, E_loc)
    bc, bo, border, bros = bf_dispatch(ids.tolist(), E, e0, E_loc)
    assert counts.tolist() == bc
    assert offsets.tolist() == bo
    assert sor.tolist() == border
    assert ros.tolist() == bros
    assert n_loc == len(border)
    assert n_bad == int(np.count_nonzero((ids < -1) | (ids >= E)))


@pytest.mark.parametrize("seed", range(6))
def test_random_routing_under_sanitizers(driver, seed):
    rng = np.random.default_rng(seed)
    T = int(rng.integers(1, 300))
    k = int(rng.integers(1, 9))
    E = int(rng.integers(k, 64))
    e0 = int(rng.integers(0, E))
    E_loc = int(rng.integers(1, E - e0 + 1))
    ids = rng.integers(-1, E, size=(T, k))      # duplicates within a token allowed
    _check(driver, ids, E, e0, E_loc)


@pytest.mark.parametrize("name", ["empty", "all_masked", "all_local_one_expert", "invalid_ids",
                                  "every_expert_local", "last_expert_only"])
def test_edge_cases_under_sanitizers(driver, name):
    E, e0, E_loc = 16, 4, 8
    if name == "empty":
        ids = np.zeros((0, 2), np.int32)
    elif name == "all_masked":
        ids = np.full((37, 3), -1)
    elif name == "all_local_one_expert":
        ids = np.full((50, 4), 7)
    elif name == "invalid_ids":
        ids = np.array([[16, -2, 5], [4, 100, -1], [-7, 11, 12]])
    elif name == "every_expert_local":
        E, e0, E_loc = 8, 0, 8
        ids = np.arange(80).reshape(20, 4) % 8
    else:
        ids = np.full((9, 2), 11)                # e0 + E_loc - 1
    _check(driver, ids, E, e0, E_loc)
