"""Properties of the generated gfx950 code, checked on the CPU (hipcc
cross-compiles; no GPU is needed):

* no scalar-cache stores or atomics anywhere in device code (every store
  goes through the vector memory path);
* no packed fp32 VALU operations (the build disables them);
* no waterfall loops (a buffer descriptor or address the compiler could not
  prove wave-uniform, re-established lane by lane around every load);
* no scratch (spill) accesses inside the innermost MFMA loop of any GEMM
  kernel.
"""
import os
import re
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

from paper_2606_22541_amd import build

SOURCES = sorted(os.path.basename(s) for s in build.sources())
GEMMS = ("gemm_bf16.hip", "gemm_bf16_small.hip", "gemm_fp8.hip")


def _asm(src):
    cmd = [build.HIPCC] + [f for f in build.flags_for(src) if f != "-fPIC"] + [
        "-S", "--offload-device-only", os.path.join(build.CSRC, src), "-o", "-"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    return r.stdout


@pytest.fixture(scope="module")
def asm():
    with ThreadPoolExecutor(max_workers=4) as ex:
        return dict(zip(SOURCES, ex.map(_asm, SOURCES)))


def _kernels(text):
    """{kernel symbol: [instruction or label lines]}"""
    out = {}
    for m in re.finditer(r"^(_Z\w+):", text, re.M):
        end = text.find(".Lfunc_end", m.end())
        lines = []
        for l in text[m.end():end].split("\n"):
            l = l.strip()
            if not l or l.startswith(";") or (l.startswith(".") and not l.startswith(".LBB")):
                continue
            lines.append(l.split(";")[0].strip())
        out[m.group(1)] = lines
    return out


def _backward_loops(lines):
    """(start, end) line ranges of loops closed by a backward branch."""
    labels = {l[:-1]: i for i, l in enumerate(lines) if l.startswith(".LBB") and l.endswith(":")}
    loops = []
    for i, l in enumerate(lines):
        m = re.match(r"s_cbranch_\w+\s+(\.LBB\w+)|s_branch\s+(\.LBB\w+)", l)
        if m:
            t = labels.get(m.group(1) or m.group(2))
            if t is not None and t < i:
                loops.append((t, i))
    return loops


@pytest.mark.parametrize("src", SOURCES)
def test_no_scalar_stores_or_packed_fp32(asm, src):
    bad = re.findall(r"^\s*(s_store\w*|s_atomic\w*|s_buffer_store\w*|s_buffer_atomic\w*|"
                     r"s_dcache_wb\w*|s_scratch_store\w*|v_pk_(?:fma|mul|add)_f32)\b",
                     asm[src], re.M)
    assert not bad, "%s: %s" % (src, sorted(set(bad)))


def _is_waterfall(body):
    """A waterfall loop is short: read one lane's operand into SGPRs, mask the
    lanes that hold the same value, do the operation, retire those lanes and
    branch back while any remain.  (Longer backward ranges are ordinary loops
    or out-of-line blocks that jump back into the kernel.)"""
    return (len(body) <= 64 and
            any(l.startswith("v_readfirstlane") for l in body) and
            any(l.startswith("s_and_saveexec") for l in body) and
            any(re.match(r"s_(xor|andn2)_b64\s+exec, exec", l) for l in body) and
            body[-1].startswith("s_cbranch_execnz"))


def test_waterfall_detector_matches_the_compiler_pattern():
    body = ["v_readfirstlane_b32 s4, v0", "v_readfirstlane_b32 s5, v1",
            "v_cmp_eq_u64_e32 vcc, s[4:5], v[0:1]", "s_and_saveexec_b64 s[6:7], vcc",
            "buffer_load_dword v2, v3, s[8:11], 0 offen", "s_xor_b64 exec, exec, s[6:7]",
            "s_cbranch_execnz .LBB0_1"]
    assert _is_waterfall(body)
    assert not _is_waterfall(body[:-1] + ["s_cbranch_scc1 .LBB0_1"])
    assert not _is_waterfall(body[:3] + ["s_nop 0"] * 80 + body[3:])


@pytest.mark.parametrize("src", SOURCES)
def test_no_waterfall_loops(asm, src):
    for name, lines in _kernels(asm[src]).items():
        for a, b in _backward_loops(lines):
            assert not _is_waterfall(lines[a:b + 1]), \
                "%s: waterfall loop in %s at line %d" % (src, name, a)


@pytest.mark.parametrize("src", GEMMS)
def test_no_spills_in_mfma_loops(asm, src):
    checked = 0
    for name, lines in _kernels(asm[src]).items():
        loops = [(a, b) for a, b in _backward_loops(lines)
                 if any("mfma" in l for l in lines[a:b + 1])]
        if not loops:
            continue
        a, b = min(loops, key=lambda ab: ab[1] - ab[0])     # innermost MFMA loop
        spills = [l for l in lines[a:b + 1] if l.startswith("scratch_") or "buffer_store" in l
                  and "scratch" in l]
        assert not spills, "%s: %d scratch accesses in the MFMA loop of %s" % (src, len(spills), name)
        checked += 1
    assert checked > 0, "no MFMA loop found in " + src
