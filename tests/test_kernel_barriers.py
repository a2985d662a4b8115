"""Every workgroup barrier of every kernel is reached with no LDS store of the
wave still outstanding.

A barrier orders LDS only if each wave's stores have completed when it
arrives (an s_waitcnt lgkmcnt(0) since its last LDS store): on gfx950 a store
still in flight can be read stale by a wave on another SIMD after the barrier
opens.  The kernels are compiled to gfx950 assembly here (the same flags as
the library) and each function's control-flow graph, loop back edges
included, is searched for a path from an LDS store to an s_barrier with no
such wait between them."""
import os
import re
import shutil
import subprocess
import tempfile
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_07001_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

WAIT0 = re.compile(r"^s_waitcnt\b.*lgkmcnt\(0\)")
LDS_STORE = re.compile(r"^ds_(write|store|add|sub|or|and|xor|max|min|inc|dec|cmpst|wrxchg|append|consume)")
LABEL = re.compile(r"^(\.LBB\d+_\d+):")
ANON = re.compile(r"^; %bb\.\d+:")
BRANCH = re.compile(r"^s_(c?branch\w*)\s+(\.LBB\d+_\d+)")


def functions(asm: str):
    """(name, instruction lines) of each kernel in an assembly listing."""
    name, body = None, []
    for raw in asm.split("\n"):
        line = raw.strip()
        m = re.match(r"^(_Z\w+):", raw)
        if m:
            name, body = m.group(1), []
            continue
        if name is None:
            continue
        if raw.startswith(".Lfunc_end"):
            yield name, body
            name = None
            continue
        body.append(line)


def stale_barriers(body):
    """Labels of the blocks holding an s_barrier that some path reaches with an
    LDS store of the wave not yet waited for."""
    blocks = [[None, []]]
    for line in body:
        m = LABEL.match(line)
        if m or ANON.match(line):
            blocks.append([m.group(1) if m else None, []])
        else:
            blocks[-1][1].append(line)
    index = {lab: i for i, (lab, _) in enumerate(blocks) if lab}
    succ = []
    for i, (_, lines) in enumerate(blocks):
        out, ends = [], False
        for line in lines:
            m = BRANCH.match(line)
            if m and m.group(2) in index:
                out.append(index[m.group(2)])
                ends |= m.group(1) == "branch"
            if line.startswith("s_endpgm") or line.startswith("s_setpc"):
                ends = True
        if not ends and i + 1 < len(blocks):
            out.append(i + 1)
        succ.append(out)
    pending_in = [False] * len(blocks)
    stale = set()
    changed = True
    while changed:
        changed = False
        for i, (lab, lines) in enumerate(blocks):
            pending = pending_in[i]
            for line in lines:
                if WAIT0.match(line):
                    pending = False
                elif LDS_STORE.match(line):
                    pending = True
                elif line.startswith("s_barrier") and pending:
                    stale.add(lab or f"block {i}")
            for t in succ[i]:
                if pending and not pending_in[t]:
                    pending_in[t] = True
                    changed = True
    return sorted(stale)


def test_checker_sees_a_store_carried_over_a_back_edge():
    # an LDS store at the end of a loop, the barrier at its top: flagged; with
    # the wait in front of the barrier: clean
    loop = [".LBB0_1:", "s_barrier", "ds_read_b32 v1, v2", "s_waitcnt lgkmcnt(0)",
            "ds_write_b32 v2, v1", "s_cbranch_scc1 .LBB0_1", "s_endpgm"]
    assert stale_barriers(loop) == [".LBB0_1"]
    fixed = [".LBB0_1:", "s_waitcnt lgkmcnt(0)", "s_barrier", "ds_read_b32 v1, v2", "s_waitcnt lgkmcnt(0)",
             "ds_write_b32 v2, v1", "s_cbranch_scc1 .LBB0_1", "s_endpgm"]
    assert stale_barriers(fixed) == []


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
def test_no_barrier_is_reached_with_an_lds_store_in_flight():
    sources = sorted(f for f in os.listdir(CSRC) if f.endswith(".hip"))
    tmp = tempfile.mkdtemp(prefix="gkv_asm_")
    flags = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature", "-Xclang",
             "-packed-fp32-ops", "-Wno-unused-result", "--cuda-device-only", "-S",
             "-I", os.path.join(ROOT, "include"), "-I", CSRC]

    def compile_one(src):
        out = os.path.join(tmp, src.replace(".hip", ".s"))
        r = subprocess.run([HIPCC] + flags + [os.path.join(CSRC, src), "-o", out], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-2000:]
        return src, open(out).read()

    try:
        with ThreadPoolExecutor(min(8, len(sources))) as ex:
            listings = list(ex.map(compile_one, sources))
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
    bad, kernels = [], 0
    for src, asm in listings:
        for name, body in functions(asm):
            kernels += 1
            stale = stale_barriers(body)
            if stale:
                bad.append((src, name, stale[:4]))
    assert kernels > 30
    assert not bad, bad
