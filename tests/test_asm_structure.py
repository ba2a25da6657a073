"""Structure of the compiled work loops (gfx950 assembly built on the CPU, no GPU).

A persistent kernel claims its next work item with `if (tid == 0) item = atomicAdd(...)`
followed by a workgroup barrier. If the compiler threads that lane-divergent test through a
loop back edge, the barrier ends up in an inner loop that lane 0 of wave 0 has left; the
hardware barrier counts waves, so the other lanes pass it without the claim and the loop
never ends. This test fails if the first barrier after any claim lies in a different loop
than the claim itself."""
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_25852_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

LABEL = re.compile(r"^(\.LBB\d+_\d+):|^; %bb\.(\d+):")
HEADER = re.compile(r"=>\s*This (?:Inner )?Loop Header: Depth=(\d+)")
IN_LOOP = re.compile(r"in Loop: Header=(BB\d+_\d+) Depth=(\d+)")


def _assemble(src, tmp_path):
    out = tmp_path / (os.path.splitext(src)[0] + ".s")
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "--cuda-device-only", "-S",
           "-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", os.path.join(CSRC, src), "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    return out.read_text().split("\n")


def _functions(lines):
    """(name, body lines) of every kernel in an assembly listing."""
    out, name, body = [], None, []
    for l in lines:
        m = re.match(r"^(_Z\S+):", l)
        if m:
            name, body = m.group(1), []
            continue
        if name and l.startswith(".Lfunc_end"):
            out.append((name, body))
            name = None
            continue
        if name:
            body.append(l)
    return out


def _loop_of_each_line(body):
    """innermost loop header of the block holding each line (None outside loops); a block's
    loop annotation is on its label line or on the comment lines right after it"""
    res, cur_loop = [], None
    for n, l in enumerate(body):
        m = LABEL.match(l)
        if m:
            blk = m.group(1)[2:] if m.group(1) else None  # ".LBB2_5" -> "BB2_5"
            notes = [l]
            k = n + 1
            while k < len(body) and body[k].lstrip().startswith(";"):
                notes.append(body[k])
                k += 1
            note = " ".join(notes)
            h = HEADER.search(note)
            il = IN_LOOP.search(note)
            if h and blk:
                cur_loop = blk
            elif il:
                cur_loop = il.group(1)
            else:
                cur_loop = None
        res.append(cur_loop)
    return res


def claims_and_barriers(lines, kernel_pattern):
    """[(kernel, loop of the claim, loop of the next barrier)] for every global atomic add
    that is followed by a barrier"""
    found = []
    for name, body in _functions(lines):
        if not re.search(kernel_pattern, name):
            continue
        loops = _loop_of_each_line(body)
        for i, l in enumerate(body):
            if "global_atomic_add" not in l:
                continue
            j = next((k for k in range(i + 1, len(body)) if "s_barrier" in body[k]), None)
            if j is not None:
                found.append((name, loops[i], loops[j]))
    return found


def test_attention_claim_and_barrier_share_a_loop(tmp_path):
    lines = _assemble("attn.hip", tmp_path)
    found = claims_and_barriers(lines, r"attn_bf16_kernel")
    assert len(found) >= 4, found  # one claim per instantiated persistent kernel
    for name, claim_loop, barrier_loop in found:
        assert claim_loop is not None and claim_loop == barrier_loop, (name, claim_loop, barrier_loop)


def test_checker_flags_a_threaded_claim():
    """The checker on a hand-written listing with the miscompiled shape: the claim in the
    outer loop, its barrier in an inner loop entered from the unit's latch."""
    listing = """_ZN2sv6kernelEv:
.LBB2_129:                              ;   in Loop: Header=BB2_130 Depth=1
\ts_cbranch_execz .LBB2_485
.LBB2_130:                              ; =>This Loop Header: Depth=1
\ts_and_saveexec_b64 s[0:1], s[42:43]
; %bb.132:                              ;   in Loop: Header=BB2_130 Depth=1
\tglobal_atomic_add v3, v73, v3, s[94:95] sc0
.LBB2_134:                              ;   in Loop: Header=BB2_130 Depth=1
\ts_branch .LBB2_137
.LBB2_137:                              ;   Parent Loop BB2_130 Depth=1
                                        ; =>  This Loop Header: Depth=2
\ts_barrier
.Lfunc_end0:
"""
    lines = listing.split("\n")
    found = claims_and_barriers(lines, r"kernel")
    assert found == [("_ZN2sv6kernelEv", "BB2_130", "BB2_137")]
