"""Static check of the built gfx950 code: no instruction touches the
destination registers of an LDS read between the read and the wait that
guarantees its data has arrived.

The kernels issue their LDS operand reads (ds_read_b128, ds_read_b64_tr_b16)
as inline assembly and wait for them with hand-counted `s_waitcnt lgkmcnt(N)`
that take the destination registers as operands.  The compiler sees the
registers as written by the read itself, so it would be free to copy them,
or to reuse them after copying, before the wait -- and either would read or
clobber data that is still in flight, giving results that change from run to
run.  This test compiles the library's device code to assembly on the host
and walks every kernel in program order: an LDS read counts as arrived once
at least N later LDS reads were issued before an `s_waitcnt lgkmcnt(N)`
(LDS reads return in order; other operations sharing the counter only make
such a wait stricter).  CPU only."""
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "paper_2511_13198_amd", "csrc", "pdyattn.hip")

REG = re.compile(r"\b([va])(?:\[(\d+):(\d+)\]|(\d+)(?!\w))")
LDS_READ = re.compile(r"^\s*(ds_read\w*|ds_load\w*)\s+(\S+),")
WAIT = re.compile(r"^\s*s_waitcnt\b(.*)$")
LGKM = re.compile(r"lgkmcnt\((\d+)\)")


def _regs(text):
    out = set()
    for m in REG.finditer(text):
        kind = m.group(1)
        if m.group(4) is not None:
            out.add((kind, int(m.group(4))))
        else:
            out.update((kind, r) for r in range(int(m.group(2)), int(m.group(3)) + 1))
    return out


def device_asm(src=SRC, extra_flags=()):
    hipcc = "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    cmd = [hipcc, "--offload-arch=gfx950", "-O3", "-std=c++17", "--cuda-device-only", "-S",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I", os.path.join(ROOT, "include"), *extra_flags, "-o", "-", src]
    res = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert res.returncode == 0, res.stderr[-2000:]
    return res.stdout


def lds_wait_hazards(asm: str):
    """(kernel, read line, offending line) for every instruction that names a
    destination register of an LDS read still in flight; also the number of
    LDS reads checked."""
    hazards = []
    checked = 0
    kernel = None
    pending = []  # [dest regs, read line, LDS reads issued after it]
    for line in asm.splitlines():
        code = line.split(";", 1)[0].rstrip()
        if re.match(r"^_Z\w+:", code):
            kernel = code[:-1]
            pending = []
            continue
        if not code.strip() or code.strip().startswith("."):
            continue
        w = WAIT.match(code)
        if w:
            m = LGKM.search(w.group(1))
            if m:
                n = int(m.group(1))
                pending = [p for p in pending if p[2] < n]
            continue
        r = LDS_READ.match(code)
        if r:
            dest = _regs(r.group(2))
            srcs = _regs(code[r.end():])
            for p in pending:
                if p[0] & (dest | srcs):
                    hazards.append((kernel, p[1].strip(), code.strip()))
                p[2] += 1
            pending.append([dest, code, 0])
            checked += 1
            continue
        used = _regs(code)
        for p in pending:
            if p[0] & used:
                hazards.append((kernel, p[1].strip(), code.strip()))
    return hazards, checked


def test_no_use_of_lds_read_destinations_before_their_wait():
    asm = device_asm()
    hazards, checked = lds_wait_hazards(asm)
    assert checked > 500, f"only {checked} LDS reads found: is the parser still matching?"
    assert not hazards, "LDS destinations touched before their wait:\n" + "\n".join(
        f"  {k}: {a}  ...  {b}" for k, a, b in hazards[:20])


def test_checker_flags_a_planted_early_use():
    """The walk itself: a copy of an in-flight destination is reported, the
    same copy after a covering wait is not, and a wait that leaves the read
    outstanding does not clear it."""
    body = """_Z1kv:
    ds_read_b128 v[4:7], v1 offset:16
    ds_read_b64_tr_b16 v[8:9], v2
    {between}
    s_waitcnt lgkmcnt({n})
    v_mov_b32 v20, v5
"""
    bad, _ = lds_wait_hazards(body.format(between="v_mov_b32 v30, v6", n=1))
    assert len(bad) == 1 and "v30" in bad[0][2]
    ok, checked = lds_wait_hazards(body.format(between="v_add_f32 v31, v1, v2", n=1))
    assert not ok and checked == 2
    # lgkmcnt(2) leaves the first read outstanding: the use after it is reported
    late, _ = lds_wait_hazards(body.format(between="", n=2))
    assert len(late) == 1 and "v20" in late[0][2]
    # a later read overwriting an in-flight destination (WAW) is reported
    waw, _ = lds_wait_hazards("_Z1kv:\n ds_read_b128 v[4:7], v1\n ds_read_b128 v[6:9], v2\n")
    assert len(waw) == 1
