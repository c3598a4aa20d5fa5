"""Generated code of the library's kernels (CPU: hipcc cross-compiles gfx950).

A branch on the lane ahead of a broadcast inside a loop (one lane takes a
ticket, every lane reads it) can be compiled into a loop that some lanes
re-enter without the lane that updates the state they wait on; an early
version's wave kernel compiled that way into a block that only tests exec
and a condition register and branches to itself, which never ends once
entered, and stalled the GPU on pieces longer than 512 bytes.  This test
compiles every HIP source to gfx950 assembly and fails on any block that
branches to itself while only testing state (s_and/s_cmp into vcc or scc),
so that such a loop is caught before it runs.
"""

import os
import re
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_29678_amd", "csrc")
PURE_TEST = re.compile(r"^(s_and_b64|s_or_b64|s_andn2_b64|s_cmp_\w+|s_cmpk_\w+)\s+(vcc|scc|s\[\d+:\d+\]|s\d+),?")


def _hipcc():
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    return None


def stuck_loops(asm: str):
    """Blocks that branch to themselves and contain only tests of existing
    state (no instruction that could change what the branch reads)."""
    out = []
    label, body, func = None, [], None
    for ln in asm.split("\n"):
        m = re.match(r"^(_Z\w+):", ln)
        if m:
            func = m.group(1)
        m = re.match(r"^(\.LBB\w+):", ln)
        if m:
            label, body = m.group(1), []
            continue
        s = ln.split(";")[0].strip()
        if not s or s.startswith("."):
            continue
        m = re.match(r"^s_cbranch_\w+\s+(\.LBB\w+)$", s)
        if m and m.group(1) == label:
            tests = body
            if all(PURE_TEST.match(t) and not t.startswith(("s_and_b64 exec", "s_or_b64 exec", "s_andn2_b64 exec"))
                   and (t.split()[1].rstrip(",") in ("vcc", "scc") or t.startswith("s_cmp"))
                   for t in tests):
                out.append((func, label, tests + [s]))
        body.append(s)
        if s.startswith(("s_branch", "s_cbranch", "s_setpc", "s_endpgm")):
            label, body = None, []
    return out


def test_checker_catches_the_pattern():
    asm = "_Zk:\n.LBB1_20:\n\ts_and_b64 vcc, exec, s[6:7]\n\ts_cbranch_vccz .LBB1_20\n"
    assert stuck_loops(asm) == [("_Zk", ".LBB1_20", ["s_and_b64 vcc, exec, s[6:7]", "s_cbranch_vccz .LBB1_20"])]
    # a spin that reloads what it tests is a wait, not a stuck loop
    ok = "_Zk:\n.LBB1_3:\n\ts_sleep 1\n\tglobal_load_dword v1, v[2:3], off\n\ts_waitcnt vmcnt(0)\n" \
         "\tv_cmp_eq_u32_e32 vcc, 0, v1\n\ts_cbranch_vccnz .LBB1_3\n"
    assert stuck_loops(ok) == []


@pytest.mark.timeout(600)
def test_no_stuck_loops_in_the_kernels(tmp_path):
    cc = _hipcc()
    if cc is None:
        pytest.skip("hipcc not found")
    srcs = sorted(f for f in os.listdir(CSRC) if f.endswith(".hip"))
    flags = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "--cuda-device-only", "-S",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]

    def one(src):
        out = str(tmp_path / (src + ".s"))
        r = subprocess.run([cc] + flags + [os.path.join(CSRC, src), "-o", out], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-2000:]
        with open(out) as f:
            return src, stuck_loops(f.read())

    with ThreadPoolExecutor(max_workers=min(4, len(srcs))) as ex:
        results = list(ex.map(one, srcs))
    bad = [(src, x) for src, found in results for x in found]
    assert not bad, bad
