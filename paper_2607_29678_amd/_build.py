"""Compile the HIP sources into ``libtoktier.so`` (gfx950) next to this file."""

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libtoktier.so")
SOURCES = ["tt_api.hip", "tt_tile.hip", "tt_batch.hip", "tt_spans.hip", "tt_session.hip", "tt_copy.cpp", "tt_noalloc.hip"]
ARCH = "gfx950"

FLAGS = [
    "--offload-arch=" + ARCH,
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    # packed FP32 instructions are kept out of the generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


# the diagnostic build with per-tile phase stamps (phase_timeline.py)
PHASES_LIB = os.path.join(HERE, "libtoktier_phases.so")


def build(verbose: bool = False, phases: bool = False) -> str:
    """Compile every source (always) and link the shared library; returns its
    path.  ``phases``: the diagnostic build with phase stamps, into its own
    library file and object directory."""
    cc = hipcc()
    objdir = os.path.join(HERE, "_build_phases" if phases else "_build")
    lib = PHASES_LIB if phases else LIB
    defines = ["-DTT_PHASE_STAMPS"] if phases else []
    os.makedirs(objdir, exist_ok=True)

    def compile_one(src):
        obj = os.path.join(objdir, os.path.splitext(src)[0] + ".o")
        cmd = [cc] + FLAGS + defines + ["-c", os.path.join(CSRC, src), "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError("compile failed: %s\n%s%s" % (" ".join(cmd), r.stdout, r.stderr))
        if verbose:
            err = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l)
            if err.strip():
                print(err, file=sys.stderr)
        return obj

    with ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    tmp = lib + ".tmp"
    cmd = [cc, "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed: %s\n%s%s" % (" ".join(cmd), r.stdout, r.stderr))
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    print(build(verbose=True, phases="--phases" in sys.argv[1:]))
