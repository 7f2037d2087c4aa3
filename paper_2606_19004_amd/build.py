"""Build libditstep.so (the gfx950 HIP kernels + C ABI) in-tree with hipcc.

    python -m paper_2606_19004_amd.build        # or build() from Python

Each .hip (and host-only .cpp) under csrc/ compiles to an object under _build/ (in parallel), then
the objects link into paper_2606_19004_amd/libditstep.so. The same objects with api.hip compiled under
DITSTEP_DEBUG link into libditstep_debug.so: every launch synchronised and checked, and every operand
range of the block path's GEMM, attention and LayerNorm launches checked against the buffers the
entry point knows.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OBJ = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libditstep.so")
LIB_DEBUG = os.path.join(HERE, "libditstep_debug.so")
ARCH = "gfx950"

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-fPIC", "-std=c++17",
    # keep the compiler from emitting packed fp32 (v_pk_*_f32) instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
    "-Wno-unused-result",
]


HOST_FLAGS = ["-x", "c++", "-O2", "-fPIC", "-std=c++17", "-Wall", "-I", os.path.join(ROOT, "include")]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libditstep.so)")


def _run(cmd):
    p = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    # the host pass does not know the packed-fp32 feature and says so; that line is noise
    out = "\n".join(l for l in p.stdout.splitlines() if "packed-fp32-ops" not in l)
    return p.returncode, out


def build(verbose: bool = False, jobs: int = 4) -> str:
    os.makedirs(OBJ, exist_ok=True)
    cc = hipcc()
    # .hip: kernels and their host code; .cpp: host-only code (planner, seed bank), plain C++
    srcs = sorted(f for f in os.listdir(CSRC) if f.endswith((".hip", ".cpp")))
    objs = [os.path.join(OBJ, f.rsplit(".", 1)[0] + ".o") for f in srcs]
    cmds = [[cc, *(HIPCC_FLAGS if f.endswith(".hip") else HOST_FLAGS), "-c", os.path.join(CSRC, f), "-o", o]
            for f, o in zip(srcs, objs)]
    api_debug = os.path.join(OBJ, "api_debug.o")
    cmds.append([cc, *HIPCC_FLAGS, "-DDITSTEP_DEBUG", "-c", os.path.join(CSRC, "api.hip"), "-o", api_debug])
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        results = list(ex.map(_run, cmds))
    for cmd, (rc, out) in zip(cmds, results):
        if verbose and out.strip():
            print(out)
        if rc != 0:
            raise RuntimeError(f"hipcc failed ({rc}) for {cmd[-3]}:\n{out}")
    debug_objs = [api_debug if os.path.basename(o) == "api.o" else o for o in objs]
    for lib, lib_objs in ((LIB, objs), (LIB_DEBUG, debug_objs)):
        tmp = lib + ".tmp"
        rc, out = _run([cc, "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp, *lib_objs])
        if rc != 0:
            raise RuntimeError(f"link failed:\n{out}")
        os.replace(tmp, lib)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
