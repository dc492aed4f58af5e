"""Build libcf.so (HIP for gfx950) in-tree with hipcc.

All device code is compiled with -ffp-contract=off (every fp64 operation is
one IEEE operation in the written order) and without packed fp32 operations.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libcf.so")
SOURCES = ["cf_abi.hip", "k_trace.hip", "k_coarse.hip", "k_select.hip", "k_reduce.hip", "k_fine.hip", "k_mc.hip", "k_enum.hip", "k_bisect.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-ffp-contract=off",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-function", "-I", os.path.join(ROOT, "include")]
# The fine kernel is one function by design: every helper is inlined so that the
# simulation state stays in registers and LDS (a call would move it to scratch).
# The gated instantiation exceeds the AMDGPU inliner's default basic-block limit.
FILE_FLAGS = {"k_fine.hip": ["-mllvm", "-amdgpu-inline-max-bb=3000"]}


def build(verbose=False, jobs=8):
    """Compile every source to an object in parallel, then link the library."""
    objdir = os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)
    procs, objs = [], []
    for s in SOURCES:
        o = os.path.join(objdir, s.replace(".hip", ".o"))
        objs.append(o)
        cmd = [HIPCC] + FLAGS + FILE_FLAGS.get(s, []) + ["-c", os.path.join(SRC, s), "-o", o]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((s, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
    failed = []
    for s, p in procs:
        out, _ = p.communicate()
        if p.returncode != 0:
            failed.append((s, out.decode(errors="replace")))
        elif verbose and out:
            print(out.decode(errors="replace"))
    if failed:
        raise RuntimeError("hipcc failed:\n" + "\n".join(f"--- {s}\n{o}" for s, o in failed))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
    print(LIB)
