"""Build ``libnuna.so`` (gfx950 HIP kernels + C ABI) in-tree with hipcc.

Each source compiles to its own object in parallel (under ``_build/`` at the
repository root), then hipcc links the shared library.  Every call compiles
every source again: the build is also the "does it compile" check.
"""
import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libnuna.so")
OBJDIR = os.path.join(ROOT, "_build", "libnuna")

SOURCES = [os.path.join(CSRC, f) for f in ("nuna_allreduce.hip", "nuna_rs_ag.hip", "nuna_moe.hip", "nuna_routed.hip",
                                           "nuna_probe.hip", "nap_planner.cpp", "nuna_api.cpp")]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "-O3", "-std=c++17", "-fPIC",
    "--offload-arch=gfx950",
    # keep the compiler from forming packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # no contraction and no fast-math: every fp32 add stays a single IEEE add
    "-ffp-contract=off", "-fno-fast-math",
    "-Wall", "-Wno-unused-command-line-argument",
    "-I" + INCLUDE, "-I" + CSRC,
]


def build(out=LIB, extra=()):
    os.makedirs(OBJDIR, exist_ok=True)
    procs = []
    objs = []
    for src in SOURCES:
        obj = os.path.join(OBJDIR, os.path.basename(src) + ".o")
        objs.append(obj)
        cmd = [HIPCC, *FLAGS, *extra, "-c", src, "-o", obj]
        procs.append((cmd, subprocess.Popen(cmd)))
    failed = [cmd for cmd, p in procs if p.wait() != 0]
    if failed:
        raise subprocess.CalledProcessError(1, failed[0])
    tmp = out + ".tmp"
    subprocess.run([HIPCC, "-shared", "-fPIC", "--offload-arch=gfx950", *objs, "-o", tmp], check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build())
