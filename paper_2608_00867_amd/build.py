"""Build ``libnuna.so`` (gfx950 HIP kernels + C ABI) in-tree with hipcc."""
import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libnuna.so")

SOURCES = [os.path.join(CSRC, "nuna_kernels.hip"), os.path.join(CSRC, "nuna_moe.hip"),
           os.path.join(CSRC, "nuna_probe.hip"), os.path.join(CSRC, "nap_planner.cpp"),
           os.path.join(CSRC, "nuna_api.cpp")]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "-shared",
    "--offload-arch=gfx950",
    # keep the compiler from forming packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # no contraction and no fast-math: every fp32 add stays a single IEEE add
    "-ffp-contract=off", "-fno-fast-math",
    "-Wall", "-Wno-unused-command-line-argument",
    "-I" + INCLUDE, "-I" + CSRC,
]


def build(out=LIB, extra=()):
    tmp = out + ".tmp"
    cmd = [HIPCC, *FLAGS, *extra, *SOURCES, "-o", tmp]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build())
