"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only, no GPU needed).

* libnuna's host side (nuna_api.cpp, nap_planner.cpp) is compiled with g++
  -fsanitize=address,undefined against a stand-in for the HIP runtime and the
  kernel launchers (tests/c/hip_host_stub.cpp), and driven through its C ABI by
  tests/c/sanitize_driver.cpp: argument checks, tunables, the all-to-all
  layout builder with upload, dispatch and combine, the placement planner and
  mirrors, the dispatch-map check.  The launch stubs read the device tables
  the host built end to end, so a table shorter than its launch believes is a
  reported out-of-bounds read.
* The plain-C oracle is compiled with the same sanitizers and its pins run
  against that build in a child process that preloads the ASan runtime.

Any sanitizer report ends the child with a non-zero status.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_00867_amd", "csrc")
OUT = os.path.join(ROOT, "_build", "asan")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:halt_on_error=1",
           UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")


def _have_gxx():
    try:
        subprocess.run(["g++", "--version"], capture_output=True, check=True)
        return os.path.exists("/opt/rocm/include/hip/hip_runtime_api.h")
    except (OSError, subprocess.CalledProcessError):
        return False


pytestmark = pytest.mark.skipif(not _have_gxx(), reason="needs g++ and the HIP headers")


def test_host_library_is_clean_under_sanitizers():
    os.makedirs(OUT, exist_ok=True)
    exe = os.path.join(OUT, "sanitize_driver")
    cmd = ["g++", "-std=c++17", *SAN, "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
           "-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
           os.path.join(CSRC, "nuna_api.cpp"), os.path.join(CSRC, "nap_planner.cpp"),
           os.path.join(ROOT, "tests", "c", "hip_host_stub.cpp"), os.path.join(ROOT, "tests", "c", "sanitize_driver.cpp"),
           "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    r = subprocess.run([exe], env=ENV, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-6000:]
    assert "0 failed expectations, 0 failed launch checks" in r.stdout, r.stdout


def test_oracle_pins_hold_under_sanitizers():
    from oracle import build as obuild
    os.makedirs(OUT, exist_ok=True)
    lib = obuild.build(os.path.join(OUT, "liboracle_san.so"), extra_flags=SAN)
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    ubsan = subprocess.run(["gcc", "-print-file-name=libubsan.so"], capture_output=True, text=True).stdout.strip()
    code = (
        "import sys; sys.path[:0] = [%r, %r]\n"
        "import oracle, oracle_pins\n"
        "orc = oracle.Oracle(%r)\n"
        "for pin in oracle_pins.ALL_PINS:\n"
        "    pin(orc)\n"
        "print('pins passed:', len(oracle_pins.ALL_PINS))\n" % (ROOT, os.path.join(ROOT, "tests"), lib))
    env = dict(ENV, LD_PRELOAD=f"{asan}:{ubsan}", ASAN_OPTIONS="detect_leaks=0:halt_on_error=1")
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True, timeout=900)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-6000:]
    assert "pins passed" in r.stdout
