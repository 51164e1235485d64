"""The multiply-and-shift division of the routed dispatch (csrc/fastdiv.h), checked on the host against the
hardware quotient (CPU only): every divisor up to 4096 over the small and the largest numerators, then random
divisors of every magnitude, with exact multiples and their neighbours."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_00867_amd", "csrc")
OUT = os.path.join(ROOT, "_build", "fastdiv")


def _have_gxx():
    try:
        subprocess.run(["g++", "--version"], capture_output=True, check=True)
        return True
    except (OSError, subprocess.CalledProcessError):
        return False


@pytest.mark.skipif(not _have_gxx(), reason="needs g++")
def test_magic_division_equals_the_quotient():
    os.makedirs(OUT, exist_ok=True)
    exe = os.path.join(OUT, "fastdiv_check")
    subprocess.run(["g++", "-std=c++17", "-O2", "-Wall", "-Werror", "-I" + CSRC,
                    os.path.join(ROOT, "tests", "c", "fastdiv_check.cpp"), "-o", exe], check=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout[-2000:]
    assert ", 0 mismatches" in r.stdout, r.stdout
