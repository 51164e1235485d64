"""The C ABI from plain C: tests/c/abi_consumer.c compiles as C99 against include/nuna.h with
warnings as errors, links libnuna.so and gets the documented status of every call it makes (host
checks, tunables, planner, placement mirror; nothing it calls launches a kernel)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIBDIR = os.path.join(ROOT, "paper_2608_00867_amd")


@pytest.mark.skipif(shutil.which("gcc") is None, reason="no C compiler")
def test_c99_consumer(tmp_path):
    if not os.path.exists(os.path.join(LIBDIR, "libnuna.so")):
        pytest.skip("library not built")
    exe = str(tmp_path / "abi_consumer")
    # HIP's own headers need the platform macro from compilers other than hipcc.
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include",
           os.path.join(ROOT, "tests", "c", "abi_consumer.c"), "-L", LIBDIR, "-lnuna",
           "-Wl,-rpath," + LIBDIR, "-o", exe]
    build = subprocess.run(cmd, capture_output=True, text=True)
    assert build.returncode == 0, build.stderr[-3000:]
    run = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert run.returncode == 0 and run.stdout.strip().endswith("ok"), run.stdout + run.stderr
