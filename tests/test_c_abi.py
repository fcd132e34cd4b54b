"""The C ABI from C: include/lg.h compiled as C99 by gcc, liblg.so linked from a C program that
checks the defaults, the sizes and the host-side argument checks of every entry point (CPU only:
every call is rejected before anything is enqueued)."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
PKG = os.path.join(ROOT, "paper_2604_10044_amd")
ROCM_INCLUDE = "/opt/rocm/include"


@pytest.mark.skipif(shutil.which("gcc") is None or not os.path.isdir(ROCM_INCLUDE),
                    reason="gcc or the HIP headers not available")
def test_c_caller(tmp_path):
    assert os.path.exists(os.path.join(PKG, "liblg.so")), "build the library first"
    exe = str(tmp_path / "c_abi")
    # the HIP runtime header needs the platform macro when it is not compiled by hipcc
    build = subprocess.run(
        ["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror=implicit-function-declaration",
         "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"), "-I", ROCM_INCLUDE,
         os.path.join(HERE, "c_abi_driver.c"), "-L", PKG, "-llg", "-Wl,-rpath," + PKG, "-o", exe],
        capture_output=True, text=True, timeout=120)
    assert build.returncode == 0, build.stderr[-3000:]
    run = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert run.returncode == 0, run.stdout + run.stderr
    assert run.stdout.strip().endswith("ok")
