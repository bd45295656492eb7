"""The C ABI used from plain C: tests/c/abi_host.c is compiled as C11 against include/trivance.h,
linked with libtrivance.so and run (host-only calls, no GPU needed)."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2602_17254_amd")


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not found")
def test_c_program_uses_the_abi(tmp_path):
    lib = os.path.join(PKG, "libtrivance.so")
    if not os.path.exists(lib):
        pytest.skip("libtrivance.so is not built")
    exe = str(tmp_path / "abi_host")
    subprocess.run(["gcc", "-std=c11", "-Wall", "-Wextra", "-Werror", "-pedantic",
                    "-I", os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "c", "abi_host.c"),
                    "-L", PKG, "-ltrivance", "-Wl,-rpath," + PKG, "-o", exe], check=True)
    res = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "abi_host ok" in res.stdout
