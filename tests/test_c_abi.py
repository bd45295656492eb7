"""The C ABI used from plain C: tests/c/abi_host.c is compiled as C11 against include/trivance.h,
linked with libtrivance.so and run (host-only calls, no GPU needed); tests/c/dispatch_split.cpp
and tests/c/fastdiv.cpp check the launch split and the invariant division with g++."""

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


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not found")
def test_dispatch_split_covers_every_workgroup(tmp_path):
    """tests/c/dispatch_split.cpp: the launch split keeps every dispatch within the work-item limit
    and covers each workgroup exactly once, also for grids above 2^32 work-items (host only)."""
    exe = str(tmp_path / "dispatch_split")
    csrc = os.path.join(PKG, "csrc")
    subprocess.run(["g++", "-std=c++17", "-O1", "-Wall", "-Wextra", "-Werror", "-I", csrc,
                    "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "c", "dispatch_split.cpp"),
                    os.path.join(csrc, "plan.cpp"), "-o", exe], check=True)
    res = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "dispatch_split ok" in res.stdout


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not found")
def test_invariant_division_is_exact(tmp_path):
    """tests/c/fastdiv.cpp: the 32-bit multiply-high division of the tree-step decode equals the
    hardware division for every divisor up to 2^16 at the extreme dividends and for 8 million
    seeded random (dividend < 2^31, divisor) pairs (host only)."""
    exe = str(tmp_path / "fastdiv")
    csrc = os.path.join(PKG, "csrc")
    subprocess.run(["g++", "-std=c++17", "-O2", "-Wall", "-Wextra", "-Werror", "-I", csrc,
                    "-I", os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "c", "fastdiv.cpp"),
                    "-o", exe], check=True)
    res = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "fastdiv ok" in res.stdout


@pytest.mark.gpu
@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not found")
def test_c_program_runs_allreduces_on_the_gpu(tmp_path):
    """tests/c/abi_gpu.c: int32 AllReduces (ring, torus, ring of 8) and congestion from plain C,
    with the HIP runtime API for device memory; exact sums and 3^k loads are checked in C."""
    lib = os.path.join(PKG, "libtrivance.so")
    if not os.path.exists(lib):
        pytest.fail("libtrivance.so is not built")
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    exe = str(tmp_path / "abi_gpu")
    subprocess.run(["gcc", "-std=c11", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
                    "-I", os.path.join(rocm, "include"), "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "c", "abi_gpu.c"),
                    "-L", PKG, "-ltrivance", "-L", os.path.join(rocm, "lib"), "-lamdhip64",
                    "-Wl,-rpath," + PKG, "-Wl,-rpath," + os.path.join(rocm, "lib"), "-o", exe],
                   check=True)
    print("[c-abi] running the C program on the GPU", flush=True)
    res = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "abi_gpu ok" in res.stdout
