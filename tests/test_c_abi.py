"""The boundary from a plain C caller: tests/c_abi/gmc_from_c.c (C11, the
HIP runtime's C API for device memory, include/gmc.h) compiles with gcc and
links against libgmc.so on the CPU; on the GPU it runs three GMC iterations
and checks message sizes, ascending in-range indices, the exact top-s
property against the residual and the residual's zeros."""
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "c_abi", "gmc_from_c.c")
PKG = os.path.join(ROOT, "paper_1905_12948_amd")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def _build(out: str):
    if not os.path.exists(os.path.join(PKG, "libgmc.so")):
        pytest.skip("libgmc.so is not built")
    if shutil.which("gcc") is None or not os.path.exists(os.path.join(ROCM, "include", "hip", "hip_runtime_api.h")):
        pytest.skip("gcc or the HIP headers are missing")
    cmd = ["gcc", "-std=c11", "-Wall", "-Wextra", "-Werror", "-O1", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"), SRC, "-o", out,
           "-L", PKG, "-lgmc", "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
           "-Wl,-rpath," + PKG, "-Wl,-rpath," + os.path.join(ROCM, "lib"), "-lm"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def test_c_caller_compiles_and_links():
    with tempfile.TemporaryDirectory() as tmp:
        _build(os.path.join(tmp, "gmc_from_c"))


@pytest.mark.gpu
def test_c_caller_runs():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    with tempfile.TemporaryDirectory() as tmp:
        exe = os.path.join(tmp, "gmc_from_c")
        _build(exe)
        print("running the C caller", flush=True)
        r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
        assert r.returncode == 0, r.stdout + r.stderr
        assert "every check holds" in r.stdout
