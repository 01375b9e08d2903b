"""The C ABI from a plain C program: include/sbw.h compiles as C11 with gcc, the
program links libsbw.so (and the HIP runtime for its own buffers) with no Python or
torch in the process, and its results match the C oracle bit for bit on the GPU."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "capi", "capi_check.c")
ORACLE = os.path.join(ROOT, "oracle", "sbw_oracle.c")
LIBDIR = os.path.join(ROOT, "paper_2609_03844_amd")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


@pytest.fixture(scope="module")
def capi_binary(tmp_path_factory):
    if not os.path.exists(os.path.join(LIBDIR, "libsbw.so")):
        pytest.fail("libsbw.so is not built; run __graft_entry__.build() first")
    out = str(tmp_path_factory.mktemp("capi") / "capi_check")
    cmd = ["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-Werror", "-ffp-contract=off",
           "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"), "-I",
           os.path.join(ROCM, "include"), SRC, ORACLE, "-o", out, "-L", LIBDIR, "-lsbw",
           f"-Wl,-rpath,{LIBDIR}", "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
           f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}", "-lm"]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    return out


def test_c_client_argument_checks(capi_binary):
    r = subprocess.run([capi_binary, "cpu"], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    assert "capi cpu ok" in r.stdout


@pytest.mark.gpu
def test_c_client_parity_on_the_gpu(capi_binary):
    r = subprocess.run([capi_binary, "gpu"], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "capi gpu ok" in r.stdout
