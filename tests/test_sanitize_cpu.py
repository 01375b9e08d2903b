"""The host code under AddressSanitizer and UndefinedBehaviorSanitizer, on the CPU.

1. The C oracle, every entry point on edge shapes (tests/capi/oracle_edges.c): a
   vocabulary of one token, rows not a multiple of 32 long, padded rows, texts of 0-2
   tokens, windows of 8, lengths below 0 and beyond L, candidate ids -1, V and
   2^31 - 1, empty arrays; every buffer at its exact size.
2. libsbw's host side (argument checks, dispatch, the C ABI) built with the sanitizers
   on the host pass only (hipcc -Xarch_host), driven by the plain C client's checks
   that return before any HIP call, unknown enum values included.
Both must finish with no sanitizer report.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE = os.path.join(ROOT, "oracle", "sbw_oracle.c")
EDGES = os.path.join(ROOT, "tests", "capi", "oracle_edges.c")
CAPI = os.path.join(ROOT, "tests", "capi", "capi_check.c")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
SANITIZE = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
REPORTS = ("runtime error", "AddressSanitizer", "LeakSanitizer", "UndefinedBehaviorSanitizer")


def _clean(r):
    text = r.stdout + r.stderr
    return r.returncode == 0 and not any(s in text for s in REPORTS), text[-4000:]


def test_oracle_edge_shapes_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_edges")
    subprocess.run(["gcc", "-std=c11", "-O1", "-g", "-Wall", "-Wextra", "-Werror",
                    "-ffp-contract=off", *SANITIZE, EDGES, ORACLE, "-o", exe, "-lm"],
                   check=True, capture_output=True, text=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    ok, text = _clean(r)
    assert ok, text
    assert "oracle edges ok" in r.stdout


@pytest.mark.skipif(not os.path.exists(os.path.join(ROCM, "bin", "hipcc")), reason="no hipcc")
def test_library_host_code_under_sanitizers(tmp_path):
    sys_path = os.path.join(ROOT, "paper_2609_03844_amd")
    import importlib.util
    spec = importlib.util.spec_from_file_location("sbw_build_helper",
                                                  os.path.join(sys_path, "_build.py"))
    helper = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(helper)
    libdir = tmp_path / "lib"
    libdir.mkdir()
    # the same build as libsbw.so, with the sanitizers on the host pass only
    host_only = []
    for flag in ("-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=all"):
        host_only += ["-Xarch_host", flag]
    helper.build(extra_flags=["-g", *host_only], output=str(libdir / "libsbw.so"))
    clang = os.path.join(ROCM, "llvm", "bin", "clang")
    if not os.path.exists(clang):
        clang = shutil.which("clang")
    exe = str(tmp_path / "capi_check")
    subprocess.run([clang, "-std=c11", "-O1", "-g", "-ffp-contract=off", *SANITIZE,
                    "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"), "-I",
                    os.path.join(ROCM, "include"), CAPI, ORACLE, "-o", exe, "-L", str(libdir),
                    "-lsbw", f"-Wl,-rpath,{libdir}", "-L", os.path.join(ROCM, "lib"),
                    "-lamdhip64", f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}", "-lm"],
                   check=True, capture_output=True, text=True)
    r = subprocess.run([exe, "cpu"], capture_output=True, text=True, timeout=300)
    ok, text = _clean(r)
    assert ok, text
    assert "capi cpu ok" in r.stdout
