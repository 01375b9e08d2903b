"""Independent Philox engines for the oracle pins (test-only).

Builds two small host libraries from open-source headers -- PyTorch's ATen
`PhiloxRNGEngine.h` and rocRAND's `rocrand_philox4x32_10.h` -- that return the
v-th 32-bit output of the Philox4x32-10 stream keyed by r.  Neither shares code
with the oracle or the HIP library.
"""
import ctypes
import os
import shutil
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))


def build(out_dir) -> dict:
    import torch
    libs = {}
    tinc = os.path.join(os.path.dirname(torch.__file__), "include")
    aten = os.path.join(str(out_dir), "libaten_x.so")
    subprocess.run(["g++", "-O2", "-std=c++17", "-fPIC", "-shared", "-I", tinc, "-o", aten,
                    os.path.join(HERE, "xcheck", "aten_philox.cpp")], check=True)
    libs["aten"] = (ctypes.CDLL(aten), "aten_stream_word")
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if os.path.exists(hipcc):
        roc = os.path.join(str(out_dir), "librocrand_x.so")
        subprocess.run([hipcc, "-x", "hip", "--offload-host-only", "-O2", "-std=c++17", "-fPIC",
                        "-shared", "-o", roc, os.path.join(HERE, "xcheck", "rocrand_philox.cpp")],
                       check=True)
        libs["rocrand"] = (ctypes.CDLL(roc), "rocrand_stream_word")
    return libs


def engine_words(libs, name, v, r) -> np.ndarray:
    lib, fn = libs[name]
    v = np.ascontiguousarray(v, dtype=np.uint32)
    r = np.ascontiguousarray(r, dtype=np.uint64)
    out = np.empty(v.shape, np.uint32)
    getattr(lib, fn)(ctypes.c_void_p(v.ctypes.data), ctypes.c_void_p(r.ctypes.data),
                     ctypes.c_int64(v.size), ctypes.c_void_p(out.ctypes.data))
    return out
