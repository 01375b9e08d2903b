"""Builds libsbw.so in-tree with hipcc for gfx950, and libsbw_rate.so, the Philox
throughput probe that only the benchmark loads (not part of the ABI)."""
from __future__ import annotations

import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIBRARY = os.path.join(PKG, "libsbw.so")
SOURCES = [os.path.join(CSRC, "sbw_kernels.hip")]
RATE_LIBRARY = os.path.join(PKG, "libsbw_rate.so")
RATE_SOURCES = [os.path.join(CSRC, "philox_rate.hip")]
HEADERS = [os.path.join(CSRC, "sbw_device.hpp"), os.path.join(INCLUDE, "sbw.h")]

HIPCC_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    # bit-exact arithmetic: no FMA contraction, no fast-math, fp32 denormals kept,
    # IEEE-rounded fp32 divide (the sampler's logarithm divides once)
    "-ffp-contract=off",
    "-fno-fast-math",
    "-fno-gpu-flush-denormals-to-zero",
    "-fhip-fp32-correctly-rounded-divide-sqrt",
    # packed fp32 VALU ops stay off
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    return "hipcc"


def build(extra_flags: list[str] | None = None, output: str = LIBRARY,
          sources: list[str] | None = None) -> str:
    cmd = [hipcc(), *HIPCC_FLAGS, *(extra_flags or []), "-I", INCLUDE, "-I", CSRC,
           *(sources or SOURCES), "-o", output + ".tmp"]
    subprocess.run(cmd, check=True)
    os.replace(output + ".tmp", output)
    return output


def build_rate() -> str:
    """The benchmark's Philox throughput probe, in a library of its own."""
    return build(output=RATE_LIBRARY, sources=RATE_SOURCES)


if __name__ == "__main__":
    print(build())
    print(build_rate())
