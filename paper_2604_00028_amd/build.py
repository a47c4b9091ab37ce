"""Builds the C-ABI library libdecode_attn.so in-tree for gfx950.

    python -m paper_2604_00028_amd.build

One hipcc invocation compiles the HIP kernels and entry points
(csrc/decode_attn.hip) and the host planner (csrc/plan.cpp) into a shared
library next to this file.  A second one builds libhbm_probe.so, the plain
streaming-read kernel the benchmark measures the HBM read ceiling with
(csrc/hbm_probe.hip; not part of the decode-attention boundary).  Packed-fp32 VALU instructions are disabled for
the device code; the host pass warns that it does not know that target
feature, which is harmless.
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB_NAME = "libdecode_attn.so"
LIB_PATH = os.path.join(HERE, LIB_NAME)
SOURCES = [os.path.join(CSRC, "decode_attn.hip"), os.path.join(CSRC, "plan.cpp")]
PROBE_NAME = "libhbm_probe.so"
PROBE_PATH = os.path.join(HERE, PROBE_NAME)
PROBE_SOURCES = [os.path.join(CSRC, "hbm_probe.hip")]
ARCH = "gfx950"


def hipcc_path() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build the HIP library)")


def compile_command(out_path: str, sources=None) -> list:
    return [
        hipcc_path(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-Wall", "-Wno-unused-command-line-argument",
        "-I", INCLUDE, "-I", CSRC,
        "-o", out_path, *(SOURCES if sources is None else sources),
    ]


def _compile(path: str, sources, verbose: bool) -> None:
    tmp = path + f".tmp{os.getpid()}"
    cmd = compile_command(tmp, sources)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"hipcc failed ({res.returncode}): {' '.join(cmd)}")
    if verbose:
        sys.stderr.write(res.stderr)
    os.replace(tmp, path)


def build(verbose: bool = False) -> str:
    """Compile both libraries (always) and return the decode library's path."""
    _compile(LIB_PATH, SOURCES, verbose)
    _compile(PROBE_PATH, PROBE_SOURCES, verbose)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose=True))
