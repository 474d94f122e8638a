"""Build libsnapstream.so (HIP, gfx950) in-tree, next to this file.

    python -m paper_2511_03092_amd.build [-v] [--debug]
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libsnapstream.so")
DEBUG_LIB = os.path.join(HERE, "libsnapstream_debug.so")
SOURCES = ["abi.hip", "compress.hip", "decode.hip", "prefill.hip", "noalloc.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def build(verbose: bool = False, debug: bool = False) -> str:
    """Build the library; debug=True builds libsnapstream_debug.so with the
    device-side invariant checks (SNAP_DEBUG_CHECKS) instead."""
    lib = DEBUG_LIB if debug else LIB
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
           # packed fp32 VALU ops stay off: plain fp32 math everywhere
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           # MFMA results in VGPRs: no per-element accumulator moves
           "-mllvm", "-amdgpu-mfma-vgpr-form=1",
           # IEEE mode off: no NaN reaches a min/max (masked lanes hold -inf),
           # so max needs no operand canonicalisation
           "-fno-honor-nans", "-mno-amdgpu-ieee",
           "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC]
    if debug:
        cmd += ["-DSNAP_DEBUG_CHECKS"]
    cmd += [os.path.join(CSRC, s) for s in SOURCES]
    cmd += ["-o", lib + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(lib + ".tmp", lib)
    return lib


if __name__ == "__main__":
    build(verbose="-v" in sys.argv, debug="--debug" in sys.argv)
