"""Build the native test programs (test infrastructure):
* tests/native/snap_native: a C++ program that drives the library through its
  C ABI with the HIP runtime alone and checks it against the C oracle.  Host
  code only (g++), linked to libsnapstream.so, liboracle.so and the system
  HIP runtime.
* tests/native/fp8_cvt_check: a HIP program (hipcc, gfx950, the library's
  compile flags) that checks the library header's hardware E4M3 conversion
  against its software encoder on every fp32 bit pattern."""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
PKG = os.path.join(ROOT, "paper_2511_03092_amd")
ORACLE = os.path.join(ROOT, "oracle")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
EXE = os.path.join(HERE, "snap_native")
CVT_EXE = os.path.join(HERE, "fp8_cvt_check")
HIPCC = os.path.join(ROCM, "bin", "hipcc")


def build(verbose: bool = False) -> str:
    cmd = ["g++", "-std=c++17", "-O1", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"),
           os.path.join(HERE, "snap_native.cpp"), "-o", EXE + ".tmp",
           "-L", PKG, "-lsnapstream", "-L", ORACLE, "-loracle", "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
           "-Wl,-rpath," + ":".join(["$ORIGIN/../../paper_2511_03092_amd", "$ORIGIN/../../oracle",
                                     os.path.join(ROCM, "lib")])]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(EXE + ".tmp", EXE)
    cvt = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature", "-Xclang",
           "-packed-fp32-ops", "-fno-honor-nans", "-mno-amdgpu-ieee", "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(PKG, "csrc"), os.path.join(HERE, "fp8_cvt_check.hip"), "-o", CVT_EXE + ".tmp"]
    if verbose:
        print(" ".join(cvt), flush=True)
    subprocess.run(cvt, check=True)
    os.replace(CVT_EXE + ".tmp", CVT_EXE)
    return EXE


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
