"""Build tests/native/snap_native (test infrastructure): a C++ program that
drives the library through its C ABI with the HIP runtime alone and checks it
against the C oracle.  Host code only (g++), linked to libsnapstream.so,
liboracle.so and the system HIP runtime."""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
PKG = os.path.join(ROOT, "paper_2511_03092_amd")
ORACLE = os.path.join(ROOT, "oracle")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
EXE = os.path.join(HERE, "snap_native")


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
    return EXE


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
