"""The library driven from C++ through its C ABI alone (no Python, no torch in
the process): tests/native/snap_native.cpp compresses a seeded 1500-token
prompt of one GQA layer (8 query / 2 KV heads, d = 128, bf16 cache, sink 4,
ring 64, K 200) and runs 80 decode steps, checking the kept set and cache
bytes against the fp64 oracle's compression (Sec. III-B) and every step's
output against the oracle's decode attention (Sec. III-C)."""
import os
import subprocess

import pytest

EXE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "native", "snap_native")
CVT_EXE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "native", "fp8_cvt_check")


def test_native_program_is_built():
    assert os.path.isfile(EXE) and os.access(EXE, os.X_OK), "tests/native/snap_native is built by build()"
    assert os.path.isfile(CVT_EXE) and os.access(CVT_EXE, os.X_OK), "tests/native/fp8_cvt_check is built by build()"


@pytest.mark.gpu
def test_native_compress_and_decode():
    r = subprocess.run([EXE], capture_output=True, text=True, timeout=100)
    print(r.stdout, r.stderr, flush=True)
    assert r.returncode == 0 and "NATIVE OK" in r.stdout, (r.returncode, r.stdout, r.stderr)


@pytest.mark.gpu
def test_fp8_conversion_instruction_matches_encoder():
    """The fp8 cache gather quantises with the conversion instruction
    (e4m3x4_hw): its codes must equal the software encoder's, which the
    oracle's E4M3 rounding pins, for every fp32 input."""
    r = subprocess.run([CVT_EXE], capture_output=True, text=True, timeout=100)
    print(r.stdout, r.stderr, flush=True)
    assert r.returncode == 0 and "2^32 patterns x 4 positions: 0" in r.stdout, (r.returncode, r.stdout, r.stderr)
