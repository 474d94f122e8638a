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


def test_native_program_is_built():
    assert os.path.isfile(EXE) and os.access(EXE, os.X_OK), "tests/native/snap_native is built by build()"


@pytest.mark.gpu
def test_native_compress_and_decode():
    r = subprocess.run([EXE], capture_output=True, text=True, timeout=100)
    print(r.stdout, r.stderr, flush=True)
    assert r.returncode == 0 and "NATIVE OK" in r.stdout, (r.returncode, r.stdout, r.stderr)
