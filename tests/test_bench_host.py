"""Host logic of bench.py (no GPU): which runs time the other workloads, how a
failing child run is reported, and the device-code hashes that decide
whether the recorded counter figures still describe the built library."""
import json
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def _args(*argv):
    old = sys.argv
    sys.argv = ["bench.py", *argv]
    try:
        return bench.parse()
    finally:
        sys.argv = old


@pytest.mark.parametrize("argv,want", [
    ((), True),
    (("--gpus", "1", "--steps", "3", "--warmup", "1"), True),
    (("--no-cpu-baseline",), True),
    (("--no-others",), False),
    (("--workload", "llama8b-32layer-b8-128k"), False),
    (("--prefill",), False),
    (("--layers", "2"), False),
    (("--decode-steps", "0"), False),
    (("--copy-calibration", "1024"), False),
])
def test_other_workloads_only_on_the_default_run(argv, want):
    assert bench.wants_others(_args(*argv)) is want


def test_other_runs_name_known_workloads():
    import synth
    for extra in bench.OTHER_RUNS:
        if "--workload" in extra:
            assert extra[extra.index("--workload") + 1] in synth.WORKLOADS


def test_failing_child_run_is_reported(monkeypatch):
    monkeypatch.setattr(bench, "OTHER_RUNS", [["--workload", "no-such-workload"]])
    recs = bench.run_others(timeout_s=120)
    assert len(recs) == 1
    r = recs[0]
    assert r["args"] == "--workload no-such-workload"
    assert r["error"].startswith("exit status") and "value" not in r
    assert "no-such-workload" in r["stderr_tail"]
    json.dumps(recs)  # the record goes into the JSON line as it is


def test_compress_streams_default():
    assert _args().compress_streams is None and bench.DEFAULT_COMPRESS_STREAMS >= 1
    assert _args("--compress-streams", "1").compress_streams == 1


def test_recorded_counter_figures_match_the_built_library():
    lib = os.path.join(ROOT, "paper_2511_03092_amd", "libsnapstream.so")
    if not os.path.exists(lib):
        pytest.skip("library not built")
    for name in ("traffic", "mfma"):
        recs = json.load(open(os.path.join(ROOT, "profiles", f"{name}.json")))
        for wl, rec in recs.items():
            h = bench.device_code_sha256(lib, rec["kernels"])
            assert h is not None, (name, wl, "no kernel matches")
            assert h == rec["device_code_sha256"], (name, wl, "kernels changed since the counters were taken")
