"""Split-K decode of small batches (Sec. III-C: attention over the compressed
cache, split into chunks merged by log-sum-exp).  A call with few (sequence,
KV head) units is split into chunks as short as one 32-row block, up to 128
per unit; merge_chunks merges calls of 33 to 128 chunks per unit (more than
the combine kernel keeps in registers) as well as those of at most 16, and
the combine those of 17 to 32.  The host test pins the chunk counts of the
benchmark shapes, from the workspace size (which holds the partials of every
chunk); the GPU tests run compress and decode steps of calls with 33 to 128
chunks against the oracle, for both value widths (64, 128) and the latent
512, both output dtypes, bf16, fp32 and fp8 caches, chunks left empty by
short prompts and a slot id the call must skip.  (Calls of at most 16 chunks
run through merge_chunks in the rest of the GPU suite.)
"""
import pytest
import torch

import paper_2511_03092_amd as snap
import synth
from snaphelp import NEAR_RTOL, TOL, params_of, run_case


def _align(x):
    return (x + 255) // 256 * 256


def n_chunks_of(p, n):
    """The chunk count behind snap_decode_workspace(p, n): partials
    [n][Hq][chunks][d_v] fp32, then (m, l) pairs [n][Hq][chunks]."""
    ws = snap.snap_decode_workspace(p, n)
    found = [c for c in range(1, 513)
             if _align(n * p.n_q_heads * c * p.d_v * 4) + _align(n * p.n_q_heads * c * 8) == ws]
    assert len(found) == 1, (ws, found)
    return found[0]


@pytest.mark.parametrize("workload,n,want", [
    ("llama8b-1layer-32k", 1, 128),         # 8 units: 32-row chunks of the 4096-row budget
    ("llama8b-32layer-b8-128k", 8, 32),     # 64 units: 2048 / 64 chunks, the combine
    ("cb-fp8-llama8b-32slot", 31, 8),       # 248 units
    ("mla-8head-61layer-b16-128k", 16, 16),  # latent: one 4-wave workgroup per CU in all
    ("mla-8head-61layer-b16-128k", 1, 128),  # latent chunks hold at least 256 rows
])
def test_chunk_counts(workload, n, want):
    p = params_of(synth.WORKLOADS[workload])
    assert n_chunks_of(p, n) == want


def _wl(name, cfg, d, kv, sink, recent, topk, batch):
    return synth.Workload(name, cfg, 8, 2, d, d, False, sink, recent, topk, 8, 7, "bf16" if kv != "f32" else "f32",
                          kv, layers=1, batch=batch, length=None, length_range=(1, 9000), decode_steps=8, rope=True,
                          plant_frac=0.01)


# (name, d, cache dtype, sink, recent, topk, lengths, slots, n_slots, output dtype, expected chunks)
CASES = [
    ("d128-33", 128, "bf16", 4, 28, 1024, [3000, 500], [1, 0], 2, torch.bfloat16, 33),
    ("d128-128", 128, "bf16", 4, 92, 4000, [9000], [0], 1, torch.float32, 128),
    ("d64-128", 64, "bf16", 4, 996, 5000, [7000], [0], 1, torch.bfloat16, 128),
    ("d64-fp8-63", 64, "fp8", 4, 60, 1936, [2500, 40], [0, 5], 2, torch.float32, 63),
    ("d128-f32-64", 128, "f32", 4, 60, 1984, [2600], [0], 1, torch.float32, 64),
]


# Latent caches (576-wide rows, values = the first 512 dims) keep chunks of at
# least 256 rows; one or two sequences with a budget above 32 such chunks are
# merged by merge_chunks in four 128-dim slices.
LATENT_CASES = [
    ("latent-bf16-36", "bf16", [9500], [0], 1, torch.bfloat16, 36),
    ("latent-fp8-36", "fp8", [9400, 3000], [1, 0], 2, torch.float32, 36),
]


@pytest.mark.gpu
@pytest.mark.parametrize("case", LATENT_CASES, ids=[c[0] for c in LATENT_CASES])
def test_many_chunk_latent_decode(case):
    name, kv, lengths, slots, n_slots, out_dtype, want = case
    wl = synth.small(synth.WORKLOADS["mla-8head-61layer-b16-128k"], sink=4, recent=60, topk=9000, kv_dtype=kv,
                     batch=len(lengths))
    p = params_of(wl, fp8_scales=snap.SNAP_FP8_SCALES_AMAX) if kv == "fp8" else params_of(wl)
    assert n_chunks_of(p, len(lengths)) == want
    print(f"\n[case] merge {name}: latent, cache {kv}, budget 4+60+9000, lengths {lengths} -> slots {slots} "
          f"of {n_slots}, {want} chunks", flush=True)
    run_case(wl, p, lengths, slots, n_slots, 6, out_dtype, TOL[kv], near_rtol=NEAR_RTOL, fused="alt")


@pytest.mark.gpu
@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_many_chunk_decode(case):
    name, d, kv, sink, recent, topk, lengths, slots, n_slots, out_dtype, want = case
    wl = _wl(f"merge-{name}", 700 + CASES.index(case), d, kv, sink, recent, topk, len(lengths))
    # fp8 scales from the kept rows (snap_compress sets them), so that a
    # skipped slot id needs no scale of its own
    p = params_of(wl, fp8_scales=snap.SNAP_FP8_SCALES_AMAX) if kv == "fp8" else params_of(wl)
    assert n_chunks_of(p, len(lengths)) == want
    print(f"\n[case] merge {name}: d {d}, cache {kv}, budget {sink}+{recent}+{topk}, lengths {lengths} "
          f"-> slots {slots} of {n_slots}, {want} chunks", flush=True)
    run_case(wl, p, lengths, slots, n_slots, 8, out_dtype, TOL[kv], near_rtol=NEAR_RTOL, fused="alt")
