"""The debug build (libsnapstream_debug.so: kernels test the invariants their
indexing rests on and record any that fails instead of faulting) runs a
spread of parity cases — ragged NaN-padded prompts with both normalisers and
pools, edge lengths, fp32 / bf16 / fp8 caches, a latent cache, the fused
decode step across ring wraps, the prefill attention — and must record no
failed check; every case is also held to the usual parity bars.

Every case prints what names it before touching the GPU.
"""
import pytest
import torch

import paper_2511_03092_amd as snap
import synth
from snaphelp import TOL, params_of, run_case

pytestmark = pytest.mark.gpu

MED = synth.Workload("dbg-med", 17, 8, 2, 128, 128, False, 4, 16, 300, 32, 13, "bf16", "bf16", layers=1, batch=3,
                     length=None, length_range=(700, 5100), decode_steps=24, rope=True, plant_frac=0.01)
EDGE = synth.Workload("dbg-edge", 18, 4, 2, 64, 64, False, 4, 8, 16, 16, 5, "f32", "f32", layers=1, batch=1,
                      length=None, length_range=(1, 100), decode_steps=12, rope=False, plant_count=3)


@pytest.fixture
def debug_library():
    prev = snap.use_library(snap.DEBUG_LIB_PATH)
    try:
        snap.snap_debug_checks(reset=True)
        yield
    finally:
        snap._lib = prev


def test_debug_build_records_no_failed_invariant(debug_library):
    cases = [
        ("ragged bf16, row normaliser, avg pool", synth.small(MED, norm=synth.NORM_ROW, pool=synth.POOL_AVG), {},
         [5000, 777, 3001], [2, 0, 1], 4, torch.bfloat16, "alt"),
        ("edge lengths fp32", EDGE, {}, [0, 1, 3, 9, 12, 13, 28, 29, 90], list(range(9)), 9, torch.float32, False),
        ("fp8 cache, data scales", synth.small(MED, kv_dtype="fp8"), {"fp8_scales": snap.SNAP_FP8_SCALES_AMAX},
         [4000, 1500], [1, 3], 4, torch.bfloat16, "alt"),
        ("latent 576, fused step", synth.small(synth.WORKLOADS["mla-8head-61layer-b16-128k"], recent=64, topk=512),
         {}, [5000, 2100], [0, 1], 3, torch.bfloat16, True),
    ]
    for name, wl, over, lengths, slots, n_slots, out_dtype, fused in cases:
        p = params_of(wl, **over)
        print(f"\n[case] debug build: {name}: lengths {lengths} -> slots {slots} of {n_slots}", flush=True)
        run_case(wl, p, lengths, slots, n_slots, 20, out_dtype, TOL[wl.kv_dtype], fused=fused, check_every=4)
        flags = snap.snap_debug_checks(reset=True)
        print(f"  failed-check bits: {flags:#x}", flush=True)
        assert flags == 0, name
    # the prefill attention and its fused compression
    wl = synth.small(MED, name="dbg-prefill")
    p = params_of(wl)
    lengths = [900, 333]
    print(f"\n[case] debug build: snap_prefill lengths {lengths}", flush=True)
    q, k, v = synth.prompt_batch(wl, 0, lengths, pad_value=float("nan"))
    n, ml = k.shape[0], k.shape[2]
    dev = "cuda"
    ck = torch.zeros((n, p.n_kv_heads, p.budget, p.d_qk), dtype=torch.bfloat16, device=dev)
    cv = torch.zeros_like(ck)
    pos = torch.zeros(n, dtype=torch.int32, device=dev)
    ntop = torch.zeros(n, dtype=torch.int32, device=dev)
    sl = torch.arange(n, dtype=torch.int32, device=dev)
    lens = torch.tensor(lengths, dtype=torch.int32, device=dev)
    out = torch.empty((n, p.n_q_heads, ml, p.d_v), dtype=torch.bfloat16, device=dev)
    ws = snap.workspace(snap.snap_prefill_workspace(p, n, ml))
    snap.snap_prefill(p, snap.cache_struct(ck, cv), pos, ntop, sl, lens, q.to(dev), k.to(dev), v.to(dev), out, ws)
    torch.cuda.synchronize()
    assert pos.cpu().tolist() == lengths
    flags = snap.snap_debug_checks(reset=True)
    print(f"  failed-check bits: {flags:#x}", flush=True)
    assert flags == 0
