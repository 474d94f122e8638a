"""snap_decode_step_noalloc (the decode step without a workspace argument,
for callers that cannot allocate) against snap_decode_step with a caller
workspace: two calls in a row on each path, the second with fewer sequences,
must give identical outputs and cache bytes (the same kernels run; only where
the split-K partials live differs), and the outputs match the fp64 oracle on
the GPU's cache.  The scratch array keeps what the first call left in it
when the second runs.

Every case prints what names it before touching the GPU.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2511_03092_amd as snap
import synth
from snaphelp import TOL, GpuCache, gpu_compress, oracle_params, params_of, raw

pytestmark = pytest.mark.gpu

GQA = synth.Workload("noalloc-gqa", 16, 8, 2, 128, 128, False, 4, 16, 300, 32, 7, "bf16", "bf16", layers=1,
                     batch=3, length=None, length_range=(700, 3000), decode_steps=2, rope=True, plant_frac=0.01)
CASES = {
    "gqa-bf16": (GQA, torch.bfloat16),
    "gqa-fp8": (synth.small(GQA, kv_dtype="fp8"), torch.bfloat16),
    "latent-bf16": (synth.small(synth.WORKLOADS["mla-8head-61layer-b16-128k"], recent=64, topk=1000),
                    torch.bfloat16),
    "tiny-fp32": (synth.small(synth.WORKLOADS["tiny-fp32"], name="noalloc-fp32"), torch.float32),
}


def _clone(c: GpuCache) -> GpuCache:
    d = GpuCache.__new__(GpuCache)
    d.p, d.n_slots = c.p, c.n_slots
    d.k = c.k.clone()
    d.v = None if c.v is None else c.v.clone()
    d.k_scale = None if c.k_scale is None else c.k_scale.clone()
    d.v_scale = None if c.v_scale is None else c.v_scale.clone()
    d.pos, d.n_topk = c.pos.clone(), c.n_topk.clone()
    return d


@pytest.mark.parametrize("name", list(CASES))
def test_noalloc_step_matches_workspace_step(name):
    wl, out_dtype = CASES[name]
    p = params_of(wl)
    lengths = [2900, 1300, 777] if wl.length is None else [wl.length, wl.length - 100, wl.length - 300]
    n_slots = 3
    print(f"\n[case] noalloc {name}: lengths {lengths}, calls with 3 then 2 sequences", flush=True)
    q, k, v = synth.prefill_batch(wl, 0, lengths)
    a = GpuCache(p, n_slots)
    if a.k_scale is not None:
        a.k_scale.fill_(0.05)
        if a.v_scale is not None:
            a.v_scale.fill_(0.05)
    gpu_compress(p, a, q, k, v, lengths, [0, 1, 2], debug=False)
    b = _clone(a)
    op = oracle_params(p)
    for call, slots in enumerate(([2, 0, 1], [1, 2])):
        sl = torch.tensor(slots, dtype=torch.int32, device="cuda")
        n = len(slots)
        ws = snap.workspace(snap.snap_decode_workspace(p, n))
        out_a = torch.zeros((n, p.n_q_heads, p.d_v), dtype=out_dtype, device="cuda")
        out_b = torch.zeros_like(out_a)
        positions = a.pos[sl.long()].cpu().tolist()
        qd, kn, vn = synth.decode_inputs(wl, 0, call, positions, device="cuda")
        snap.snap_decode_step(p, a.c(), a.pos, a.n_topk, sl, qd, kn, vn, out_a, ws)
        snap.snap_decode_step_noalloc(p, b.c(), b.pos, b.n_topk, sl, qd, kn, vn, out_b)
        torch.cuda.synchronize()
        assert torch.equal(raw(out_a), raw(out_b)), call
        assert torch.equal(raw(a.k), raw(b.k)), call
        if a.v is not None:
            assert torch.equal(raw(a.v), raw(b.v)), call
        assert torch.equal(a.pos, b.pos)
        ck, cv = b.host_values()
        nt = b.n_topk.cpu().numpy()
        exp = oracle.decode_attn(op, positions, nt[slots], qd.cpu(), ck[slots], None if cv is None else cv[slots])
        err = float(np.max(np.abs(out_b.double().cpu().numpy() - exp)))
        print(f"  call {call} ({n} sequences): identical to the workspace path; max abs err vs oracle {err:.3e}",
              flush=True)
        assert err <= TOL[wl.kv_dtype]
        snap.snap_advance(a.pos, sl)
        snap.snap_advance(b.pos, sl)
        torch.cuda.synchronize()
