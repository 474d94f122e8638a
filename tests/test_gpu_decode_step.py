"""snap_decode_step (append + attend for one layer in one call) against the two
calls it replaces, snap_cache_append then snap_decode_attn: outputs and cache
bytes must be identical bit for bit at every step, and the fused outputs match
the fp64 oracle.  Cases cover the fused kernels (bf16 and fp8 GQA MFMA, bf16
latent) and the two-launch one (fp32), a prompt shorter than the sinks (new
tokens land in sink rows), the ring wrapping, and an invalid slot id.

Every case prints what names it before touching the GPU.
"""
import pytest
import torch

import paper_2511_03092_amd as snap
import synth
from snaphelp import TOL, GpuCache, decode_steps, gpu_compress, params_of

pytestmark = pytest.mark.gpu

GQA = synth.Workload("step-gqa", 12, 8, 2, 128, 128, False, 4, 16, 300, 32, 7, "bf16", "bf16", layers=1, batch=3,
                     length=None, length_range=(700, 3000), decode_steps=40, rope=True, plant_frac=0.01)


def _announce(msg):
    print(f"\n[case] {msg}", flush=True)


def _clone(cache: GpuCache) -> GpuCache:
    c2 = GpuCache.__new__(GpuCache)
    c2.p, c2.n_slots = cache.p, cache.n_slots
    c2.k = cache.k.clone()
    c2.v = None if cache.v is None else cache.v.clone()
    c2.k_scale = None if cache.k_scale is None else cache.k_scale.clone()
    c2.v_scale = None if cache.v_scale is None else cache.v_scale.clone()
    c2.pos = cache.pos.clone()
    c2.n_topk = cache.n_topk.clone()
    return c2


def _fused_vs_two_calls(wl, p, lengths, slots, n_slots, steps, out_dtype, invalid_slot=False):
    q, k, v = synth.prefill_batch(wl, 0, lengths)
    a = GpuCache(p, n_slots)
    if a.k_scale is not None:
        a.k_scale.fill_(0.05)
        if a.v_scale is not None:
            a.v_scale.fill_(0.05)
    gpu_compress(p, a, q, k, v, lengths, slots, debug=False)
    b = _clone(a)
    call_slots = list(slots) + ([-1] if invalid_slot else [])
    sl = torch.tensor(call_slots, dtype=torch.int32, device="cuda")
    n = len(call_slots)
    ws_a = snap.workspace(snap.snap_decode_workspace(p, n))
    ws_b = snap.workspace(snap.snap_decode_workspace(p, n))
    out_a = torch.zeros((n, p.n_q_heads, p.d_v), dtype=out_dtype, device="cuda")
    out_b = torch.zeros_like(out_a)
    for step in range(steps):
        positions = [int(x) for x in a.pos[sl.clamp_min(0).long()].cpu()]
        qd, kn, vn = synth.decode_inputs(wl, 0, step, positions, device="cuda")
        vn_ = None if vn is None else vn
        snap.snap_cache_append(p, a.c(), a.pos, sl, kn, vn_)
        snap.snap_decode_attn(p, a.c(), a.pos, a.n_topk, sl, qd, out_a, ws_a)
        snap.snap_advance(a.pos, sl)
        snap.snap_decode_step(p, b.c(), b.pos, b.n_topk, sl, qd, kn, vn_, out_b, ws_b)
        snap.snap_advance(b.pos, sl)
        torch.cuda.synchronize()
        nv = len(slots)  # the invalid slot's output row is never written by either path
        assert torch.equal(out_a[:nv].view(torch.int16 if out_dtype == torch.bfloat16 else torch.int32),
                           out_b[:nv].view(torch.int16 if out_dtype == torch.bfloat16 else torch.int32)), step
        assert torch.equal(a.k.view(torch.uint8), b.k.view(torch.uint8)), step
        if a.v is not None:
            assert torch.equal(a.v.view(torch.uint8), b.v.view(torch.uint8)), step
        assert torch.equal(a.pos, b.pos)
    return b


def test_step_gqa_bf16_fused_kernel():
    wl = GQA
    p = params_of(wl)
    lengths = [2900, 2, 1200]
    _announce(f"decode_step bf16 GQA (fused MFMA kernel): lengths {lengths}, ring 16 wraps, one prompt < sinks")
    b = _fused_vs_two_calls(wl, p, lengths, [2, 0, 1], 4, 40, torch.bfloat16, invalid_slot=True)
    # the fused path also matches the oracle from this state on
    err = decode_steps(p, wl, b, [2, 0, 1], 6, torch.bfloat16, TOL["bf16"], salt=7, fused=True)
    print(f"  fused decode max abs err vs oracle: {err:.3e}", flush=True)


def test_step_latent_bf16_fused_kernel():
    wl = synth.small(synth.WORKLOADS["mla-8head-61layer-b16-128k"], recent=64, topk=1000)
    p = params_of(wl)
    lengths = [3000, 3, 1500]
    _announce(f"decode_step bf16 latent (fused LDS kernel): lengths {lengths}, ring 64 wraps")
    b = _fused_vs_two_calls(wl, p, lengths, [0, 1, 2], 3, 80, torch.bfloat16, invalid_slot=True)
    err = decode_steps(p, wl, b, [0, 1, 2], 4, torch.bfloat16, TOL["bf16"], salt=7, fused=True)
    print(f"  fused decode max abs err vs oracle: {err:.3e}", flush=True)


def test_step_fp8_fused_and_fp32_two_launch_paths():
    wl = synth.small(GQA, kv_dtype="fp8")
    p = params_of(wl)
    lengths = [2000, 900, 3]
    _announce(f"decode_step fp8 GQA (fused kernel, new row quantised in LDS): lengths {lengths}, one prompt < sinks")
    _fused_vs_two_calls(wl, p, lengths, [1, 0, 2], 3, 24, torch.bfloat16, invalid_slot=True)
    wl = synth.WORKLOADS["tiny-fp32"]
    p = params_of(wl)
    _announce("decode_step fp32 tiny (generic kernel, two launches)")
    _fused_vs_two_calls(wl, p, [wl.length], [0], 1, 24, torch.float32)


@pytest.mark.parametrize("kv_reuse", [snap.SNAP_KV_AUTO, snap.SNAP_KV_STREAM])
def test_fp8_query_products(kv_reuse):
    """snap_params.fp8_qk = 1 over a GQA fp8 cache: the query is quantised per
    head and Q K^T runs on the fp8 MFMA.  Checked against the oracle attending
    with the same quantised query (oracle.fp8_scale / quantize), to the fp8
    tolerance; the deviation from the exact query is reported beside it.  The
    fused step (new row quantised in LDS) and the two-call path both run, with
    ordinary loads (the default at this size) and with streaming loads."""
    from snaphelp import fp8_query
    wl = synth.small(GQA, kv_dtype="fp8")
    p = params_of(wl, fp8_qk=1, kv_reuse=kv_reuse)
    lengths = [2000, 900, 3]
    _announce(f"fp8 query products (fp8_qk=1, kv_reuse {kv_reuse}): lengths {lengths}, fused step then two calls")
    q, k, v = synth.prefill_batch(wl, 0, lengths)
    c = GpuCache(p, 3)
    c.k_scale.fill_(0.05)
    c.v_scale.fill_(0.05)
    gpu_compress(p, c, q, k, v, lengths, [0, 1, 2], debug=False)
    stats = {}
    err = decode_steps(p, wl, c, [0, 1, 2], 6, torch.bfloat16, TOL["fp8"], salt=3, fused=True, q_oracle=fp8_query,
                       stats=stats)
    err2 = decode_steps(p, wl, c, [0, 1, 2], 3, torch.bfloat16, TOL["fp8"], salt=4, fused=False, q_oracle=fp8_query,
                        stats=stats)
    print(f"  max abs err vs oracle with the fp8 query: {max(err, err2):.3e}; "
          f"deviation from the exact query: {stats['exact_query_dev']:.3e}", flush=True)


@pytest.mark.parametrize("kind", ["gqa-bf16", "gqa-fp8", "latent-bf16", "latent-fp8"])
def test_load_hint_keeps_results(kind):
    """snap_params.kv_reuse only changes how the cache rows are loaded: the
    same decode call with ordinary (SNAP_KV_KEEP) and streaming
    (SNAP_KV_STREAM) loads gives the same bits, except the bf16 GQA kernel,
    which adds the dot products' pieces in another order under streaming
    loads (outputs then agree to a few bf16 ulps)."""
    if kind.startswith("gqa"):
        wl = synth.small(GQA, kv_dtype="fp8") if kind == "gqa-fp8" else GQA
        lengths = [2900, 40, 1200]
    else:
        wl = synth.small(synth.WORKLOADS["mla-8head-61layer-b16-128k"], recent=64, topk=1000,
                         kv_dtype="fp8" if kind == "latent-fp8" else "bf16")
        lengths = [3000, 70, 1500]
    p = params_of(wl)
    _announce(f"load hint keep vs stream: {kind}, lengths {lengths}")
    q, k, v = synth.prefill_batch(wl, 0, lengths)
    c = GpuCache(p, 3)
    if c.k_scale is not None:
        c.k_scale.fill_(0.05)
        if c.v_scale is not None:
            c.v_scale.fill_(0.05)
    gpu_compress(p, c, q, k, v, lengths, [0, 1, 2], debug=False)
    sl = torch.tensor([0, 1, 2], dtype=torch.int32, device="cuda")
    positions = [int(x) for x in c.pos.cpu()]
    qd, _, _ = synth.decode_inputs(wl, 0, 0, positions, device="cuda")
    outs = {}
    for hint in (snap.SNAP_KV_KEEP, snap.SNAP_KV_STREAM):
        ph = params_of(wl, kv_reuse=hint)
        out = torch.zeros((3, p.n_q_heads, p.d_v), dtype=torch.float32, device="cuda")
        ws = snap.workspace(snap.snap_decode_workspace(ph, 3))
        snap.snap_decode_attn(ph, c.c(), c.pos, c.n_topk, sl, qd, out, ws)
        torch.cuda.synchronize()
        outs[hint] = out
    a, b = outs[snap.SNAP_KV_KEEP], outs[snap.SNAP_KV_STREAM]
    assert torch.isfinite(a).all()
    if kind == "gqa-bf16":
        diff = float((a - b).abs().max())
        print(f"  max abs difference: {diff:.3e}", flush=True)
        assert diff <= 1e-4 * max(1.0, float(a.abs().max()))
    else:
        assert torch.equal(a.view(torch.int32), b.view(torch.int32))
