"""Decode steps captured in a HIP graph (torch.cuda.CUDAGraph over the C ABI):
per-sequence positions and n_topk are device data and the library neither
allocates nor synchronises, so one step (snap_decode_step + snap_advance) can
be captured once and replayed.  Every replay, with eager work and a
synchronisation in between, must match the same step run eagerly on a copy of
the cache, bit for bit (outputs and cache bytes).

Every case prints what names it before touching the GPU.
"""
import pytest
import torch

import paper_2511_03092_amd as snap
import synth
from snaphelp import GpuCache, gpu_compress, params_of

pytestmark = pytest.mark.gpu

GQA = synth.Workload("graph-gqa", 13, 8, 2, 128, 128, False, 4, 16, 300, 32, 7, "bf16", "bf16", layers=1, batch=3,
                     length=None, length_range=(700, 3000), decode_steps=8, rope=True, plant_frac=0.01)


def _clone(c: GpuCache) -> GpuCache:
    d = GpuCache.__new__(GpuCache)
    d.p, d.n_slots = c.p, c.n_slots
    d.k = c.k.clone()
    d.v = None if c.v is None else c.v.clone()
    d.k_scale = None if c.k_scale is None else c.k_scale.clone()
    d.v_scale = None if c.v_scale is None else c.v_scale.clone()
    d.pos, d.n_topk = c.pos.clone(), c.n_topk.clone()
    return d


def _graph_vs_eager(wl, p, lengths, replays):
    n = len(lengths)
    q, k, v = synth.prefill_batch(wl, 0, lengths)
    eager = GpuCache(p, n)
    if eager.k_scale is not None:
        eager.k_scale.fill_(0.05)
        if eager.v_scale is not None:
            eager.v_scale.fill_(0.05)
    gpu_compress(p, eager, q, k, v, lengths, list(range(n)), debug=False)
    graphed = _clone(eager)
    sl = torch.arange(n, dtype=torch.int32, device="cuda")
    # static inputs of the captured step, refilled before every replay
    qd0, kn0, vn0 = synth.decode_inputs(wl, 0, 0, [0] * n, device="cuda")
    sq, sk = torch.empty_like(qd0), torch.empty_like(kn0)
    sv = None if vn0 is None else torch.empty_like(vn0)
    ws_g = snap.workspace(snap.snap_decode_workspace(p, n))
    ws_e = snap.workspace(snap.snap_decode_workspace(p, n))
    out_g = torch.zeros((n, p.n_q_heads, p.d_v), dtype=torch.bfloat16, device="cuda")
    out_e = torch.zeros_like(out_g)

    def fill(step):
        positions = eager.pos.cpu().tolist()
        qd, kn, vn = synth.decode_inputs(wl, 0, step, positions, device="cuda")
        sq.copy_(qd)
        sk.copy_(kn)
        if sv is not None:
            sv.copy_(vn)

    # warm up the library's launch path on a side stream, then capture one step
    fill(0)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        snap.snap_decode_step(p, graphed.c(), graphed.pos, graphed.n_topk, sl, sq, sk, sv, out_g, ws_g)
        snap.snap_advance(graphed.pos, sl)
    torch.cuda.synchronize()
    # capture does not execute: the graphed cache is still at step 0
    assert torch.equal(graphed.pos, eager.pos)
    for step in range(replays):
        fill(step)
        torch.cuda.synchronize()
        g.replay()
        snap.snap_decode_step(p, eager.c(), eager.pos, eager.n_topk, sl, sq, sk, sv, out_e, ws_e)
        snap.snap_advance(eager.pos, sl)
        torch.cuda.synchronize()
        assert torch.equal(out_g.view(torch.int16), out_e.view(torch.int16)), step
        assert torch.equal(graphed.k.view(torch.uint8), eager.k.view(torch.uint8)), step
        if eager.v is not None:
            assert torch.equal(graphed.v.view(torch.uint8), eager.v.view(torch.uint8)), step
        assert torch.equal(graphed.pos, eager.pos), step
        _ = torch.zeros(1 << 20, device="cuda").sum()  # eager work between replays


def test_graph_replay_gqa_bf16():
    wl = GQA
    print("\n[case] graph replay: bf16 GQA decode step (fused kernel + combine + advance), 6 replays", flush=True)
    _graph_vs_eager(wl, params_of(wl), [2900, 40, 1200], 6)


def test_graph_replay_latent_bf16():
    wl = synth.small(synth.WORKLOADS["mla-8head-61layer-b16-128k"], recent=64, topk=1000)
    print("\n[case] graph replay: bf16 latent decode step, 6 replays", flush=True)
    _graph_vs_eager(wl, params_of(wl), [3000, 1500], 6)


def test_graph_replay_fp8_fused():
    wl = synth.small(GQA, kv_dtype="fp8")
    print("\n[case] graph replay: fp8 GQA decode step (fused kernel + combine + advance), 4 replays", flush=True)
    _graph_vs_eager(wl, params_of(wl), [2000, 900], 4)


def test_graph_replay_fp32_two_launch_path():
    wl = synth.WORKLOADS["tiny-fp32"]
    print("\n[case] graph replay: fp32 decode step (append + attend launches), 4 replays", flush=True)
    _graph_vs_eager(wl, params_of(wl), [1024, 700], 4)


def test_graph_replay_prefill():
    """snap_prefill (V transpose, attention with the window statistics, then
    the compression) captured once and replayed on new prompts of the same
    lengths: every replay matches the eager call bit for bit (attention
    output, cache bytes, selection, metadata)."""
    wl = synth.Workload("graph-prefill", 15, 8, 2, 128, 128, False, 4, 32, 100, 32, 7, "bf16", "bf16", layers=1,
                        batch=2, length=None, length_range=(64, 1000), decode_steps=0, rope=True, plant_frac=0.01)
    p = params_of(wl)
    lengths = [900, 333]
    print(f"\n[case] graph replay: snap_prefill, lengths {lengths}, 3 replays", flush=True)
    dev = "cuda"
    n, ml = len(lengths), max(lengths)
    lens = torch.tensor(lengths, dtype=torch.int32, device=dev)
    sl = torch.arange(n, dtype=torch.int32, device=dev)
    q0, k0, v0 = (x.to(dev) for x in synth.prompt_batch(wl, 0, lengths))
    sq, sk, sv = torch.empty_like(q0), torch.empty_like(k0), torch.empty_like(v0)
    cg, ce = GpuCache(p, n), GpuCache(p, n)
    ws_g = snap.workspace(snap.snap_prefill_workspace(p, n, ml))
    ws_e = snap.workspace(snap.snap_prefill_workspace(p, n, ml))
    out_g = torch.zeros((n, p.n_q_heads, ml, p.d_v), dtype=torch.bfloat16, device=dev)
    out_e = torch.zeros_like(out_g)
    sel_g = torch.zeros((n, p.n_kv_heads, p.topk), dtype=torch.int32, device=dev)
    sel_e = torch.zeros_like(sel_g)
    sq.copy_(q0)
    sk.copy_(k0)
    sv.copy_(v0)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        snap.snap_prefill(p, cg.c(), cg.pos, cg.n_topk, sl, lens, sq, sk, sv, out_g, ws_g, sel_g)
    torch.cuda.synchronize()
    for rep in range(3):
        q, k, v = (x.to(dev) for x in synth.prompt_batch(wl, 0, lengths, salt=rep + 1))
        sq.copy_(q)
        sk.copy_(k)
        sv.copy_(v)
        torch.cuda.synchronize()
        g.replay()
        snap.snap_prefill(p, ce.c(), ce.pos, ce.n_topk, sl, lens, sq, sk, sv, out_e, ws_e, sel_e)
        torch.cuda.synchronize()
        assert torch.equal(out_g.view(torch.int16), out_e.view(torch.int16)), rep
        assert torch.equal(sel_g, sel_e), rep
        assert torch.equal(cg.k.view(torch.int16), ce.k.view(torch.int16)), rep
        assert torch.equal(cg.v.view(torch.int16), ce.v.view(torch.int16)), rep
        assert torch.equal(cg.pos, ce.pos) and torch.equal(cg.n_topk, ce.n_topk), rep
        _ = torch.zeros(1 << 20, device="cuda").sum()  # eager work between replays
