"""Library calls running concurrently on several HIP streams give the same
bytes as the same calls run one after another:

* one prompt compressed into four layers' caches on four streams at once (the
  layers share the slot's pos / n_topk entries, which compression only writes,
  with equal values), bf16 and fp8 caches with scales from the data;
* a new prompt compressed into one slot while the other slots take decode
  steps on a second stream (disjoint slots of the same caches and metadata).

Every case prints what names it before touching the GPU.
"""
from dataclasses import replace

import pytest
import torch

import paper_2511_03092_amd as snap
import synth
from snaphelp import GpuCache, params_of

pytestmark = pytest.mark.gpu

WL = synth.Workload("streams-gqa", 14, 8, 2, 128, 128, False, 4, 64, 400, 32, 7, "bf16", "bf16", layers=4, batch=1,
                    length=None, length_range=(900, 4000), decode_steps=3, rope=True, plant_frac=0.01)
LAYERS = 4


def _announce(msg):
    print(f"\n[case] {msg}", flush=True)


def _bytes_equal(a, b):
    return a is None and b is None or torch.equal(a.contiguous().view(torch.uint8), b.contiguous().view(torch.uint8))


def _compress_layers(p, wl, inputs, slot, n_slots, streams):
    """Compress the prompt of every layer into its own cache; with streams,
    layer l runs on streams[l % len(streams)] after the current stream's work
    so far, and the current stream waits for all of them."""
    caches = [GpuCache(p, n_slots) for _ in range(LAYERS)]
    pos, ntop = caches[0].pos, caches[0].n_topk  # slot metadata shared by the layers
    sl = torch.tensor([slot], dtype=torch.int32, device="cuda")
    cur = torch.cuda.current_stream()
    if streams:
        start = torch.cuda.Event()
        start.record(cur)
        for s in streams:
            s.wait_event(start)
    for l, (q, k, v, lens, ws) in enumerate(inputs):
        st = streams[l % len(streams)].cuda_stream if streams else None
        snap.snap_compress(p, caches[l].c(), pos, ntop, sl, lens, q, k, v, ws, stream=st)
    for s in streams:
        done = torch.cuda.Event()
        done.record(s)
        cur.wait_event(done)
    torch.cuda.synchronize()
    return caches


@pytest.mark.parametrize("kind", ["bf16", "fp8-amax"])
def test_layers_compressed_on_concurrent_streams(kind):
    wl = WL if kind == "bf16" else replace(WL, kv_dtype="fp8")
    p = params_of(wl) if kind == "bf16" else params_of(wl, fp8_scales=snap.SNAP_FP8_SCALES_AMAX)
    L = 3500
    _announce(f"{LAYERS} layers compressed on {LAYERS} streams, {kind} cache, L={L}")
    inputs = []
    for l in range(LAYERS):
        q, k, v = synth.prefill_batch(wl, l, [L], device="cuda")
        lens = torch.tensor([L], dtype=torch.int32, device="cuda")
        ws = snap.workspace(snap.snap_compress_workspace(p, 1, L))  # one workspace per concurrent call
        inputs.append((q, k, v, lens, ws))
    seq = _compress_layers(p, wl, inputs, 1, 2, [])
    conc = _compress_layers(p, wl, inputs, 1, 2, [torch.cuda.Stream() for _ in range(LAYERS)])
    for l in range(LAYERS):
        a, b = seq[l], conc[l]
        assert _bytes_equal(a.k, b.k) and _bytes_equal(a.v, b.v), l
        assert _bytes_equal(a.k_scale, b.k_scale) and _bytes_equal(a.v_scale, b.v_scale), l
    assert torch.equal(seq[0].pos, conc[0].pos) and torch.equal(seq[0].n_topk, conc[0].n_topk)
    assert int(conc[0].pos[1]) == L and int(conc[0].pos[0]) == -1


def test_compress_overlaps_decode_of_other_slots():
    wl, p = WL, params_of(WL)
    n_slots, first = 3, [2600, 1800]
    new_prompts = [3900, 950, 2200]  # one per step, each into slot 2
    _announce(f"compress into slot 2 on one stream, decode slots 0-1 on another, {len(new_prompts)} steps")

    def run(overlap):
        cache = GpuCache(p, n_slots)
        q, k, v = synth.prefill_batch(wl, 0, first, device="cuda")
        ws_c = snap.workspace(snap.snap_compress_workspace(p, 2, max(new_prompts + first)))
        snap.snap_compress(p, cache.c(), cache.pos, cache.n_topk, torch.tensor([0, 1], dtype=torch.int32,
                           device="cuda"), torch.tensor(first, dtype=torch.int32, device="cuda"), q, k, v, ws_c)
        torch.cuda.synchronize()
        dec_slots = torch.tensor([0, 1], dtype=torch.int32, device="cuda")
        ws_d = snap.workspace(snap.snap_decode_workspace(p, 2))
        outs = []
        s_c = torch.cuda.Stream() if overlap else torch.cuda.current_stream()
        s_d = torch.cuda.Stream() if overlap else torch.cuda.current_stream()
        positions = list(first)
        for t, Ln in enumerate(new_prompts):
            qn, kn_, vn_ = synth.prefill_batch(wl, 0, [Ln], device="cuda", salt=10 + t)
            qd, kd, vd = synth.decode_inputs(wl, 0, t, positions, device="cuda")
            lens = torch.tensor([Ln], dtype=torch.int32, device="cuda")
            out = torch.zeros((2, p.n_q_heads, p.d_v), dtype=torch.bfloat16, device="cuda")
            torch.cuda.synchronize()  # inputs made on the current stream are ready for both
            snap.snap_compress(p, cache.c(), cache.pos, cache.n_topk, torch.tensor([2], dtype=torch.int32,
                               device="cuda"), lens, qn, kn_, vn_, ws_c, stream=s_c.cuda_stream)
            snap.snap_decode_step(p, cache.c(), cache.pos, cache.n_topk, dec_slots, qd, kd, vd, out, ws_d,
                                  stream=s_d.cuda_stream)
            snap.snap_advance(cache.pos, dec_slots, stream=s_d.cuda_stream)
            torch.cuda.synchronize()
            outs.append(out)
            positions = [x + 1 for x in positions]
        return cache, outs

    a, oa = run(False)
    b, ob = run(True)
    for t in range(len(new_prompts)):
        assert _bytes_equal(oa[t], ob[t]), t
    assert _bytes_equal(a.k, b.k) and _bytes_equal(a.v, b.v)
    assert torch.equal(a.pos, b.pos) and torch.equal(a.n_topk, b.n_topk)
    assert a.pos.tolist() == [first[0] + 3, first[1] + 3, new_prompts[-1]]
