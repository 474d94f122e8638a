"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Every case prints what names it before touching the GPU.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2511_03092_amd as snap
import synth
from snaphelp import (DECISION_RTOL, NEAR_RTOL, NEAR_RTOL_ONE_ROW, TOL, GpuCache, check_compress, decode_steps,
                      gpu_compress, oracle_params, params_of, run_case)

pytestmark = pytest.mark.gpu

def _announce(msg):
    print(f"\n[case] {msg}", flush=True)


def _run_case(wl, p, lengths, slots, n_slots, steps, out_dtype, tol, **kw):
    return run_case(wl, p, lengths, slots, n_slots, steps, out_dtype, tol, **kw)


def test_tiny_fp32_workload():
    wl = synth.WORKLOADS["tiny-fp32"]
    _announce("tiny-fp32: L=1024, 4/2 heads, D64, budget 128, 16 decode steps")
    p = params_of(wl)
    _run_case(wl, p, [wl.length], [0], 1, wl.decode_steps, torch.float32, TOL["f32"])


def test_llama_one_layer_32k_workload():
    wl = synth.WORKLOADS["llama8b-1layer-32k"]
    _announce("llama8b-1layer-32k: L=32768, 32/8 heads, budget 4096, 256 decode steps")
    p = params_of(wl)
    _run_case(wl, p, [wl.length], [0], 1, wl.decode_steps, torch.bfloat16, TOL["bf16"],
                         check_every=8)


MED = synth.Workload("med", 11, 8, 2, 128, 128, False, 4, 16, 300, 32, 13, "bf16", "bf16", layers=1, batch=3,
                     length=None, length_range=(700, 5100), decode_steps=40, rope=True, plant_frac=0.01)


@pytest.mark.parametrize("norm", [snap.SNAP_NORM_CAND, snap.SNAP_NORM_ROW])
@pytest.mark.parametrize("pool", [snap.SNAP_POOL_MAX, snap.SNAP_POOL_AVG])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_variants_ragged_batch(norm, pool, dtype):
    """Both normaliser domains and pool types, three ragged prompts padded with
    NaN to one max_len, window (32) longer than the ring (16) so the causal
    mask inside the window matters."""
    wl = synth.small(MED, in_dtype=dtype, kv_dtype=dtype, pool=pool, norm=norm)
    _announce(f"variants norm={norm} pool={pool} dtype={dtype}")
    p = params_of(wl)
    lengths = [5000, 777, 3001]
    _run_case(wl, p, lengths, [2, 0, 1], 3, 24, torch.float32 if dtype == "f32" else torch.bfloat16,
                         TOL[dtype])


EDGE = synth.Workload("edge", 12, 4, 2, 64, 64, False, 4, 8, 16, 16, 5, "f32", "f32", layers=1, batch=1,
                      length=None, length_range=(1, 100), decode_steps=12, rope=False, plant_count=3)


@pytest.mark.parametrize("topk", [0, 16])
def test_edge_lengths(topk):
    """L = 0, 1, inside the sinks, inside sinks+ring (no candidates), exactly
    sinks+ring, one candidate, candidates == K, one more than K, longer than
    the window; decode steps then wrap the ring from every start."""
    wl = synth.small(EDGE, topk=topk)
    p = params_of(wl)
    s, r = wl.sink, wl.recent
    lengths = [0, 1, 3, s + 5, s + r, s + r + 1, s + r + topk, s + r + topk + 1, 90]
    _announce(f"edge lengths {lengths} topk={topk}")
    _run_case(wl, p, lengths, list(range(len(lengths))), len(lengths), 20, torch.float32, TOL["f32"])


# Selection policies beside the default: StreamingLLM alone (no selected
# rows), a SAGE-KV-like choice (the last query only, no pooling), and the
# paper's two hyper-parameter presets (Table 6: Llama 768 sinks / 6400 selected
# / 1024 recent; DeepSeek 512 / 512 / 31744; window 32, pool kernel 13).
# With a single window row the pooled score of a key sums only G = 4 weights,
# so the fp32 rounding of one logit is not averaged down over G*w rows: the
# near-band bound is NEAR_RTOL_ONE_ROW there.  The decision band (re-scored in
# fp64) and the selection rule (swaps only within 1e-6) are unchanged.
POLICIES = {
    "streamingllm": (lambda: synth.small(MED, topk=0), [5000, 777, 3001], 24, 1, NEAR_RTOL),
    "sagekv-like": (lambda: synth.small(MED, obs_window=1, pool_kernel=1), [5000, 777, 3001], 24, 1,
                    NEAR_RTOL_ONE_ROW),
    "table6-llama": (lambda: synth.small(synth.WORKLOADS["llama8b-1layer-32k"], sink=768, recent=1024, topk=6400,
                                         pool_kernel=13), [32768, 9000], 8, 4, NEAR_RTOL),
    "table6-deepseek": (lambda: synth.small(synth.WORKLOADS["mla-8head-61layer-b16-128k"], sink=512, recent=31744,
                                            topk=512, pool_kernel=13), [40000], 4, 2, NEAR_RTOL),
}


@pytest.mark.parametrize("scale", [0.3, 0.02])
def test_caller_softmax_scale(scale):
    """A softmax scale the caller sets (sm_scale > 0) in place of 1/sqrt(d):
    0.3 gives logits 3.4 times the default's, 0.02 flattens the softmax.
    Compression and decode against the oracle with the same scale (Eq. 3,
    Sec. III-C).  The pooled scores' fp32 error comes from the rounding of
    the logits (it is proportional to their magnitude), so the score bounds,
    set for the default scale, grow by sm_scale * sqrt(d) when that exceeds
    1; the selection rule and the decode bound do not change."""
    wl = synth.small(MED, topk=200)
    p = params_of(wl, sm_scale=scale)
    lengths = [4000, 1500]
    factor = max(1.0, scale * wl.d_qk ** 0.5)
    _announce(f"sm_scale {scale}: G=4 D=128, lengths {lengths}, 16 decode steps, score bounds x{factor:.2f}")
    _run_case(wl, p, lengths, [1, 0], 2, 16, torch.bfloat16, TOL["bf16"], score_rtol_factor=factor)


@pytest.mark.parametrize("name", list(POLICIES))
def test_selection_policies(name):
    make, lengths, steps, every, band = POLICIES[name]
    wl = make()
    p = params_of(wl)
    _announce(f"policy {name}: sink {wl.sink}, recent {wl.recent}, topk {wl.topk}, window {wl.obs_window}, "
              f"pool kernel {wl.pool_kernel}, lengths {lengths}")
    _run_case(wl, p, lengths, list(range(len(lengths))), len(lengths), steps, torch.bfloat16, TOL["bf16"],
              check_every=every, near_rtol=band)


def test_streamingllm_assembly_only():
    """topk = 0 without the debug outputs: the call only assembles sinks and
    ring (nothing is scored); cache bytes and metadata against the oracle's
    assembly, then decode steps against the oracle."""
    wl = synth.small(MED, topk=0)
    p = params_of(wl)
    lengths = [5000, 12, 3001]
    _announce(f"streamingllm, assembly only: lengths {lengths}")
    q, k, v = synth.prefill_batch(wl, 0, lengths, pad_value=float("nan"))
    cache = GpuCache(p, 3)
    gpu_compress(p, cache, q, k, v, lengths, [2, 0, 1], debug=False)
    ck, cv = cache.host_values()
    for b, (L, sl) in enumerate(zip(lengths, [2, 0, 1])):
        assert int(cache.pos[sl]) == L and int(cache.n_topk[sl]) == 0
        for g in range(p.n_kv_heads):
            ek = oracle.assemble(L, p.sink, p.recent, 0, oracle.f64(k[b, g, :L]), np.zeros(0, np.int32))
            ev = oracle.assemble(L, p.sink, p.recent, 0, oracle.f64(v[b, g, :L]), np.zeros(0, np.int32))
            assert np.array_equal(ck[sl, g], ek) and np.array_equal(cv[sl, g], ev), (b, g)
    err = decode_steps(p, wl, cache, [2, 0, 1], 24, torch.bfloat16, TOL["bf16"])
    print(f"  decode max abs err over 24 steps: {err:.3e}", flush=True)


def test_invalid_slots_are_skipped():
    wl = synth.small(EDGE, topk=16)
    p = params_of(wl)
    _announce("invalid slot ids -1 and n_slots are skipped")
    lengths = [60, 70, 80]
    q, k, v = synth.prefill_batch(wl, 0, lengths)
    cache = GpuCache(p, 2)
    cache.k.fill_(7.0)
    cache.v.fill_(7.0)
    slots = [-1, 1, 2]
    sel, pooled = gpu_compress(p, cache, q, k, v, lengths, slots)
    assert torch.all(cache.k[0] == 7.0) and torch.all(cache.v[0] == 7.0)
    assert int(cache.pos[0]) == -1 and int(cache.pos[1]) == 70
    check_compress(p, cache, q, k, v, lengths, slots, sel, pooled)
    # decode on a batch that names a bad slot leaves everything else right
    sl = torch.tensor([1, 5], dtype=torch.int32, device="cuda")
    ws = snap.workspace(snap.snap_decode_workspace(p, 2))
    out = torch.full((2, p.n_q_heads, p.d_v), 3.0, device="cuda")
    qd, kn, vn = synth.decode_inputs(wl, 0, 0, [70, 0])
    snap.snap_cache_append(p, cache.c(), cache.pos, sl, kn.cuda(), vn.cuda())
    snap.snap_decode_attn(p, cache.c(), cache.pos, cache.n_topk, sl, qd.cuda(), out, ws)
    snap.snap_advance(cache.pos, sl)
    torch.cuda.synchronize()
    assert torch.all(out[1] == 3.0)
    assert int(cache.pos[1]) == 71
    ck, cv = cache.host_values()
    exp = oracle.decode_attn(oracle_params(p), [70], cache.n_topk.cpu().numpy()[[1]],
                             qd[:1], ck[[1]], cv[[1]])
    assert np.max(np.abs(out[:1].double().cpu().numpy() - exp)) <= TOL["f32"]


def test_fp8_cache_continuous_batching_shape():
    """fp8 E4M3 cache with per-(slot, head) scales, the continuous-batching
    workload's budget split (768 sinks, 1024 recent, 6400 selected)."""
    wl = synth.WORKLOADS["cb-fp8-llama8b-32slot"]
    p = params_of(wl)
    lengths = [9000, 20000]
    _announce(f"fp8 cache lengths {lengths} into slots [5, 2] of 8")
    _run_case(wl, p, lengths, [5, 2], 8, 32, torch.bfloat16, TOL["fp8"], fp8_scales=True,
                         check_every=4)


def test_fp8_scales_from_data():
    """SNAP_FP8_SCALES_AMAX: compress sets each (slot, KV head) scale to the
    oracle's data scale of the rows the cache keeps (K and V apart; the
    scales the caller left are overwritten), the codes are the oracle's
    quantisation with it (checked by check_compress), and decode steps that
    append past the kept rows' range match the oracle.  One prompt is shorter
    than sinks + ring (no candidates), one has every candidate kept."""
    wl = synth.WORKLOADS["cb-fp8-llama8b-32slot"]
    p = params_of(wl, fp8_scales=snap.SNAP_FP8_SCALES_AMAX)
    s, r, K = p.sink, p.recent, p.topk
    lengths = [9000, 20000, 1500, s + r + 100]
    slots = [5, 2, 7, 0]
    _announce(f"fp8 scales from the data: lengths {lengths} into slots {slots} of 8")
    q, k, v = synth.prefill_batch(wl, 0, lengths, pad_value=float("nan"))
    cache = GpuCache(p, 8)
    cache.k_scale.fill_(3.0)
    cache.v_scale.fill_(3.0)
    sel, pooled = gpu_compress(p, cache, q, k, v, lengths, slots)
    stats = check_compress(p, cache, q, k, v, lengths, slots, sel, pooled)
    assert stats["decision_rel_err"] <= DECISION_RTOL and stats["near_rel_err"] <= NEAR_RTOL
    nt = cache.n_topk.cpu().numpy()
    for b, (L, sl) in enumerate(zip(lengths, slots)):
        for g in range(p.n_kv_heads):
            used = sel[b, g, :nt[sl]]
            for src, scales in ((k, cache.k_scale), (v, cache.v_scale)):
                rows = oracle.assemble(L, s, r, K, oracle.f64(src[b, g, :L]), used)
                assert float(scales[sl, g]) == oracle.fp8_scale(rows), (b, g)
    untouched = [x for x in range(8) if x not in slots]
    assert torch.all(cache.k_scale[untouched] == 3.0) and torch.all(cache.v_scale[untouched] == 3.0)
    err = decode_steps(p, wl, cache, slots, 16, torch.bfloat16, TOL["fp8"], check_every=4)
    print(f"  decode max abs err over 16 steps: {err:.3e}", flush=True)


def test_mla_latent_cache_reduced_length():
    """Latent (MLA) cache: 8 heads share one 576-wide row, values are its first
    512 dims; the workload's split at a shorter prompt."""
    wl = synth.small(synth.WORKLOADS["mla-8head-61layer-b16-128k"], recent=512, topk=2048)
    p = params_of(wl)
    lengths = [8192, 5000]
    _announce(f"mla latent lengths {lengths}")
    _run_case(wl, p, lengths, [1, 0], 2, 8, torch.bfloat16, TOL["bf16"])


def test_compress_is_deterministic():
    wl = synth.small(MED, norm=snap.SNAP_NORM_CAND)
    p = params_of(wl)
    lengths = [5000, 4096]
    _announce("determinism: two identical compress calls")
    q, k, v = synth.prefill_batch(wl, 0, lengths)
    outs = []
    for _ in range(2):
        cache = GpuCache(p, 2)
        sel, pooled = gpu_compress(p, cache, q, k, v, lengths, [0, 1])
        outs.append((sel, pooled, cache.k.cpu(), cache.v.cpu()))
    assert np.array_equal(outs[0][0], outs[1][0])
    assert np.array_equal(outs[0][1], outs[1][1], equal_nan=True)
    assert torch.equal(outs[0][2], outs[1][2]) and torch.equal(outs[0][3], outs[1][3])
