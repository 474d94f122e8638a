"""Seeded random sweep over the configurations the C ABI accepts: for each
case a fresh draw of the head layout (G, KV heads), widths (64/128, the
576/512 latent cache, 64/128 caches with values inside the key rows), input
and cache dtypes (bf16, fp8 with given or data scales, fp32), observation
window, pool kernel and type, normaliser domain, sink / recent / top-K
budget, load hint, output dtype, batch and prompt lengths (edge lengths
below sink + recent among them), all compressed into random slots of a
canary-filled cache and decoded across ring wraps, each checked against the
fp64 oracle by run_case (selection, pooled scores, cache bytes, untouched
slots, decode on the GPU's cache and end to end).

The draws come from random.Random(seed) alone; test_random_configs_are_accepted
(CPU) checks that every draw is inside what the ABI accepts.  Every case
prints its configuration before touching the GPU.
"""
import random

import pytest
import torch

import paper_2511_03092_amd as snap
import synth
from snaphelp import NEAR_RTOL, NEAR_RTOL_ONE_ROW, TOL, params_of, run_case

N_CASES = 64
SEED = 2511


def draw(i: int):
    """Case i of the sweep: (workload, params overrides, lengths, slots,
    n_slots, decode steps, out dtype, near-band tolerance, fp8 scales set by
    the harness)."""
    r = random.Random(SEED * 1000 + i)
    kind = r.choice(["gqa64", "gqa128", "latent576", "vink64", "vink128"])
    if kind == "latent576":
        d_qk, d_v, v_in_k, hkv = 576, 512, True, 1
        dts = r.choice([("bf16", "bf16"), ("bf16", "fp8")])
    else:
        d = 64 if kind.endswith("64") else 128
        d_qk, d_v, v_in_k, hkv = d, d, kind.startswith("vink"), r.choice([1, 2, 4])
        dts = r.choice([("bf16", "bf16"), ("bf16", "fp8"), ("f32", "f32")])
    rows_max = 128 if dts[0] == "f32" else 256
    while True:
        G = r.choice([1, 2, 3, 4, 6, 8, 16])
        w = r.choice([1, 2, 5, 8, 16, 32])
        if G * w <= rows_max:
            break
    sink = r.randint(0, 8)
    recent = r.randint(1, 64)
    topk = r.choice([0, r.randint(1, 64), r.randint(65, 700)])
    pool_kernel = r.choice([1, 3, 5, 7, 13])
    pool = r.choice([synth.POOL_MAX, synth.POOL_AVG])
    norm = r.choice([synth.NORM_CAND, synth.NORM_ROW])
    batch = r.randint(1, 3)
    sr = sink + recent
    lengths = [r.choice([r.randint(1, sr + 3), r.randint(sr + 1, 4000), r.randint(2000, 4000)]) for _ in range(batch)]
    n_slots = batch + r.randint(0, 2)
    slots = r.sample(range(n_slots), batch)
    latent_recipe = v_in_k
    wl = synth.Workload(f"rand-{i}", 100 + i, G * hkv, hkv, d_qk, d_v, v_in_k, sink, recent, topk, w, pool_kernel,
                        dts[0], dts[1], layers=1, batch=batch, length=None, length_range=(1, 4000),
                        decode_steps=12, rope=not latent_recipe, plant_frac=None if latent_recipe else 0.01,
                        pool=pool, norm=norm)
    over = {"kv_reuse": r.choice([snap.SNAP_KV_AUTO, snap.SNAP_KV_STREAM, snap.SNAP_KV_KEEP])}
    given = False
    if dts[1] == "fp8":
        if r.random() < 0.5:
            over["fp8_scales"] = snap.SNAP_FP8_SCALES_AMAX
        else:
            given = True
    out_dtype = torch.float32 if (dts[0] == "f32" or r.random() < 0.3) else torch.bfloat16
    near = NEAR_RTOL_ONE_ROW if G * w < 8 else NEAR_RTOL
    return wl, over, lengths, slots, n_slots, 12, out_dtype, near, given


def test_random_configs_are_accepted():
    """Every draw passes the library's parameter checks (host only)."""
    for i in range(N_CASES):
        wl, over, lengths, slots, n_slots, *_ = draw(i)
        p = params_of(wl, **over)
        assert snap.snap_compress_workspace(p, len(lengths), max(lengths)) > 0, (i, wl)
        assert snap.snap_decode_workspace(p, len(lengths)) > 0, (i, wl)


@pytest.mark.gpu
@pytest.mark.parametrize("i", range(N_CASES))
def test_random_config(i):
    wl, over, lengths, slots, n_slots, steps, out_dtype, near, given = draw(i)
    p = params_of(wl, **over)
    print(f"\n[case] random {i}: Hq {p.n_q_heads} Hkv {p.n_kv_heads} d ({p.d_qk},{p.d_v}) v_in_k {int(p.v_in_k)} "
          f"in {wl.in_dtype} cache {wl.kv_dtype} fp8_scales {p.fp8_scales} given {given} window {p.obs_window} "
          f"pool {p.pool}/{p.pool_kernel} norm {p.norm} sink {p.sink} recent {p.recent} topk {p.topk} "
          f"kv_reuse {p.kv_reuse} out {out_dtype} lengths {lengths} -> slots {slots} of {n_slots}", flush=True)
    # even steps: snap_cache_append + snap_decode_attn; odd steps: snap_decode_step
    run_case(wl, p, lengths, slots, n_slots, steps, out_dtype, TOL[wl.kv_dtype], check_every=3, fp8_scales=given,
             near_rtol=near, salt=i, fused="alt")


N_PREFILL = 16


def draw_prefill(i: int):
    """Prefill case i: a configuration snap_prefill accepts (bf16 inputs, d 64
    or 128 with a separate V, G in 1, 2, 4, 8, 16) with a bf16 or fp8 cache."""
    r = random.Random(SEED * 1000 + 500 + i)
    d = r.choice([64, 128])
    hkv = r.choice([1, 2])
    while True:
        G = r.choice([1, 2, 4, 8, 16])
        w = r.choice([1, 4, 16, 32])
        if G * w <= 256:
            break
    sink, recent = r.randint(0, 8), r.randint(1, 48)
    topk = r.choice([0, r.randint(1, 300)])
    kv = r.choice(["bf16", "fp8"])
    batch = r.randint(1, 3)
    lengths = [r.choice([r.randint(1, sink + recent + 3), r.randint(100, 1200)]) for _ in range(batch)]
    n_slots = batch + r.randint(0, 1)
    slots = r.sample(range(n_slots), batch)
    wl = synth.Workload(f"rand-pf-{i}", 200 + i, G * hkv, hkv, d, d, False, sink, recent, topk, w,
                        r.choice([1, 3, 7]), "bf16", kv, layers=1, batch=batch, length=None, length_range=(1, 1200),
                        decode_steps=0, rope=True, plant_frac=0.01, pool=r.choice([synth.POOL_MAX, synth.POOL_AVG]),
                        norm=r.choice([synth.NORM_CAND, synth.NORM_ROW]))
    over = {"fp8_scales": snap.SNAP_FP8_SCALES_AMAX} if kv == "fp8" else {}
    near = NEAR_RTOL_ONE_ROW if G * w < 8 else NEAR_RTOL
    return wl, over, lengths, slots, n_slots, near


def test_random_prefill_configs_are_accepted():
    for i in range(N_PREFILL):
        wl, over, lengths, slots, n_slots, _ = draw_prefill(i)
        p = params_of(wl, **over)
        assert snap.snap_prefill_workspace(p, len(lengths), max(lengths)) > 0, (i, wl)


@pytest.mark.gpu
@pytest.mark.parametrize("i", range(N_PREFILL))
def test_random_prefill_config(i):
    """snap_prefill on a random accepted configuration: the attention output
    of every position and the fused compression against the oracle."""
    from test_gpu_prefill import _run
    wl, over, lengths, slots, n_slots, near = draw_prefill(i)
    p = params_of(wl, **over)
    print(f"\n[case] random prefill {i}: Hq {p.n_q_heads} Hkv {p.n_kv_heads} d {p.d_qk} cache {wl.kv_dtype} "
          f"window {p.obs_window} pool {p.pool}/{p.pool_kernel} norm {p.norm} sink {p.sink} recent {p.recent} "
          f"topk {p.topk} lengths {lengths} -> slots {slots} of {n_slots}", flush=True)
    _run(wl, p, lengths, slots=slots, n_slots=n_slots, near_rtol=near)
