"""GPU parity of snap_prefill (causal prefill attention with the SnapKV window
statistics taken from the attention pass, then the compression) against the
fp64 oracle: the attention output of every position, within the error bf16
arithmetic allows (attention_bound), and the compression result (selection,
pooled scores, cache bytes, metadata) for the observation window formed by
the last w prompt queries.

Every case prints what names it before touching the GPU.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2511_03092_amd as snap
import synth
from snaphelp import (ALL_RTOL, DECISION_RTOL, NEAR_RTOL, GpuCache, check_compress, check_selection,
                      oracle_params, params_of, score_errors)

pytestmark = pytest.mark.gpu

# 8 query heads over 2 KV heads (G = 4, the Llama grouping), D = 128
GQA = synth.Workload("prefill-gqa", 14, 8, 2, 128, 128, False, 4, 32, 100, 32, 7, "bf16", "bf16", layers=1, batch=4,
                     length=None, length_range=(64, 1000), decode_steps=0, rope=True, plant_frac=0.01)


def _announce(msg):
    print(f"\n[case] {msg}", flush=True)


def _gpu_prefill(p, wl, lengths, slots, n_slots, max_len=None, salt=0):
    q, k, v = synth.prompt_batch(wl, 0, lengths, salt=salt, max_len=max_len, pad_value=float("nan"), slots=slots)
    dev = "cuda"
    n, ml = k.shape[0], k.shape[2]
    cache = GpuCache(p, n_slots)
    qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
    lens = torch.tensor(lengths, dtype=torch.int32, device=dev)
    sl = torch.tensor(slots, dtype=torch.int32, device=dev)
    ws = snap.workspace(snap.snap_prefill_workspace(p, n, ml))
    # canary: rows at or past each prompt's length must stay untouched
    out = torch.full((n, p.n_q_heads, ml, p.d_v), float("nan"), dtype=torch.bfloat16, device=dev)
    sel = torch.empty((n, p.n_kv_heads, max(p.topk, 1)), dtype=torch.int32, device=dev)
    pooled = torch.empty((n, p.n_kv_heads, ml), dtype=torch.float32, device=dev)
    snap.snap_prefill(p, cache.c(), cache.pos, cache.n_topk, sl, lens, qd, kd, vd, out, ws, sel, pooled)
    torch.cuda.synchronize()
    return q, k, v, cache, out, sel.cpu().numpy(), pooled.cpu().numpy()


# bf16's unit roundoff (8-bit significand, rounding to nearest)
U_BF16 = 2.0 ** -8


def attention_bound(exp, exp_absv):
    """The largest error a bf16 attention output may carry, element by element:
    the probabilities enter the P V product rounded to bf16 (each within u,
    relative) and the output is stored in bf16 (within u, relative), so
    |got - exp| <= u (|exp| + sum_j p_j |v_j|) (1 + 2u), where sum_j p_j |v_j| is
    the oracle's attention over |v|; 1e-5 covers the fp32 logits and sums."""
    return U_BF16 * (np.abs(exp) + exp_absv) * (1 + 2 * U_BF16) + 1e-5


def _check_attention(p, lengths, q, k, v, out):
    """Every output position against the oracle within attention_bound (the
    attention over |v| is formed for the sequences whose error the |exp| term
    alone does not cover).  Returns the largest absolute error and the largest
    ratio of error to bound."""
    op = oracle_params(p)
    exp = oracle.prefill_attn(op, lengths, q, k, v)
    worst, worst_ratio = 0.0, 0.0
    for b, L in enumerate(lengths):
        assert torch.all(torch.isnan(out[b, :, L:].float())), f"rows past L={L} written"
        if not L:
            continue
        got = out[b, :, :L].double().cpu().numpy()
        err = np.abs(got - exp[b])
        absv = 0.0
        if not np.all(err <= attention_bound(exp[b], 0.0)):
            absv = oracle.prefill_attn(op, [L], q[b:b + 1], k[b:b + 1], np.abs(oracle.f64(v[b:b + 1])))[0]
        ratio = float(np.max(err / attention_bound(exp[b], absv)))
        assert ratio <= 1.0, (b, L, float(np.max(err)), ratio)
        worst, worst_ratio = max(worst, float(np.max(err))), max(worst_ratio, ratio)
    return worst, worst_ratio


def _run(wl, p, lengths, slots=None, n_slots=None, near_rtol=NEAR_RTOL, max_len=None):
    slots = list(range(len(lengths))) if slots is None else slots
    n_slots = len(lengths) if n_slots is None else n_slots
    q, k, v, cache, out, sel, pooled = _gpu_prefill(p, wl, lengths, slots, n_slots, max_len=max_len)
    err, ratio = _check_attention(p, lengths, q, k, v, out)
    qobs = oracle.window_queries(oracle_params(p), lengths, q)
    st = check_compress(p, cache, qobs, k, v, lengths, slots, sel, pooled)
    print(f"  attention max abs err {err:.3e} ({ratio:.2f} of the bf16 bound); swaps {st['swaps']}, pooled max rel err "
          f"{st['pooled_rel_err']:.3e}, decision band {st['decision_rel_err']:.3e}, near band "
          f"{st['near_rel_err']:.3e}", flush=True)
    assert st["decision_rel_err"] <= DECISION_RTOL and st["near_rel_err"] <= near_rtol
    assert st["pooled_rel_err"] <= ALL_RTOL
    return st


@pytest.mark.parametrize("norm", [synth.NORM_CAND, synth.NORM_ROW])
def test_prefill_gqa_ragged_batch(norm):
    wl = synth.small(GQA, norm=norm)
    p = params_of(wl)
    lengths = [1000, 333, 97, 1]
    _announce(f"snap_prefill G=4 D=128 norm={'cand' if norm == 0 else 'row'}: lengths {lengths} (ragged tiles, "
              "one prompt of one token)")
    _run(wl, p, lengths, slots=[2, 0, 3, 1], n_slots=5)


@pytest.mark.parametrize("hq,hkv,d", [(4, 4, 64), (8, 4, 64), (8, 1, 64), (16, 2, 128), (16, 1, 128), (32, 2, 64)])
def test_prefill_group_sizes(hq, hkv, d):
    wl = synth.small(GQA, n_q_heads=hq, n_kv_heads=hkv, d_qk=d, d_v=d, obs_window=16)
    p = params_of(wl)
    lengths = [777, 130]
    _announce(f"snap_prefill Hq={hq} Hkv={hkv} (G={hq // hkv}) D={d}: lengths {lengths}")
    _run(wl, p, lengths)


@pytest.mark.parametrize("hq,hkv,d,w,recent,norm", [(8, 1, 64, 32, 16, synth.NORM_CAND),
                                                    (8, 2, 128, 64, 40, synth.NORM_ROW)])
def test_prefill_largest_window(hq, hkv, d, w, recent, norm):
    """The largest window (G * w = 256 score rows: exactly one attention
    workgroup's block of 256 / G positions) with w > recent, so the causal
    mask also cuts the candidate domain of the first window rows."""
    wl = synth.small(GQA, n_q_heads=hq, n_kv_heads=hkv, d_qk=d, d_v=d, obs_window=w, recent=recent, norm=norm)
    p = params_of(wl)
    lengths = [700, 161, 90, 50]
    _announce(f"snap_prefill window {w} = one block of {256 // (hq // hkv)} positions, G={hq // hkv} D={d} "
              f"recent={recent} norm={'cand' if norm == 0 else 'row'}: lengths {lengths}")
    _run(wl, p, lengths)


def test_prefill_short_prompts_and_window_longer_than_prompt():
    wl = synth.small(GQA, sink=8, recent=16, topk=20, obs_window=32)
    p = params_of(wl)
    lengths = [20, 24, 25, 31, 45, 2, 0]
    _announce(f"snap_prefill short prompts (L <= sink+recent, L < w, an empty prompt), padded to 300: "
              f"lengths {lengths}")
    _run(wl, p, lengths, max_len=300)


def test_prefill_streaming_only():
    wl = synth.small(GQA, topk=0)
    p = params_of(wl)
    lengths = [900, 150]
    _announce(f"snap_prefill with topk = 0 (sinks and ring only): lengths {lengths}")
    q, k, v, cache, out, sel, pooled = _gpu_prefill(p, wl, lengths, [0, 1], 2)
    _check_attention(p, lengths, q, k, v, out)
    op = oracle_params(p)
    for b, L in enumerate(lengths):
        assert int(cache.pos[b]) == L and int(cache.n_topk[b]) == 0
        for g in range(p.n_kv_heads):
            ek = oracle.assemble(L, p.sink, p.recent, 0, oracle.f64(k[b, g, :L]), np.zeros(0, np.int32))
            assert np.array_equal(cache.k[b, g].double().cpu().numpy(), ek)


def _sampled_rows(p, qc, kc, vc, out, L, rows, heads):
    """Output rows of one sequence recomputed by the oracle one by one: row i
    of head h needs q_{h,i} and the keys and values of positions 0..i only.
    qc [Hq][L][dk], kc / vc [Hkv][L][d] fp64 on the host."""
    op = oracle_params(p)
    G = op.group
    worst = 0.0
    for h in heads:
        g = h // G
        for i in rows:
            qq = np.zeros((1, i + 1, p.d_qk))
            qq[0, i] = qc[h, i]
            exp = oracle.prefill_attn_group(op, i + 1, qq, kc[g, :i + 1], vc[g, :i + 1], rows=(i, i + 1))
            expa = oracle.prefill_attn_group(op, i + 1, qq, kc[g, :i + 1], np.abs(vc[g, :i + 1]), rows=(i, i + 1))
            got = out[h, i].double().cpu().numpy()
            e = np.abs(got - exp[0, 0])
            err = float(np.max(e))
            worst = max(worst, err)
            assert np.all(e <= attention_bound(exp[0, 0], expa[0, 0])), (h, i, err)
    return worst


def test_prefill_full_size_llama_32k():
    """The one-layer 32k Llama shape at full size, in the launch bench.py
    times: sampled output rows (first tiles, tile edges, the window, random)
    of every head against the oracle one by one, every output row finite,
    and the selection of three KV heads against the oracle's compression."""
    wl = synth.WORKLOADS["llama8b-1layer-32k"]
    p = params_of(wl)
    L = wl.length
    _announce(f"snap_prefill llama8b-1layer-32k at full size: L={L}, 32/8 heads")
    dev = "cuda"
    q, k, v = synth.prompt_batch(wl, 0, [L], device=dev)
    cache = GpuCache(p, 1)
    ws = snap.workspace(snap.snap_prefill_workspace(p, 1, L))
    out = torch.empty((1, p.n_q_heads, L, p.d_v), dtype=torch.bfloat16, device=dev)
    sel = torch.empty((1, p.n_kv_heads, p.topk), dtype=torch.int32, device=dev)
    pooled = torch.empty((1, p.n_kv_heads, L), dtype=torch.float32, device=dev)
    one = torch.zeros(1, dtype=torch.int32, device=dev)
    lens = torch.tensor([L], dtype=torch.int32, device=dev)
    snap.snap_prefill(p, cache.c(), cache.pos, cache.n_topk, one, lens, q, k, v, out, ws, sel, pooled)
    torch.cuda.synchronize()
    assert torch.isfinite(out.float()).all()
    gen = np.random.default_rng(5)
    rows = sorted(set([0, 1, 63, 64, 65, 127, 4095, 4096] + list(range(L - 33, L)) +
                      gen.integers(0, L, 6).tolist()))
    qc, kc, vc = oracle.f64(q[0]), oracle.f64(k[0]), oracle.f64(v[0])
    err = _sampled_rows(p, qc, kc, vc, out[0], L, rows[::3], range(p.n_q_heads))
    err = max(err, _sampled_rows(p, qc, kc, vc, out[0], L, rows, [0, 13, 31]))
    op = oracle_params(p)
    qobs = oracle.window_queries(op, [L], qc[None])
    G = op.group
    worst, worst_near = 0.0, 0.0
    for g in [0, 3, 7]:
        res = oracle.compress_group(op, L, qobs[0, g * G:(g + 1) * G], kc[g], vc[g])
        gs = sel[0, g].cpu().numpy()
        swaps = check_selection(gs, res.P, L, p.sink, p.recent, p.topk)
        keff = min(L - p.sink - p.recent, p.topk)
        e = score_errors(pooled[0, g, p.sink:L - p.recent].double().cpu().numpy(), res.P[p.sink:L - p.recent], keff)
        worst = max(worst, e["decision"])
        worst_near = max(worst_near, e["near"])
        ek = oracle.assemble(L, p.sink, p.recent, p.topk, kc[g], gs[:keff])
        assert np.array_equal(cache.k[0, g].double().cpu().numpy(), ek)
        print(f"  head {g}: swaps {swaps}, pooled-score rel err: decision band {e['decision']:.3e}, near band "
              f"{e['near']:.3e}", flush=True)
    print(f"  sampled attention max abs err {err:.3e}", flush=True)
    assert worst <= DECISION_RTOL and worst_near <= NEAR_RTOL
    assert int(cache.pos[0]) == L and int(cache.n_topk[0]) == p.topk


def test_prefill_attn_alone_matches_prefill_output():
    """snap_prefill_attn runs the same attention without the compression: its
    output equals snap_prefill's bit for bit and matches the oracle."""
    wl = GQA
    p = params_of(wl)
    lengths = [1000, 333, 97, 1]
    _announce(f"snap_prefill_attn alone vs snap_prefill: lengths {lengths}")
    q, k, v, cache, out, sel, pooled = _gpu_prefill(p, wl, lengths, [0, 1, 2, 3], 4)
    dev = "cuda"
    n, ml = k.shape[0], k.shape[2]
    lens = torch.tensor(lengths, dtype=torch.int32, device=dev)
    ws = snap.workspace(snap.snap_prefill_workspace(p, n, ml))
    out2 = torch.full_like(out, float("nan"))
    snap.snap_prefill_attn(p, lens, q.to(dev), k.to(dev), v.to(dev), out2, ws)
    torch.cuda.synchronize()
    assert torch.equal(out2.view(torch.int16), out.view(torch.int16))
    _check_attention(p, lengths, q, k, v, out2)


@pytest.mark.parametrize("scales", ["given", "amax"])
def test_prefill_into_fp8_cache(scales):
    """snap_prefill into an fp8 cache: caller-set scales, or scales from the
    kept rows (SNAP_FP8_SCALES_AMAX); every code against the oracle's
    quantisation of the oracle's assembly, selection as for bf16."""
    wl = synth.small(GQA, kv_dtype="fp8")
    p = params_of(wl, fp8_scales=snap.SNAP_FP8_SCALES_AMAX if scales == "amax" else snap.SNAP_FP8_SCALES_GIVEN)
    lengths = [1000, 333]
    _announce(f"snap_prefill into an fp8 cache, scales {scales}: lengths {lengths}")
    slots = [1, 0]
    q, k, v = synth.prompt_batch(wl, 0, lengths, pad_value=float("nan"), slots=slots)
    dev = "cuda"
    n, ml = k.shape[0], k.shape[2]
    cache = GpuCache(p, 2)
    if scales == "given":
        for b, s_ in enumerate(slots):
            L = lengths[b]
            cache.k_scale[s_] = k[b, :, :L].float().abs().amax(dim=(1, 2)).to(dev) / 448.0
            cache.v_scale[s_] = v[b, :, :L].float().abs().amax(dim=(1, 2)).to(dev) / 448.0
    lens = torch.tensor(lengths, dtype=torch.int32, device=dev)
    sl = torch.tensor(slots, dtype=torch.int32, device=dev)
    ws = snap.workspace(snap.snap_prefill_workspace(p, n, ml))
    out = torch.full((n, p.n_q_heads, ml, p.d_v), float("nan"), dtype=torch.bfloat16, device=dev)
    sel = torch.empty((n, p.n_kv_heads, p.topk), dtype=torch.int32, device=dev)
    pooled = torch.empty((n, p.n_kv_heads, ml), dtype=torch.float32, device=dev)
    snap.snap_prefill(p, cache.c(), cache.pos, cache.n_topk, sl, lens, q.to(dev), k.to(dev), v.to(dev), out, ws,
                      sel, pooled)
    torch.cuda.synchronize()
    _check_attention(p, lengths, q, k, v, out)
    qobs = oracle.window_queries(oracle_params(p), lengths, q)
    gsel = sel.cpu().numpy()
    if scales == "amax":
        # the scales the compression set: the oracle's data scale of the rows
        # the cache keeps (for the selection the GPU made)
        nt = cache.n_topk.cpu().numpy()
        for b, s_ in enumerate(slots):
            L = lengths[b]
            for g in range(p.n_kv_heads):
                used = gsel[b, g, :nt[s_]]
                for src, sc in ((k, cache.k_scale), (v, cache.v_scale)):
                    rows = oracle.assemble(L, p.sink, p.recent, p.topk, oracle.f64(src[b, g, :L]), used)
                    assert float(sc[s_, g]) == oracle.fp8_scale(rows), (b, g)
    st = check_compress(p, cache, qobs, k, v, lengths, slots, gsel, pooled.cpu().numpy())
    print(f"  swaps {st['swaps']}, decision band {st['decision_rel_err']:.3e}, near band {st['near_rel_err']:.3e}",
          flush=True)
    assert st["decision_rel_err"] <= DECISION_RTOL and st["near_rel_err"] <= NEAR_RTOL


def test_prefill_full_size_llama_batch_128k():
    """One layer of the 8-prompt Llama batch (72k-131k tokens) at full size, as
    `bench.py --prefill --workload llama8b-32layer-b8-128k` runs it: sampled
    output rows of sampled heads of the longest and shortest prompts against
    the oracle one by one, and the selection of two (prompt, KV head) units
    against the oracle's compression."""
    wl = synth.WORKLOADS["llama8b-32layer-b8-128k"]
    p = params_of(wl)
    lengths = synth.draw_lengths(wl, 0, wl.batch)
    n, ml = len(lengths), max(lengths)
    _announce(f"snap_prefill llama8b-32layer-b8-128k layer 0 at full size: lengths {lengths}")
    dev = "cuda"
    q, k, v = synth.prompt_batch(wl, 0, lengths, device=dev, max_len=ml, pad_value=float("nan"))
    cache = GpuCache(p, n)
    ws = snap.workspace(snap.snap_prefill_workspace(p, n, ml))
    out = torch.empty((n, p.n_q_heads, ml, p.d_v), dtype=torch.bfloat16, device=dev)
    sel = torch.empty((n, p.n_kv_heads, p.topk), dtype=torch.int32, device=dev)
    pooled = torch.empty((n, p.n_kv_heads, ml), dtype=torch.float32, device=dev)
    lens = torch.tensor(lengths, dtype=torch.int32, device=dev)
    sl = torch.arange(n, dtype=torch.int32, device=dev)
    snap.snap_prefill(p, cache.c(), cache.pos, cache.n_topk, sl, lens, q, k, v, out, ws, sel, pooled)
    torch.cuda.synchronize()
    op = oracle_params(p)
    G = op.group
    gen = np.random.default_rng(11)
    worst, worst_band, worst_near = 0.0, 0.0, 0.0
    for b in [int(np.argmax(lengths)), int(np.argmin(lengths))]:
        L = lengths[b]
        assert torch.isfinite(out[b, :, :L].float()).all()
        qc, kc, vc = oracle.f64(q[b]), oracle.f64(k[b]), oracle.f64(v[b])
        rows = sorted(set([0, 63, 64, L - 33, L - 1] + gen.integers(0, L, 3).tolist()))
        worst = max(worst, _sampled_rows(p, qc, kc, vc, out[b], L, rows, [0, 17, 31]))
        qobs = oracle.window_queries(op, [L], qc[None])
        g = int(gen.integers(0, p.n_kv_heads))
        res = oracle.compress_group(op, L, qobs[0, g * G:(g + 1) * G], kc[g, :L], vc[g, :L])
        gs = sel[b, g].cpu().numpy()
        swaps = check_selection(gs, res.P, L, p.sink, p.recent, p.topk)
        keff = min(L - p.sink - p.recent, p.topk)
        e = score_errors(pooled[b, g, p.sink:L - p.recent].double().cpu().numpy(), res.P[p.sink:L - p.recent], keff)
        worst_band = max(worst_band, e["decision"])
        worst_near = max(worst_near, e["near"])
        ek = oracle.assemble(L, p.sink, p.recent, p.topk, kc[g, :L], gs[:keff])
        assert np.array_equal(cache.k[b, g].double().cpu().numpy(), ek)
        print(f"  prompt {b} (L={L}), head {g}: swaps {swaps}, pooled-score rel err: decision band "
              f"{e['decision']:.3e}, near band {e['near']:.3e}", flush=True)
    print(f"  sampled attention max abs err {worst:.3e}", flush=True)
    assert worst_band <= DECISION_RTOL and worst_near <= NEAR_RTOL


def test_prefill_avg_pool_kernel13_explicit_scale():
    """Average pooling with the Table 6 kernel (13) and an explicit softmax
    scale, which the attention and the window statistics both take."""
    wl = synth.small(GQA, pool=synth.POOL_AVG, pool_kernel=13)
    p = params_of(wl, sm_scale=0.05)
    lengths = [950, 500]
    _announce(f"snap_prefill avg pool, kernel 13, sm_scale 0.05: lengths {lengths}")
    _run(wl, p, lengths)
