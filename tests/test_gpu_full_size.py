"""GPU parity at the benchmark's full sizes, in the launch configuration
bench.py times: one layer of the 128k workloads (all sequences compressed in
one call).  The fp64 oracle recomputes sampled (sequence, KV head) units one
by one; every unit is checked for the properties that hold at any size, and
decode outputs are recomputed by the oracle on the GPU's own cache bytes.
"""
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle
import paper_2511_03092_amd as snap
import synth
from snaphelp import (DECISION_RTOL, NEAR_RTOL, SEL_RTOL, TOL, GpuCache, check_selection, oracle_params, params_of,
                      score_errors)

pytestmark = pytest.mark.gpu


def _announce(msg):
    print(f"\n[case] {msg}", flush=True)


def _compress_full(wl, lengths):
    """Inputs generated on the GPU (as bench.py does), one compress call."""
    p = params_of(wl)
    dev = "cuda"
    max_len = max(lengths)
    q, k, v = synth.prefill_batch(wl, 0, lengths, device=dev, max_len=max_len, pad_value=float("nan"))
    cache = GpuCache(p, len(lengths))
    n = len(lengths)
    lens = torch.tensor(lengths, dtype=torch.int32, device=dev)
    sl = torch.arange(n, dtype=torch.int32, device=dev)
    ws = snap.workspace(snap.snap_compress_workspace(p, n, max_len))
    sel = torch.empty((n, p.n_kv_heads, p.topk), dtype=torch.int32, device=dev)
    pooled = torch.empty((n, p.n_kv_heads, max_len), dtype=torch.float32, device=dev)
    snap.snap_compress(p, cache.c(), cache.pos, cache.n_topk, sl, lens, q, k, v, ws, sel, pooled)
    torch.cuda.synchronize()
    return p, q, k, v, cache, sel, pooled


def _structural(p, k, v, cache, sel, pooled, lengths):
    """Properties every unit must satisfy, checked on the GPU's own data."""
    s, r, K = p.sink, p.recent, p.topk
    pos = cache.pos.cpu().tolist()
    nt = cache.n_topk.cpu().tolist()
    for b, L in enumerate(lengths):
        keff = min(max(L - s - r, 0), K)
        assert pos[b] == L and nt[b] == keff
        for g in range(p.n_kv_heads):
            S = sel[b, g]
            kept = S[:keff]
            assert torch.all(S[keff:] == -1)
            assert torch.all(kept[1:] > kept[:-1]) and int(kept[0]) >= s and int(kept[-1]) < L - r
            src = torch.cat([torch.arange(min(s, L), device="cuda"),
                             torch.arange(max(s, L - r), L, device="cuda"), kept.long()])
            rows = torch.cat([torch.arange(min(s, L), device="cuda"),
                              torch.tensor([oracle.slot_of(t, s, r) for t in range(max(s, L - r), L)],
                                           device="cuda", dtype=torch.long),
                              s + r + torch.arange(keff, device="cuda")])
            ck = cache.k[b, g]
            assert torch.equal(ck[rows].view(torch.int16), k[b, g, src].view(torch.int16)), (b, g)
            assert torch.all(ck[s + r + keff:] == 0)
            if v is not None:
                assert torch.equal(cache.v[b, g][rows].view(torch.int16), v[b, g, src].view(torch.int16))
            P = pooled[b, g]
            assert torch.all(torch.isnan(P[:s])) and torch.all(torch.isnan(P[L - r:L]))
            assert torch.all(P[s:L - r] >= 0)


def _oracle_units(p, q, k, v, cache, sel, pooled, lengths, units):
    op = oracle_params(p)
    G = op.group

    def run(u):
        b, g = u
        L = lengths[b]
        res = oracle.compress_group(op, L, oracle.f64(q[b, g * G:(g + 1) * G]), oracle.f64(k[b, g, :L]),
                                    None if v is None else oracle.f64(v[b, g, :L]))
        return u, res

    with ThreadPoolExecutor(len(units)) as ex:
        results = list(ex.map(run, units))
    worst_dec, worst_near = 0.0, 0.0
    for (b, g), res in results:
        L = lengths[b]
        s, r = p.sink, p.recent
        gs = sel[b, g].cpu().numpy()
        swaps = check_selection(gs, res.P, L, s, r, p.topk, SEL_RTOL)
        keff = min(max(L - s - r, 0), p.topk)
        ek = oracle.assemble(L, s, r, p.topk, oracle.f64(k[b, g, :L]), gs[:keff])
        assert np.array_equal(cache.k[b, g].double().cpu().numpy(), ek)
        e = score_errors(pooled[b, g, s:L - r].double().cpu().numpy(), res.P[s:L - r], keff)
        worst_dec, worst_near = max(worst_dec, e["decision"]), max(worst_near, e["near"])
        print(f"  unit (seq {b}, head {g}, L={L}): swaps {swaps}, pooled-score rel err: decision band "
              f"{e['decision']:.3e}, near band {e['near']:.3e}", flush=True)
    assert worst_dec <= DECISION_RTOL and worst_near <= NEAR_RTOL


def _decode_check(p, wl, cache, steps, check_slots):
    n = cache.n_slots
    sl = torch.arange(n, dtype=torch.int32, device="cuda")
    ws = snap.workspace(snap.snap_decode_workspace(p, n))
    out = torch.empty((n, p.n_q_heads, p.d_v), dtype=torch.bfloat16, device="cuda")
    op = oracle_params(p)
    worst = 0.0
    for step in range(steps):
        positions = cache.pos.cpu().tolist()
        qd, kn, vn = synth.decode_inputs(wl, 0, step, positions, device="cuda")
        snap.snap_cache_append(p, cache.c(), cache.pos, sl, kn, vn)
        snap.snap_decode_attn(p, cache.c(), cache.pos, cache.n_topk, sl, qd, out, ws)
        snap.snap_advance(cache.pos, sl)
        torch.cuda.synchronize()
        nt = cache.n_topk.cpu().numpy()
        for b in check_slots:
            ck = cache.k[b:b + 1].double().cpu().numpy()
            cv = None if cache.v is None else cache.v[b:b + 1].double().cpu().numpy()
            exp = oracle.decode_attn(op, [positions[b]], nt[[b]], qd[b:b + 1].cpu(), ck, cv)
            err = float(np.max(np.abs(out[b:b + 1].double().cpu().numpy() - exp)))
            worst = max(worst, err)
            assert err <= TOL["bf16"], (step, b, err)
    print(f"  decode max abs err: {worst:.3e}", flush=True)


def test_llama_32layer_workload_one_layer_full_size():
    wl = synth.WORKLOADS["llama8b-32layer-b8-128k"]
    lengths = synth.draw_lengths(wl, 0, wl.batch)
    _announce(f"llama8b-32layer-b8-128k layer 0 at full size, lengths {lengths}")
    p, q, k, v, cache, sel, pooled = _compress_full(wl, lengths)
    _structural(p, k, v, cache, sel, pooled, lengths)
    big = int(np.argmax(lengths))
    small = int(np.argmin(lengths))
    _oracle_units(p, q, k, v, cache, sel, pooled, lengths, [(big, 0), (small, 7), (3, 4)])
    _decode_check(p, wl, cache, 2, list(range(wl.batch)))


def test_mla_workload_one_layer_full_size():
    wl = synth.WORKLOADS["mla-8head-61layer-b16-128k"]
    lengths = synth.draw_lengths(wl, 0, wl.batch)
    _announce(f"mla-8head-61layer-b16-128k layer 0 at full size: {wl.batch} x {lengths[0]}")
    p, q, k, v, cache, sel, pooled = _compress_full(wl, lengths)
    _structural(p, k, v, cache, sel, pooled, lengths)
    _oracle_units(p, q, k, v, cache, sel, pooled, lengths, [(0, 0), (5, 0), (15, 0)])
    _decode_check(p, wl, cache, 4, [0, 5, 15])


def test_cb_fp8_workload_full_size():
    """The continuous-batching shape: 8 prompts of the workload's length mix
    (4k-128k) compressed into 8 of the 32 fp8 slots, per-(slot, head) scales
    = amax / 448.  Every unit: metadata, index-set structure, zero padding.
    Sampled units: selection and every fp8 code against the oracle's
    quantisation of the oracle's assembly.  Then two fused decode steps,
    checked against the oracle on the GPU's cache bytes for three slots."""
    wl = synth.WORKLOADS["cb-fp8-llama8b-32slot"]
    slots = [3, 17, 0, 31, 8, 22, 12, 5]
    lengths = synth.draw_lengths(wl, 0, len(slots))
    _announce(f"cb-fp8-llama8b-32slot at full size: lengths {lengths} into slots {slots} of {wl.slots}")
    p = params_of(wl)
    s, r, K = p.sink, p.recent, p.topk
    max_len = max(lengths)
    q, k, v = synth.prefill_batch(wl, 0, lengths, device="cuda", max_len=max_len, pad_value=float("nan"),
                                  slots=slots)
    cache = GpuCache(p, wl.slots)
    for b, s_ in enumerate(slots):
        L = lengths[b]
        cache.k_scale[s_] = k[b, :, :L].float().abs().amax(dim=(1, 2)).clamp_min(1e-6) / 448.0
        cache.v_scale[s_] = v[b, :, :L].float().abs().amax(dim=(1, 2)).clamp_min(1e-6) / 448.0
    n = len(slots)
    sl = torch.tensor(slots, dtype=torch.int32, device="cuda")
    lens = torch.tensor(lengths, dtype=torch.int32, device="cuda")
    ws = snap.workspace(snap.snap_compress_workspace(p, n, max_len))
    sel = torch.empty((n, p.n_kv_heads, K), dtype=torch.int32, device="cuda")
    pooled = torch.empty((n, p.n_kv_heads, max_len), dtype=torch.float32, device="cuda")
    snap.snap_compress(p, cache.c(), cache.pos, cache.n_topk, sl, lens, q, k, v, ws, sel, pooled)
    torch.cuda.synchronize()

    pos, nt = cache.pos.cpu().tolist(), cache.n_topk.cpu().tolist()
    for b, L in enumerate(lengths):
        keff = min(max(L - s - r, 0), K)
        assert pos[slots[b]] == L and nt[slots[b]] == keff
        S = sel[b]
        assert torch.all(S[:, keff:] == -1)
        assert torch.all(S[:, 1:keff] > S[:, :keff - 1]) and int(S[:, :keff].min()) >= s
        assert int(S[:, :keff].max()) < L - r
        assert torch.all(cache.k[slots[b], :, s + r + keff:] == 0)
        assert torch.all(cache.v[slots[b], :, s + r + keff:] == 0)
    untouched = [x for x in range(wl.slots) if x not in slots]
    cache.assert_untouched(untouched)

    op = oracle_params(p)
    G = op.group
    units = [(int(np.argmax(lengths)), 0), (int(np.argmin(lengths)), 7), (2, 3)]

    def run(u):
        b, g = u
        L = lengths[b]
        return u, oracle.compress_group(op, L, oracle.f64(q[b, g * G:(g + 1) * G]), oracle.f64(k[b, g, :L]),
                                        oracle.f64(v[b, g, :L]))

    with ThreadPoolExecutor(len(units)) as ex:
        results = list(ex.map(run, units))
    worst_dec, worst_near = 0.0, 0.0
    for (b, g), res in results:
        L, s_ = lengths[b], slots[b]
        keff = min(max(L - s - r, 0), K)
        gs = sel[b, g].cpu().numpy()
        swaps = check_selection(gs, res.P, L, s, r, K, SEL_RTOL)
        for src, dst, sc in ((k, cache.k, cache.k_scale), (v, cache.v, cache.v_scale)):
            rows = oracle.assemble(L, s, r, K, oracle.f64(src[b, g, :L]), gs[:keff])
            codes = oracle.quantize(rows, float(sc[s_, g])).reshape(rows.shape)
            assert np.array_equal(dst[s_, g].cpu().numpy(), codes), (b, g)
        c = slice(s, L - r)
        e = score_errors(pooled[b, g, c].double().cpu().numpy(), res.P[c], keff)
        worst_dec, worst_near = max(worst_dec, e["decision"]), max(worst_near, e["near"])
        print(f"  unit (seq {b} -> slot {s_}, head {g}, L={L}): swaps {swaps}, pooled-score rel err: decision band "
              f"{e['decision']:.3e}, near band {e['near']:.3e}", flush=True)
    assert worst_dec <= DECISION_RTOL and worst_near <= NEAR_RTOL

    dws = snap.workspace(snap.snap_decode_workspace(p, n))
    out = torch.empty((n, p.n_q_heads, p.d_v), dtype=torch.bfloat16, device="cuda")
    worst = 0.0
    for step in range(2):
        positions = cache.pos[sl.long()].cpu().tolist()
        qd, kn, vn = synth.decode_inputs(wl, 0, step, positions, device="cuda")
        snap.snap_decode_step(p, cache.c(), cache.pos, cache.n_topk, sl, qd, kn, vn, out, dws)
        snap.snap_advance(cache.pos, sl)
        torch.cuda.synchronize()
        ntv = cache.n_topk.cpu().numpy()
        for i in (0, 3, 6):
            s_ = slots[i]
            table = torch.tensor([oracle.e4m3_value(x) for x in range(256)], dtype=torch.float64)
            ck = (table[cache.k[s_].cpu().long()] * cache.k_scale[s_].cpu().double()[:, None, None]).numpy()
            cv = (table[cache.v[s_].cpu().long()] * cache.v_scale[s_].cpu().double()[:, None, None]).numpy()
            exp = oracle.decode_attn(op, [positions[i]], ntv[[s_]], qd[i:i + 1].cpu(), ck[None], cv[None])
            err = float(np.max(np.abs(out[i:i + 1].double().cpu().numpy() - exp)))
            worst = max(worst, err)
            assert err <= TOL["fp8"], (step, s_, err)
    print(f"  decode max abs err: {worst:.3e}", flush=True)
