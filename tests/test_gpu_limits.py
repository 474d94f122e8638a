"""Launches at the ABI's largest accepted batch: snap_compress with
n_seq * n_kv_heads = 65535 and snap_decode_step with n * n_q_heads = 65535
(one more is refused on the host, tests/test_abi.py).  13107 short prompts of
5 KV heads each (one query head per KV head), d = 64 (the generic decode
kernel) and d = 128 (the MFMA decode kernel).  Every sequence's metadata is
checked, and sampled sequences (the first, the last and 48 drawn at random)
against the oracle: the kept set (Eq. 2's swap rule), the cache bytes
(Sec. III-A), the appended row and the decode output (Sec. III-C).

Every case prints what names it before touching the GPU.
"""
import random

import numpy as np
import pytest
import torch

import oracle
import paper_2511_03092_amd as snap
import synth
from snaphelp import GpuCache, check_selection, expected_cache, gpu_compress, oracle_params, params_of

pytestmark = pytest.mark.gpu

N_SEQ, HKV = 13107, 5  # 65535 (sequence, KV head) groups and (sequence, query head) pairs
assert N_SEQ * HKV == 65535


def _wl(d):
    return synth.Workload(f"limits-d{d}", 15, HKV, HKV, d, d, False, 4, 8, 8, 4, 3, "bf16", "bf16", layers=1,
                          batch=N_SEQ, length=None, length_range=(8, 40), decode_steps=1, rope=False,
                          plant_frac=0.0)


@pytest.mark.parametrize("d", [64, 128])
def test_largest_accepted_batch(d):
    wl = _wl(d)
    p = params_of(wl)
    op = oracle_params(p)
    s, r, K = p.sink, p.recent, p.topk
    print(f"\n[case] {N_SEQ} sequences x {HKV} KV heads, d={d}, L in {wl.length_range}", flush=True)
    lengths = synth.draw_lengths(wl, 0, N_SEQ)
    q, k, v = synth.prefill_batch(wl, 0, lengths)
    cache = GpuCache(p, N_SEQ)
    gsel, _ = gpu_compress(p, cache, q, k, v, lengths, list(range(N_SEQ)), debug=True)

    want_nt = [oracle.n_topk(L, s, r, K) for L in lengths]
    assert cache.pos.cpu().tolist() == lengths
    assert cache.n_topk.cpu().tolist() == want_nt

    rng = random.Random(65535 + d)
    sample = sorted({0, N_SEQ - 1, *rng.sample(range(N_SEQ), 48)})
    ck = cache.k.cpu()
    cv = cache.v.cpu()
    for b in sample:
        L = lengths[b]
        res = oracle.compress(op, [L], q[b:b + 1], k[b:b + 1], v[b:b + 1], threads=1)
        for g in range(HKV):
            check_selection(gsel[b, g], res.groups[0][g].P, L, s, r, K)
            keff = want_nt[b]
            ek = expected_cache(L, s, r, K, oracle.f64(k[b, g]), gsel[b, g][:keff])
            ev = expected_cache(L, s, r, K, oracle.f64(v[b, g]), gsel[b, g][:keff])
            assert np.array_equal(ck[b, g].double().numpy(), ek), (b, g)
            assert np.array_equal(cv[b, g].double().numpy(), ev), (b, g)

    # one decode step of every sequence (append at pos, attend, advance)
    qd, kn, vn = synth.decode_inputs(wl, 0, 0, lengths, device="cuda")
    ws = snap.workspace(snap.snap_decode_workspace(p, N_SEQ))
    out = torch.zeros((N_SEQ, p.n_q_heads, p.d_v), dtype=torch.bfloat16, device="cuda")
    sl = torch.arange(N_SEQ, dtype=torch.int32, device="cuda")
    snap.snap_decode_step(p, cache.c(), cache.pos, cache.n_topk, sl, qd, kn, vn, out, ws)
    snap.snap_advance(cache.pos, sl)
    torch.cuda.synchronize()
    assert cache.pos.cpu().tolist() == [L + 1 for L in lengths]
    ck = cache.k.cpu()
    cv = cache.v.cpu()
    o = out.cpu().double().numpy()
    qh, knh, vnh = qd.cpu(), kn.cpu(), vn.cpu()
    worst = 0.0
    for b in sample:
        L = lengths[b]
        row = oracle.slot_of(L, s, r)
        for g in range(HKV):
            assert torch.equal(ck[b, g, row].view(torch.int16), knh[b, g].view(torch.int16)), (b, g)
            assert torch.equal(cv[b, g, row].view(torch.int16), vnh[b, g].view(torch.int16)), (b, g)
            exp = oracle.decode_attn_group(op, L, want_nt[b], oracle.f64(qh[b, g:g + 1]),
                                           ck[b, g].double().numpy(), cv[b, g].double().numpy())
            worst = max(worst, float(np.abs(o[b, g:g + 1] - exp).max()))
    print(f"decode max abs err over {len(sample)} sampled sequences: {worst:.3e}", flush=True)
    assert worst <= 2e-2
