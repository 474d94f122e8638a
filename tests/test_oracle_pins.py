"""Pins of the fp64 oracle against what the paper and the mathematics fix.

None of these re-types the oracle's own loops: each compares it with the
paper's printed example or closed form, an invariant, a special case that a
textbook/library routine computes, or brute force on tiny inputs.
"""
import itertools
import math
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import NORM_CAND, NORM_ROW, POOL_AVG, POOL_MAX, Params

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
rng = np.random.default_rng(20251103)


# ---------------------------------------------------------------- ring / slot map
def _read_fixture(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                rows.append(line.split())
    return rows


def test_fig4_ring_worked_example():
    """Fig. 4 (Sec. III-B.1): L=26, one sink, recent 4 -> ring contents and the
    token replaced by the second decoded token."""
    rows = _read_fixture("fig4_ring.txt")
    kv = {r[0]: r[1:] for r in rows if r[0] in ("L", "sink", "recent")}
    L, s, r = int(kv["L"][0]), int(kv["sink"][0]), int(kv["recent"][0])
    # token t's key is the constant vector t, so a cache row names its token
    x = np.repeat(np.arange(L, dtype=np.float64)[:, None], 3, axis=1)
    cache = oracle.assemble(L, s, r, 0, x, np.zeros(0, np.int32))
    for rec in rows:
        if rec[0] == "ring":
            idx, tok = int(rec[1]), int(rec[2])
            assert cache[s + idx, 0] == tok, (idx, tok, cache[:, 0])
        if rec[0] == "replace":
            new_tok, old_tok = int(rec[1]), int(rec[2])
            row_old = int(np.where(cache[:, 0] == old_tok)[0][0])
            # decode tokens 26, 27, ... are appended in order
            for t in range(L, new_tok + 1):
                cache[oracle.slot_of(t, s, r)] = t
            assert cache[row_old, 0] == new_tok
    # sink row holds token 0
    assert cache[0, 0] == 0


@pytest.mark.parametrize("s", range(0, 6))
@pytest.mark.parametrize("r", range(1, 7))
def test_slot_map_matches_paper_closed_form(s, r):
    """Sec. III-C: L_rb = (L - L_sink + L_recent) mod L_recent + L_sink for a
    token at L >= L_sink; tokens inside the sinks stay in place."""
    for p in range(0, 60):
        got = oracle.slot_of(p, s, r)
        if p >= s:
            assert got == (p - s + r) % r + s
        else:
            assert got == p


@pytest.mark.parametrize("s,r", [(0, 1), (1, 4), (3, 5), (4, 64)])
def test_ring_keeps_exactly_last_r_tokens(s, r):
    """Decoding evicts the least recently used ring token (Sec. III-A, Case 2):
    after any number of appends the ring rows hold exactly the last r tokens."""
    for L in range(s + r, s + r + 3 * r + 2):
        x = np.arange(L, dtype=np.float64)[:, None]
        cache = oracle.assemble(L, s, r, 0, x, np.zeros(0, np.int32))
        for p in range(L, L + 2 * r + 1):
            cache[oracle.slot_of(p, s, r)] = p
            ring = sorted(int(t) for t in cache[s:s + r, 0])
            assert ring == list(range(p - r + 1, p + 1))
            assert [int(t) for t in cache[:s, 0]] == list(range(s))


def test_n_topk_counts_candidates():
    """Padding metadata (Sec. III-B.2): real top-K rows = candidates that exist, capped at K."""
    for L in range(0, 40):
        for s, r, K in [(0, 1, 5), (4, 8, 3), (2, 3, 100), (4, 64, 0)]:
            cands = [t for t in range(L) if s <= t < L - r]
            assert oracle.n_topk(L, s, r, K) == min(len(cands), K)


# ---------------------------------------------------------------- top-K
def _brute_topk(P, c0, c1, K):
    """Brute force: the unique K-subset in which every kept candidate outranks
    every dropped one under (score desc, index asc)."""
    C = list(range(c0, c1))
    keff = min(K, len(C))
    found = []
    for S in itertools.combinations(C, keff):
        Sset = set(S)
        ok = all((P[a] > P[b]) or (P[a] == P[b] and a < b)
                 for a in S for b in C if b not in Sset)
        if ok:
            found.append(list(S))
    assert len(found) == 1
    return found[0]


@pytest.mark.parametrize("trial", range(40))
def test_topk_brute_force_with_ties(trial):
    L = int(rng.integers(3, 14))
    s = int(rng.integers(0, 3))
    r = int(rng.integers(1, 3))
    K = int(rng.integers(0, 8))
    # few distinct values -> many exact ties
    P = rng.integers(0, 4, size=L).astype(np.float64)
    got = oracle.topk(L, s, r, K, P).tolist()
    exp = _brute_topk(P, s, L - r, K) if L - r > s else []
    assert got == exp


def test_topk_matches_stable_argsort():
    """Large case: equals numpy's stable argsort on (-P) then ascending order."""
    L, s, r, K = 5000, 4, 64, 300
    P = np.round(rng.random(L) * 50) / 50  # ties
    got = oracle.topk(L, s, r, K, P)
    c = np.arange(s, L - r)
    order = c[np.argsort(-P[s:L - r], kind="stable")][:K]
    assert got.tolist() == sorted(order.tolist())


def test_topk_on_many_threads_matches_one_thread():
    """The oracle runs (sequence, KV head) units on threads at once: the
    selection of every unit must equal the same unit's selection run alone
    (no state shared between concurrent rankings)."""
    from concurrent.futures import ThreadPoolExecutor
    L, s, r, K = 20000, 4, 64, 3000
    Ps = [np.round(np.random.default_rng(100 + i).random(L) * 1000) / 1000 for i in range(16)]
    alone = [oracle.topk(L, s, r, K, P) for P in Ps]
    for _ in range(3):
        with ThreadPoolExecutor(8) as ex:
            together = list(ex.map(lambda P: oracle.topk(L, s, r, K, P), Ps))
        for a, b in zip(alone, together):
            assert np.array_equal(a, b)


# ---------------------------------------------------------------- Eq. 1 & 3
def test_two_candidate_logistic_closed_form():
    """With exactly two candidates, Eq. 3's softmax is the logistic function of
    the logit difference; Eq. 1 sums it over heads and window rows.  Distinct
    query rows and asymmetric keys catch a transposed product or a wrong row."""
    G, w, D, s, r = 2, 3, 3, 2, 3
    L = s + 2 + r
    q = np.array([[[1.0, 2.0, -0.5], [0.3, -1.0, 0.8], [2.0, 0.1, 0.0]],
                  [[-1.5, 0.4, 1.0], [0.0, 0.0, 1.0], [0.7, -0.7, 0.2]]])
    k = rng.normal(size=(L, D))
    k[s] = [0.5, -1.0, 2.0]
    k[s + 1] = [2.0, 0.25, -0.5]
    scale = 0.37
    A = oracle.window_scores(G, w, D, L, s, r, NORM_CAND, scale, q, k)
    exp0 = 0.0
    for h in range(G):
        for ii in range(w):
            z0 = scale * float(q[h, ii] @ k[s])
            z1 = scale * float(q[h, ii] @ k[s + 1])
            exp0 += 1.0 / (1.0 + math.exp(z1 - z0))
    assert A[s] == pytest.approx(exp0, rel=1e-13)
    assert A[s + 1] == pytest.approx(G * w - exp0, rel=1e-13)
    assert np.all(A[:s] == 0) and np.all(A[s + 2:] == 0)


@pytest.mark.parametrize("norm", [NORM_CAND, NORM_ROW])
@pytest.mark.parametrize("w,r", [(4, 6), (8, 3), (16, 16), (5, 1)])
def test_scores_match_library_softmax(norm, w, r):
    """Eq. 1 with Eq. 3 computed by torch (fp64 matmul + masked softmax).  The
    window is the last w positions and the causal mask applies when w > r."""
    G, D, s = 3, 8, 2
    L = 40
    q = rng.normal(size=(G, w, D))
    k = rng.normal(size=(L, D)) * 1.5
    scale = 1 / math.sqrt(D)
    A = oracle.window_scores(G, w, D, L, s, r, norm, scale, q, k)
    qt, kt = torch.tensor(q), torch.tensor(k)
    z = scale * (qt @ kt.T)  # [G][w][L]
    pos = torch.arange(L - w, L)[:, None]
    j = torch.arange(L)[None, :]
    cand = (j >= s) & (j < L - r)
    dom = (j <= pos) & (cand if norm == NORM_CAND else torch.ones_like(cand))
    zm = z.masked_fill(~dom, float("-inf"))
    has = dom.any(-1, keepdim=True)
    Wt = torch.where(has, torch.softmax(zm, dim=-1), torch.zeros(()))
    Wt = Wt.nan_to_num(0.0) * (cand & (j <= pos))
    exp = Wt.sum(dim=(0, 1)).numpy()
    np.testing.assert_allclose(A, exp, rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("G,w,r", [(1, 1, 1), (4, 16, 64), (2, 8, 8)])
def test_cand_normalised_mass_is_group_times_window(G, w, r):
    """Each window row's softmax over the candidates sums to one, so with w <= r
    (every candidate causally visible) the summed attention is exactly G*w."""
    D, s, L = 16, 4, 300
    q = rng.normal(size=(G, w, D))
    k = rng.normal(size=(L, D))
    A = oracle.window_scores(G, w, D, L, s, r, NORM_CAND, 0.25, q, k)
    assert A.sum() == pytest.approx(G * w, rel=1e-12)
    assert np.all(A[:s] == 0) and np.all(A[L - r:] == 0)
    Ar = oracle.window_scores(G, w, D, L, s, r, NORM_ROW, 0.25, q, k)
    assert Ar.sum() < G * w and np.all(Ar >= 0)


def test_identical_keys_give_uniform_attention():
    G, w, D, s, r, L = 2, 4, 6, 3, 5, 50
    q = rng.normal(size=(G, w, D))
    k = np.tile(rng.normal(size=(1, D)), (L, 1))
    A = oracle.window_scores(G, w, D, L, s, r, NORM_CAND, 1.0, q, k)
    n = L - s - r
    np.testing.assert_allclose(A[s:L - r], np.full(n, G * w / n), rtol=1e-13)


def test_window_shorter_than_window_size():
    """L < w: only the L existing positions are window rows."""
    G, w, D, s, r, L = 1, 16, 4, 1, 1, 5
    q = rng.normal(size=(G, w, D))
    k = rng.normal(size=(L, D))
    A = oracle.window_scores(G, w, D, L, s, r, NORM_ROW, 1.0, q, k)
    qt, kt = torch.tensor(q[0, w - L:]), torch.tensor(k)
    z = qt @ kt.T
    causal = torch.arange(L)[None, :] <= torch.arange(L)[:, None]
    W = torch.softmax(z.masked_fill(~causal, float("-inf")), -1)
    exp = W.sum(0).numpy()
    exp[:s] = 0
    exp[L - r:] = 0
    np.testing.assert_allclose(A, exp, rtol=1e-12, atol=1e-15)


# ---------------------------------------------------------------- Eq. 2 pooling
@pytest.mark.parametrize("kp", [1, 3, 7, 13])
def test_pool_matches_library(kp):
    L, s, r = 200, 4, 16
    # scores outside the candidates are large: the pool must see candidates only
    # (sink and recent scores never leak into the first / last k//2 candidates)
    A = 100.0 + rng.random(L)
    A[s:L - r] = rng.random(L - s - r)
    Pm = oracle.pool(L, s, r, kp, POOL_MAX, A)
    Pa = oracle.pool(L, s, r, kp, POOL_AVG, A)
    a = torch.tensor(A[s:L - r])[None, None]
    em = torch.nn.functional.max_pool1d(a, kp, 1, kp // 2)[0, 0].numpy()
    ea = torch.nn.functional.avg_pool1d(a, kp, 1, kp // 2, count_include_pad=True)[0, 0].numpy()
    np.testing.assert_array_equal(Pm[s:L - r], em)
    np.testing.assert_allclose(Pa[s:L - r], ea, rtol=1e-14)
    assert np.all(Pm[s:L - r] >= A[s:L - r])
    if kp == 1:
        np.testing.assert_array_equal(Pm[s:L - r], A[s:L - r])
        np.testing.assert_allclose(Pa[s:L - r], A[s:L - r])


# ---------------------------------------------------------------- whole compression
def _params(**kw):
    base = dict(n_q_heads=4, n_kv_heads=2, d_qk=16, d_v=12, sink=3, recent=8, topk=10,
                obs_window=4, pool_kernel=3)
    base.update(kw)
    return Params(**base)


def _rand_inputs(p, L, n_seq=1):
    q = rng.normal(size=(n_seq, p.n_q_heads, p.obs_window, p.d_qk))
    k = rng.normal(size=(n_seq, p.n_kv_heads, L, p.d_qk))
    v = rng.normal(size=(n_seq, p.n_kv_heads, L, p.d_v))
    return q, k, v


def test_streaming_only_when_topk_is_zero():
    """K = 0 is plain StreamingLLM: sinks + last r tokens, no selection."""
    p = _params(topk=0)
    L = 60
    q, k, v = _rand_inputs(p, L)
    res = oracle.compress(p, [L], q, k, v)
    ck = res.cache_k[0, 1]
    assert ck.shape[0] == p.sink + p.recent
    np.testing.assert_array_equal(ck[:p.sink], k[0, 1, :p.sink])
    for t in range(L - p.recent, L):
        np.testing.assert_array_equal(ck[oracle.slot_of(t, p.sink, p.recent)], k[0, 1, t])
    assert res.n_topk[0] == 0


def test_all_candidates_kept_when_budget_covers_them():
    p = _params(topk=30)
    L = 35  # candidates [3, 27): 24 <= 30
    q, k, v = _rand_inputs(p, L)
    res = oracle.compress(p, [L], q, k, v)
    g = res.groups[0][0]
    assert g.sel.tolist() == list(range(p.sink, L - p.recent))
    s_r = p.sink + p.recent
    np.testing.assert_array_equal(res.cache_v[0, 0, s_r:s_r + 24], v[0, 0, p.sink:L - p.recent])
    assert np.all(res.cache_v[0, 0, s_r + 24:] == 0)
    assert res.n_topk[0] == 24


@pytest.mark.parametrize("L", [0, 1, 2, 3, 7, 11])
def test_short_prompt_is_plain_static_cache(L):
    """Sec. III-A Case 1 (L < L_sink + L_recent): tokens sit at their own
    positions, everything after is padding."""
    p = _params()
    q, k, v = _rand_inputs(p, max(L, 1))
    res = oracle.compress(p, [L], q, k[:, :, :max(L, 1)], v[:, :, :max(L, 1)])
    ck = res.cache_k[0, 0]
    np.testing.assert_array_equal(ck[:L], k[0, 0, :L])
    assert np.all(ck[L:] == 0)
    assert res.n_topk[0] == 0 and res.pos[0] == L


def test_last_query_argmax_when_window_and_pool_are_one():
    """w = 1, kernel 1, K = 1: the kept token is the candidate the last query
    attends to most, i.e. the argmax of its logits over the candidates."""
    p = _params(n_q_heads=1, n_kv_heads=1, obs_window=1, pool_kernel=1, topk=1)
    L = 80
    for _ in range(10):
        q, k, v = _rand_inputs(p, L)
        res = oracle.compress(p, [L], q, k, v)
        z = k[0, 0, p.sink:L - p.recent] @ q[0, 0, 0]
        assert res.groups[0][0].sel.tolist() == [p.sink + int(np.argmax(z))]


def test_invariants_of_compressed_cache():
    p = _params(topk=12, pool_kernel=5)
    L = 120
    q, k, v = _rand_inputs(p, L, n_seq=2)
    res = oracle.compress(p, [L, 90], q, k, v)
    for b, Lb in enumerate([L, 90]):
        for g in range(p.n_kv_heads):
            gr = res.groups[b][g]
            sel = gr.sel
            assert res.cache_k.shape[2] == p.budget
            assert len(sel) == len(set(sel.tolist())) == min(p.topk, Lb - p.sink - p.recent)
            assert np.all((sel >= p.sink) & (sel < Lb - p.recent))
            assert np.all(np.diff(sel) > 0)
            # every kept candidate outranks every dropped one
            cand = np.arange(p.sink, Lb - p.recent)
            dropped = np.setdiff1d(cand, sel)
            assert gr.P[sel].min() >= gr.P[dropped].max()
            np.testing.assert_array_equal(res.cache_k[b, g, :p.sink], k[b, g, :p.sink])
            for t in range(Lb - p.recent, Lb):
                np.testing.assert_array_equal(
                    res.cache_k[b, g, oracle.slot_of(t, p.sink, p.recent)], k[b, g, t])


def test_planted_heavy_hitters_are_selected():
    """Behavioural check of the whole selection on the tiny workload's inputs.
    Max pooling gives each planted heavy hitter's neighbours its score, so with
    the workload's kernel every kept token lies within kernel//2 of a planted
    key; with kernel 1 every planted key is kept (K >= number planted)."""
    import synth
    wl = synth.WORKLOADS["tiny-fp32"]
    L = wl.length
    q, k, v = synth.prefill_batch(wl, 0, [L])
    planted = np.array(sorted(synth.plant_positions(wl, 0, 0, L).tolist()))
    for kp in (wl.pool_kernel, 1):
        p = Params(wl.n_q_heads, wl.n_kv_heads, wl.d_qk, wl.d_v, wl.sink, wl.recent, wl.topk,
                   wl.obs_window, kp)
        res = oracle.compress(p, [L], q, k, v)
        for g in range(wl.n_kv_heads):
            sel = res.groups[0][g].sel
            assert len(sel) == wl.topk
            if kp == 1:
                assert set(planted.tolist()) <= set(sel.tolist())
            else:
                dist = np.abs(sel[:, None] - planted[None, :]).min(axis=1)
                assert dist.max() <= kp // 2


# ---------------------------------------------------------------- decode
def _sdpa(q, keys, vals, scale):
    """Library attention in fp64: q [G][D], keys [n][D], vals [n][Dv]."""
    qt = torch.tensor(q)[None, :, None, :]
    kt = torch.tensor(keys)[None, None].expand(1, q.shape[0], -1, -1)
    vt = torch.tensor(vals)[None, None].expand(1, q.shape[0], -1, -1)
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, scale=scale)
    return o[0, :, 0].numpy()


def test_decode_over_uncompressed_budget_is_full_attention():
    """Budget >= length: every prompt token is in the cache, so attention over
    the fresh cache equals full attention over the prompt."""
    p = _params(topk=64)
    L = 50
    q, k, v = _rand_inputs(p, L)
    res = oracle.compress(p, [L], q, k, v)
    qd = rng.normal(size=(1, p.n_q_heads, p.d_qk))
    out = oracle.decode_attn(p, [L - 1], res.n_topk, qd, res.cache_k, res.cache_v)
    G = p.group
    for g in range(p.n_kv_heads):
        exp = _sdpa(qd[0, g * G:(g + 1) * G], k[0, g], v[0, g], p.scale)
        np.testing.assert_allclose(out[0, g * G:(g + 1) * G], exp, rtol=1e-12, atol=1e-13)


def test_decode_without_wrap_is_causal_attention():
    """L + steps <= L_sink + L_recent: no eviction ever happens, so each step
    equals attention over every token so far."""
    p = _params(sink=2, recent=20, topk=5)
    L, steps = 9, 12
    q, k, v = _rand_inputs(p, L)
    res = oracle.compress(p, [L], q, k, v)
    ck, cv = res.cache_k.copy(), res.cache_v.copy()
    keys, vals = [k[0, :, :L]], [v[0, :, :L]]
    allk, allv = k[0, :, :L].copy(), v[0, :, :L].copy()
    for t in range(steps):
        pos = L + t
        kn = rng.normal(size=(1, p.n_kv_heads, p.d_qk))
        vn = rng.normal(size=(1, p.n_kv_heads, p.d_v))
        qd = rng.normal(size=(1, p.n_q_heads, p.d_qk))
        oracle.append(p, [pos], ck, cv, kn, vn)
        allk = np.concatenate([allk, kn[0][:, None]], axis=1)
        allv = np.concatenate([allv, vn[0][:, None]], axis=1)
        out = oracle.decode_attn(p, [pos], res.n_topk, qd, ck, cv)
        G = p.group
        for g in range(p.n_kv_heads):
            exp = _sdpa(qd[0, g * G:(g + 1) * G], allk[g], allv[g], p.scale)
            np.testing.assert_allclose(out[0, g * G:(g + 1) * G], exp, rtol=1e-12, atol=1e-13)


def test_ring_decode_equals_naive_sliding_window():
    """The ring buffer is an in-place version of the naive decode that rebuilds
    [sinks, last r tokens, top-K] by slicing and concatenation each step (the
    appendix's naive decode update): same rows, same attention, over 3r steps."""
    p = _params(sink=3, recent=5, topk=6)
    L = 40
    q, k, v = _rand_inputs(p, L)
    res = oracle.compress(p, [L], q, k, v)
    ck, cv = res.cache_k.copy(), res.cache_v.copy()
    s, r = p.sink, p.recent
    G = p.group
    toks_k = {t: k[0, :, t] for t in range(L)}
    toks_v = {t: v[0, :, t] for t in range(L)}
    for step in range(3 * r + 2):
        pos = L + step
        kn = rng.normal(size=(1, p.n_kv_heads, p.d_qk))
        vn = rng.normal(size=(1, p.n_kv_heads, p.d_v))
        qd = rng.normal(size=(1, p.n_q_heads, p.d_qk))
        toks_k[pos], toks_v[pos] = kn[0], vn[0]
        oracle.append(p, [pos], ck, cv, kn, vn)
        out = oracle.decode_attn(p, [pos], res.n_topk, qd, ck, cv)
        for g in range(p.n_kv_heads):
            sel = res.groups[0][g].sel.tolist()
            window = list(range(s)) + list(range(pos - r + 1, pos + 1)) + sel
            nk = np.stack([toks_k[t][g] for t in window])
            nv = np.stack([toks_v[t][g] for t in window])
            exp = _sdpa(qd[0, g * G:(g + 1) * G], nk, nv, p.scale)
            np.testing.assert_allclose(out[0, g * G:(g + 1) * G], exp, rtol=1e-12, atol=1e-13)


def test_latent_cache_values_are_key_prefix():
    """Latent (MLA) caches store one row per token; values are its first d_v dims."""
    p = _params(n_q_heads=8, n_kv_heads=1, d_qk=24, d_v=16, v_in_k=True)
    L = 70
    q = rng.normal(size=(1, 8, p.obs_window, 24))
    k = rng.normal(size=(1, 1, L, 24))
    res = oracle.compress(p, [L], q, k, None)
    assert res.cache_v is None
    qd = rng.normal(size=(1, 8, 24))
    out = oracle.decode_attn(p, [L - 1], res.n_topk, qd, res.cache_k, None)
    out2 = oracle.decode_attn(p, [L - 1], res.n_topk, qd, res.cache_k,
                              np.ascontiguousarray(res.cache_k[..., :16]))
    np.testing.assert_array_equal(out, out2)


# ---------------------------------------------------------------- fp8 E4M3
def test_e4m3_values_match_library():
    codes = torch.arange(256, dtype=torch.uint8)
    lib = codes.view(torch.float8_e4m3fn).to(torch.float64).numpy()
    mine = np.array([oracle.e4m3_value(c) for c in range(256)])
    nan = np.isnan(lib)
    assert np.array_equal(nan, np.isnan(mine))
    np.testing.assert_array_equal(mine[~nan], lib[~nan])


def test_e4m3_encode_matches_library_cast():
    """Round-to-nearest-even, saturating: equals torch's cast after clamping to
    +-448, on every code value, every midpoint and random values."""
    vals = np.array([oracle.e4m3_value(c) for c in range(256)])
    vals = vals[~np.isnan(vals)]
    pos = np.unique(np.abs(vals))
    mids = (pos[1:] + pos[:-1]) / 2
    xs = np.concatenate([vals, mids, -mids, rng.normal(size=2000) * 50,
                         rng.normal(size=500) * 1e-3, [500.0, -1e4, 447.9, 464.0, 1e-12]])
    xs = xs.astype(np.float32)
    lib = torch.tensor(np.clip(xs, -448, 448)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    mine = np.array([oracle.e4m3_encode(float(x)) for x in xs], np.uint8)
    # torch keeps the sign of zero; so does the encoder
    np.testing.assert_array_equal(mine, lib)


def test_quantize_uses_fp32_quotient():
    x = rng.normal(size=300).astype(np.float32).astype(np.float64)
    scale = np.float32(0.0123)
    codes = oracle.quantize(x, float(scale))
    q32 = (x.astype(np.float32) / scale).astype(np.float32)
    lib = torch.tensor(np.clip(q32, -448, 448)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    np.testing.assert_array_equal(codes, lib)


def test_fp8_scale_from_data():
    """The data-chosen scale puts the largest magnitude on the top E4M3 code
    (448) and nothing beyond it; with a largest magnitude of exactly 448 it is
    1 and the codes are torch's plain cast; all-zero data gets scale 1."""
    assert oracle.fp8_scale(np.zeros(7)) == 1.0
    for trial in range(20):
        x = rng.normal(size=500) * 10 ** rng.uniform(-3, 3)
        x = x.astype(np.float32).astype(np.float64)
        sc = oracle.fp8_scale(x)
        codes = oracle.quantize(x, sc)
        i = int(np.argmax(np.abs(x)))
        assert codes[i] == (0xFE if x[i] < 0 else 0x7E), trial
        # nothing saturates: every quotient is within 448, the largest on it
        quo = np.abs(x.astype(np.float32) / np.float32(sc))
        assert np.all(quo <= 448.0 * (1 + 2.0 ** -22)), trial
        assert abs(quo[i] - 448.0) <= 448.0 * 2.0 ** -22, trial
    x = rng.normal(size=400).astype(np.float32).astype(np.float64)
    x = x / np.max(np.abs(x)) * 448.0
    x[3] = -448.0
    x = x.astype(np.float32).astype(np.float64)
    assert oracle.fp8_scale(x) == 1.0
    lib = torch.tensor(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    np.testing.assert_array_equal(oracle.quantize(x, 1.0), lib)


# ---------------------------------------------------------------- prefill attention
def _prefill_case(G=3, L=37, dk=8, dv=6, scale=0.41, seed=7):
    r = np.random.default_rng(seed)
    p = Params(n_q_heads=G, n_kv_heads=1, d_qk=dk, d_v=dv, sink=2, recent=4, topk=5, obs_window=4,
               pool_kernel=3, sm_scale=scale)
    q = r.standard_normal((G, L, dk))
    k = r.standard_normal((L, dk))
    v = r.standard_normal((L, dv))
    return p, q, k, v


def test_prefill_attn_matches_library_sdpa():
    """Causal attention of the prefill graph (Sec. IV-A, MHA kernel) against
    torch's scaled_dot_product_attention in fp64 (the G heads share K and V),
    and the rows' normalisers against torch.logsumexp of the masked logits."""
    p, q, k, v = _prefill_case()
    G, L = q.shape[0], q.shape[1]
    out, lse = oracle.prefill_attn_group(p, L, q, k, v, want_lse=True)
    qt, kt, vt = (torch.from_numpy(x) for x in (q, k, v))
    ref = torch.nn.functional.scaled_dot_product_attention(
        qt[None], kt[None, None].expand(1, G, L, -1), vt[None, None].expand(1, G, L, -1), is_causal=True,
        scale=p.sm_scale)[0]
    np.testing.assert_allclose(out, ref.numpy(), rtol=1e-12, atol=1e-12)
    z = p.sm_scale * torch.einsum("hid,jd->hij", qt, kt)
    z = z.masked_fill(torch.ones(L, L, dtype=torch.bool).triu(1), float("-inf"))
    np.testing.assert_allclose(lse, torch.logsumexp(z, dim=-1).numpy(), rtol=1e-12, atol=1e-12)


def test_prefill_first_row_and_equal_keys():
    """Position 0 sees only itself: its output is v_0 exactly.  With every key
    equal the softmax is uniform over the causal prefix: out_i is the mean of
    v_0..v_i and the normaliser is z + log(i+1)."""
    p, q, k, v = _prefill_case(L=23)
    G, L = q.shape[0], q.shape[1]
    out = oracle.prefill_attn_group(p, L, q, k, v)
    for h in range(G):
        assert np.array_equal(out[h, 0], v[0])
    k_eq = np.repeat(k[:1], L, axis=0)
    out, lse = oracle.prefill_attn_group(p, L, q, k_eq, v, want_lse=True)
    means = np.cumsum(v, axis=0) / np.arange(1, L + 1)[:, None]
    for h in range(G):
        np.testing.assert_allclose(out[h], means, rtol=1e-12, atol=1e-12)
        z = p.sm_scale * (q[h] @ k[0])
        np.testing.assert_allclose(lse[h], z + np.log(np.arange(1, L + 1)), rtol=1e-12, atol=1e-12)


def test_prefill_dominant_key_selects_its_value():
    """A key far more aligned with every query than the rest (logit gap > 50)
    takes all the weight of every row that can see it; rows before it average
    only what precedes them."""
    p, q, k, v = _prefill_case(L=30, scale=1.0)
    G, L = q.shape[0], q.shape[1]
    j0 = 11
    k2 = k * 0.01
    k2[j0] = 0.0
    q2 = np.repeat(np.eye(p.d_qk)[:1][None], G, axis=0).repeat(L, axis=1) * 1.0
    k2[j0, 0] = 60.0
    out = oracle.prefill_attn_group(p, L, q2, k2, v)
    for h in range(G):
        np.testing.assert_allclose(out[h, j0:], np.repeat(v[j0:j0 + 1], L - j0, axis=0), atol=1e-20, rtol=1e-12)
        assert not np.allclose(out[h, j0 - 1], v[j0])


def test_window_queries_are_the_last_w_positions():
    """Sec. III-B.2: Q_obs holds the queries of the last L_obs prompt tokens;
    row w-1 is position L-1, and rows before position 0 are empty."""
    p = Params(n_q_heads=2, n_kv_heads=1, d_qk=3, d_v=3, sink=1, recent=2, topk=1, obs_window=4, pool_kernel=1)
    q = np.arange(2 * 9 * 3, dtype=np.float64).reshape(1, 2, 9, 3)
    got = oracle.window_queries(p, [9], q)
    assert np.array_equal(got[0], q[0, :, 5:9])
    got = oracle.window_queries(p, [2], q)
    assert np.array_equal(got[0, :, 2:], q[0, :, 0:2]) and not got[0, :, :2].any()


def test_prefill_row_range_matches_whole_prompt():
    """A range of query rows (as the full-size tests sample them) equals the
    same rows of the whole-prompt attention, against the library routine."""
    p, q, k, v = _prefill_case(L=41)
    G, L = q.shape[0], q.shape[1]
    qt, kt, vt = (torch.from_numpy(x) for x in (q, k, v))
    ref = torch.nn.functional.scaled_dot_product_attention(
        qt[None], kt[None, None].expand(1, G, L, -1), vt[None, None].expand(1, G, L, -1), is_causal=True,
        scale=p.sm_scale)[0].numpy()
    for i0, i1 in [(0, 1), (5, 9), (17, 41), (40, 41)]:
        out = oracle.prefill_attn_group(p, L, q, k, v, rows=(i0, i1))
        np.testing.assert_allclose(out, ref[:, i0:i1], rtol=1e-12, atol=1e-12)
