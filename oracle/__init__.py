"""fp64 CPU oracle of the SnapStream hot path -- TEST INFRASTRUCTURE ONLY.

Thin ctypes wrapper around ``oracle.c`` (plain C, fp64).  Only tests, the
smoke check and the benchmark's CPU-baseline leg may import this package; the
HIP library never does, and the two share no code.

Array conventions (numpy, float64 unless stated):
  q_obs : [n_seq][Hq][w][dk]    (row w-1 is the last prompt token, position L-1)
  k     : [n_seq][Hkv][Lmax][k_width]
  v     : [n_seq][Hkv][Lmax][dv] or None (latent cache: V = first dv dims of K)
  cache : [n_seq][Hkv][B][width] with B = sink + recent + topk
"""
from __future__ import annotations

import ctypes
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# SNAP_ORACLE_LIB names another build of oracle.c (the mutation tests load
# deliberately broken copies this way); by default the in-tree library
_LIB_PATH = os.environ.get("SNAP_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")
_lib = None

POOL_MAX, POOL_AVG = 0, 1
NORM_CAND, NORM_ROW = 0, 1

_dp = ctypes.POINTER(ctypes.c_double)
_ip = ctypes.POINTER(ctypes.c_int32)
_u8p = ctypes.POINTER(ctypes.c_uint8)


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b
        _b.build()
    lib = ctypes.CDLL(_LIB_PATH)
    i64, i32, dbl = ctypes.c_int64, ctypes.c_int, ctypes.c_double
    lib.oracle_slot_of.argtypes = [i64, i32, i32]
    lib.oracle_slot_of.restype = i32
    lib.oracle_n_topk.argtypes = [i64, i32, i32, i32]
    lib.oracle_n_topk.restype = i32
    lib.oracle_window_scores.argtypes = [i32, i32, i32, i64, i32, i32, i32, dbl, _dp, _dp, _dp]
    lib.oracle_window_scores.restype = None
    lib.oracle_pool.argtypes = [i64, i32, i32, i32, i32, _dp, _dp]
    lib.oracle_pool.restype = None
    lib.oracle_topk.argtypes = [i64, i32, i32, i32, _dp, _ip]
    lib.oracle_topk.restype = i32
    lib.oracle_assemble.argtypes = [i64, i32, i32, i32, i32, _dp, _ip, i32, _dp]
    lib.oracle_assemble.restype = None
    lib.oracle_compress_group.argtypes = [i32, i32, i32, i32, i64, i32, i32, i32, i32, i32, i32,
                                          dbl, _dp, _dp, _dp, _dp, _dp, _ip, _dp, _dp]
    lib.oracle_compress_group.restype = i32
    lib.oracle_decode_attn.argtypes = [i32, i32, i32, i32, i32, i32, i32, i64, i32, dbl,
                                       _dp, _dp, _dp, _dp]
    lib.oracle_decode_attn.restype = None
    lib.oracle_prefill_attn.argtypes = [i32, i32, i32, i64, i64, i64, dbl, _dp, _dp, _dp, _dp, _dp]
    lib.oracle_prefill_attn.restype = None
    lib.oracle_e4m3_value.argtypes = [ctypes.c_uint8]
    lib.oracle_e4m3_value.restype = dbl
    lib.oracle_e4m3_encode.argtypes = [ctypes.c_float]
    lib.oracle_e4m3_encode.restype = ctypes.c_uint8
    lib.oracle_quantize.argtypes = [_dp, i64, ctypes.c_float, _u8p]
    lib.oracle_quantize.restype = None
    lib.oracle_fp8_scale.argtypes = [_dp, i64]
    lib.oracle_fp8_scale.restype = ctypes.c_float
    _lib = lib
    return lib


def _d(a: np.ndarray):
    assert a.dtype == np.float64 and a.flags.c_contiguous
    return a.ctypes.data_as(_dp)


def _i(a: np.ndarray):
    assert a.dtype == np.int32 and a.flags.c_contiguous
    return a.ctypes.data_as(_ip)


def f64(x) -> np.ndarray:
    """Exact conversion of a torch tensor / array of any float dtype to fp64."""
    try:
        import torch
        if isinstance(x, torch.Tensor):
            return np.ascontiguousarray(x.detach().to("cpu", torch.float64).numpy())
    except ImportError:  # pragma: no cover
        pass
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


@dataclass
class Params:
    """The method's hyper-parameters (names follow the paper's notation)."""
    n_q_heads: int
    n_kv_heads: int
    d_qk: int
    d_v: int
    sink: int
    recent: int
    topk: int
    obs_window: int
    pool_kernel: int
    pool: int = POOL_MAX
    norm: int = NORM_CAND
    v_in_k: bool = False
    sm_scale: float = 0.0

    @property
    def budget(self) -> int:
        return self.sink + self.recent + self.topk

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def scale(self) -> float:
        return self.sm_scale if self.sm_scale > 0 else 1.0 / np.sqrt(self.d_qk)


def slot_of(p: int, s: int, r: int) -> int:
    return int(_load().oracle_slot_of(int(p), int(s), int(r)))


def n_topk(L: int, s: int, r: int, K: int) -> int:
    return int(_load().oracle_n_topk(int(L), int(s), int(r), int(K)))


def window_scores(G, w, D, L, s, r, norm, sm_scale, q, k) -> np.ndarray:
    """A[j] for one group. q: [G][w][D], k: [>=L][D]."""
    q = np.ascontiguousarray(q, dtype=np.float64)
    k = np.ascontiguousarray(k[:L], dtype=np.float64)
    A = np.zeros(L, np.float64)
    _load().oracle_window_scores(G, w, D, L, s, r, norm, float(sm_scale), _d(q), _d(k), _d(A))
    return A


def pool(L, s, r, kp, pool_type, A) -> np.ndarray:
    A = np.ascontiguousarray(A, dtype=np.float64)
    P = np.zeros(L, np.float64)
    _load().oracle_pool(L, s, r, kp, pool_type, _d(A), _d(P))
    return P


def topk(L, s, r, K, P) -> np.ndarray:
    P = np.ascontiguousarray(P, dtype=np.float64)
    sel = np.full(max(K, 1), -1, np.int32)
    keff = _load().oracle_topk(L, s, r, K, _d(P), _i(sel))
    return sel[:keff].copy()


def assemble(L, s, r, K, x, sel) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float64)
    sel = np.ascontiguousarray(sel, dtype=np.int32)
    width = x.shape[-1]
    out = np.zeros((s + r + K, width), np.float64)
    _load().oracle_assemble(L, s, r, K, width, _d(x), _i(sel) if sel.size else _i(np.zeros(1, np.int32)),
                            int(sel.size), _d(out))
    return out


@dataclass
class GroupResult:
    A: np.ndarray       # [L] summed window attention on the candidates
    P: np.ndarray       # [L] pooled scores on the candidates
    sel: np.ndarray     # [keff] selected token indices, ascending
    cache_k: np.ndarray  # [B][k_width]
    cache_v: np.ndarray | None  # [B][dv]


def compress_group(p: Params, L: int, q, k, v) -> GroupResult:
    """Compression of one (sequence, KV head): q [G][w][dk], k [>=L][k_width], v [>=L][dv] or None."""
    lib = _load()
    q = np.ascontiguousarray(q, dtype=np.float64)
    kw = k.shape[-1]
    k = np.ascontiguousarray(k[:L], dtype=np.float64)
    vv = None if v is None else np.ascontiguousarray(v[:L], dtype=np.float64)
    B = p.budget
    A = np.zeros(max(L, 1), np.float64)
    P = np.zeros(max(L, 1), np.float64)
    sel = np.full(max(p.topk, 1), -1, np.int32)
    ck = np.zeros((B, kw), np.float64)
    cv = None if vv is None else np.zeros((B, p.d_v), np.float64)
    if L == 0:
        return GroupResult(A[:0], P[:0], sel[:0], ck, cv)
    # The score pass reads the first d_qk dims of each stored K row.
    assert kw == p.d_qk
    keff = lib.oracle_compress_group(
        p.group, p.obs_window, p.d_qk, p.d_v, L, p.sink, p.recent, p.topk, p.pool_kernel,
        p.pool, p.norm, float(p.scale), _d(q), _d(k), _d(vv) if vv is not None else None,
        _d(A), _d(P), _i(sel), _d(ck), _d(cv) if cv is not None else None)
    return GroupResult(A[:L], P[:L], sel[:keff].copy(), ck, cv)


@dataclass
class CompressResult:
    groups: list        # [n_seq][Hkv] GroupResult
    cache_k: np.ndarray  # [n_seq][Hkv][B][k_width]
    cache_v: np.ndarray | None
    n_topk: np.ndarray  # [n_seq]
    pos: np.ndarray     # [n_seq]


def compress(p: Params, lengths, q_obs, k, v=None, threads: int | None = None) -> CompressResult:
    """Compression of a padded batch; independent (seq, head) units run in threads
    (ctypes releases the GIL, each unit is the single-threaded C routine)."""
    q_obs = f64(q_obs)
    k = f64(k)
    v = None if v is None else f64(v)
    n_seq, Hkv = k.shape[0], k.shape[1]
    G = p.group
    units = [(b, g) for b in range(n_seq) for g in range(Hkv)]

    def run(u):
        b, g = u
        L = int(lengths[b])
        return compress_group(p, L, q_obs[b, g * G:(g + 1) * G], k[b, g],
                              None if v is None else v[b, g])

    threads = threads or min(len(units), os.cpu_count() or 1)
    if threads > 1 and len(units) > 1:
        with ThreadPoolExecutor(threads) as ex:
            res = list(ex.map(run, units))
    else:
        res = [run(u) for u in units]
    groups = [[res[b * Hkv + g] for g in range(Hkv)] for b in range(n_seq)]
    ck = np.stack([np.stack([r.cache_k for r in row]) for row in groups])
    cv = None if v is None else np.stack([np.stack([r.cache_v for r in row]) for row in groups])
    nt = np.array([n_topk(int(lengths[b]), p.sink, p.recent, p.topk) for b in range(n_seq)], np.int32)
    return CompressResult(groups, ck, cv, nt, np.asarray(lengths, np.int32).copy())


def decode_attn_group(p: Params, pos: int, ntopk: int, q, ck, cv) -> np.ndarray:
    """Attention of the G heads of one group: q [G][dk], ck [B][k_width], cv [B][v_width] or
    None for a latent cache (values = first dv dims of ck).  Returns [G][dv]."""
    q = np.ascontiguousarray(q, dtype=np.float64)
    ck = np.ascontiguousarray(ck, dtype=np.float64)
    cvv = ck if cv is None else np.ascontiguousarray(cv, dtype=np.float64)
    out = np.zeros((p.group, p.d_v), np.float64)
    _load().oracle_decode_attn(p.group, p.d_qk, p.d_v, ck.shape[-1], cvv.shape[-1], p.sink,
                               p.recent, int(pos), int(ntopk), float(p.scale), _d(q), _d(ck),
                               _d(cvv), _d(out))
    return out


def decode_attn(p: Params, pos, ntopk, q, cache_k, cache_v=None) -> np.ndarray:
    """Batch decode attention: q [n][Hq][dk], caches [n][Hkv][B][width] -> [n][Hq][dv]."""
    q = f64(q)
    cache_k = f64(cache_k)
    cache_v = None if cache_v is None else f64(cache_v)
    n, Hkv = cache_k.shape[0], cache_k.shape[1]
    G = p.group
    out = np.zeros((n, p.n_q_heads, p.d_v), np.float64)
    for b in range(n):
        for g in range(Hkv):
            out[b, g * G:(g + 1) * G] = decode_attn_group(
                p, int(pos[b]), int(ntopk[b]), q[b, g * G:(g + 1) * G], cache_k[b, g],
                None if cache_v is None else cache_v[b, g])
    return out


def prefill_attn_group(p: Params, L: int, q, k, v, want_lse: bool = False, rows=None):
    """Causal attention of the G heads of one group over the first L positions:
    q [G][>=L][dk], k [>=L][dk], v [>=L][dv] -> out [G][n][dv] for the query
    positions rows = (i0, i1) (default every position, n = i1 - i0), and the
    rows' natural-log normalisers [G][n] when want_lse."""
    G = q.shape[0]
    i0, i1 = (0, L) if rows is None else rows
    assert 0 <= i0 <= i1 <= L
    qq = np.ascontiguousarray(f64(q)[:, :L])
    kk = np.ascontiguousarray(f64(k)[:L])
    vv = np.ascontiguousarray(f64(v)[:L])
    assert qq.shape[1] == L and kk.shape[0] == L and vv.shape[0] == L, "inputs shorter than L"
    n = i1 - i0
    out = np.zeros((G, max(n, 1), p.d_v), np.float64)
    lse = np.zeros((G, max(n, 1)), np.float64) if want_lse else None
    if n > 0:
        _load().oracle_prefill_attn(G, p.d_qk, p.d_v, L, i0, i1, float(p.scale), _d(qq), _d(kk), _d(vv), _d(out),
                                    _d(lse) if want_lse else None)
    out = out[:, :n]
    return (out, lse[:, :n]) if want_lse else out


def window_queries(p: Params, lengths, q) -> np.ndarray:
    """The observation-window queries of a padded batch of prompt queries
    q [n][Hq][max_len][dk]: row ii of sequence b is position L_b - w + ii
    (zeros where that position is negative), shape [n][Hq][w][dk] (Sec. III-B.2)."""
    q = f64(q)
    n, Hq, _, dk = q.shape
    w = p.obs_window
    out = np.zeros((n, Hq, w, dk), np.float64)
    for b in range(n):
        L = int(lengths[b])
        for ii in range(w):
            i = L - w + ii
            if i >= 0:
                out[b, :, ii] = q[b, :, i]
    return out


def prefill_attn(p: Params, lengths, q, k, v, threads: int | None = None) -> list:
    """Causal attention of a padded batch: q [n][Hq][max_len][dk], k/v [n][Hkv][max_len][d].
    Returns, per sequence, out [Hq][L][dv] (fp64)."""
    q, k, v = f64(q), f64(k), f64(v)
    n, Hkv = k.shape[0], k.shape[1]
    G = p.group
    units = [(b, g) for b in range(n) for g in range(Hkv)]

    def run(u):
        b, g = u
        return prefill_attn_group(p, int(lengths[b]), q[b, g * G:(g + 1) * G], k[b, g], v[b, g])

    threads = threads or min(len(units), os.cpu_count() or 1)
    if threads > 1 and len(units) > 1:
        with ThreadPoolExecutor(threads) as ex:
            res = list(ex.map(run, units))
    else:
        res = [run(u) for u in units]
    return [np.concatenate([res[b * Hkv + g] for g in range(Hkv)], axis=0) for b in range(n)]


def append(p: Params, pos, cache_k, cache_v, k_new, v_new=None):
    """Decode update (Sec. III-C): write token pos[b]'s K/V at row slot_of(pos[b]), in place."""
    for b in range(cache_k.shape[0]):
        row = slot_of(int(pos[b]), p.sink, p.recent)
        cache_k[b, :, row] = f64(k_new[b])
        if cache_v is not None and v_new is not None:
            cache_v[b, :, row] = f64(v_new[b])


def e4m3_value(code: int) -> float:
    return float(_load().oracle_e4m3_value(int(code)))


def e4m3_encode(x: float) -> int:
    return int(_load().oracle_e4m3_encode(float(x)))


def quantize(x, scale: float) -> np.ndarray:
    """fp8 E4M3 codes of x / scale (quotient in fp32, round-nearest-even, saturating)."""
    x = np.ascontiguousarray(f64(x)).reshape(-1)
    out = np.zeros(x.size, np.uint8)
    _load().oracle_quantize(_d(x), x.size, float(scale), out.ctypes.data_as(_u8p))
    return out


def fp8_scale(x) -> float:
    """Scale from the data: max |x| / 448 in fp32 (1 when x is all zero)."""
    x = np.ascontiguousarray(f64(x)).reshape(-1)
    return float(_load().oracle_fp8_scale(_d(x), x.size))


def dequantize(codes, scale: float) -> np.ndarray:
    codes = np.asarray(codes, np.uint8)
    table = np.array([e4m3_value(c) for c in range(256)], np.float64)
    return table[codes] * float(np.float32(scale))
