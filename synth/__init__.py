"""Seeded synthetic inputs shaped like the paper's workloads.

This module holds NO arithmetic of the method (no scoring, pooling, selection,
cache layout or attention).  It only draws inputs: Gaussian queries, keys and
values, rotary position encoding applied the way a model would before the KV
cache is formed, and planted heavy-hitter keys so that selection has real
structure to find.  Both the fp64 oracle and the HIP path are fed the very same
tensors from here.

The paper's datasets and model weights are not available; these generators
stand in for them (lengths up to 128k tokens, Llama-3.1-8B and DeepSeek MLA
attention shapes, the paper's hyper-parameter tables where a choice is left).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field, replace

import torch

POOL_MAX, POOL_AVG = 0, 1
NORM_CAND, NORM_ROW = 0, 1

# purposes mixed into every seed so each tensor has its own stream
P_Q, P_K, P_V, P_PLANT_POS, P_PLANT_DIR, P_DEC_Q, P_DEC_K, P_DEC_V, P_LEN, P_Q_ALL = range(10)


@dataclass(frozen=True)
class Workload:
    name: str
    cfg_id: int
    n_q_heads: int
    n_kv_heads: int
    d_qk: int
    d_v: int
    v_in_k: bool
    sink: int
    recent: int
    topk: int
    obs_window: int
    pool_kernel: int
    in_dtype: str          # "f32" | "bf16": q/k/v inputs
    kv_dtype: str          # "f32" | "bf16" | "fp8": cache storage
    layers: int
    batch: int             # sequences compressed per layer (slots)
    length: int | None     # fixed prompt length, or None for a uniform draw
    length_range: tuple | None
    decode_steps: int
    rope: bool
    rope_theta: float = 500000.0
    plant_count: int | None = None     # fixed count of heavy hitters
    plant_frac: float | None = None    # or a fraction of the prompt length
    plant_gain: float = 4.0
    pool: int = POOL_MAX
    norm: int = NORM_CAND
    slots: int | None = None           # static cache slots (continuous batching)
    extra: dict = field(default_factory=dict)

    @property
    def budget(self) -> int:
        return self.sink + self.recent + self.topk

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def k_width(self) -> int:
        return self.d_qk

    @property
    def max_len(self) -> int:
        return self.length if self.length is not None else self.length_range[1]


WORKLOADS = {
    # Tiny single layer in fp32; the oracle finishes it in well under a second.
    "tiny-fp32": Workload(
        "tiny-fp32", 1, 4, 2, 64, 64, False, 4, 64, 60, 16, 7, "f32", "f32",
        layers=1, batch=1, length=1024, length_range=None, decode_steps=16,
        rope=False, plant_count=32),
    # Llama-3.1-8B attention shape, one layer, 32k prompt, budget 4096.
    "llama8b-1layer-32k": Workload(
        "llama8b-1layer-32k", 2, 32, 8, 128, 128, False, 4, 1024, 3068, 32, 7, "bf16", "bf16",
        layers=1, batch=1, length=32768, length_range=None, decode_steps=256,
        rope=True, plant_frac=0.01),
    # Llama-3.1-8B shape, 32 layers, 8 sequences of 8k..128k, budget 16384.
    "llama8b-32layer-b8-128k": Workload(
        "llama8b-32layer-b8-128k", 3, 32, 8, 128, 128, False, 4, 2048, 14332, 32, 7, "bf16", "bf16",
        layers=32, batch=8, length=None, length_range=(8192, 131072), decode_steps=512,
        rope=True, plant_frac=0.01),
    # DeepSeek-V3-style MLA, one GPU's share of 16-way head TP: 8 query heads on a
    # shared 576-wide latent (512 latent + 64 rope dims; values = first 512 dims).
    "mla-8head-61layer-b16-128k": Workload(
        "mla-8head-61layer-b16-128k", 4, 8, 1, 576, 512, True, 4, 4096, 28668, 32, 7, "bf16", "bf16",
        layers=61, batch=16, length=131072, length_range=None, decode_steps=256,
        rope=False),
    # Continuous batching over 32 static slots, fp8 E4M3 cache with per-head scales;
    # split of the 8192 budget from the paper's Llama hyper-parameters (768/1024/6400).
    "cb-fp8-llama8b-32slot": Workload(
        "cb-fp8-llama8b-32slot", 5, 32, 8, 128, 128, False, 768, 1024, 6400, 32, 7, "bf16", "fp8",
        layers=32, batch=1, length=None, length_range=(4096, 131072), decode_steps=2000,
        rope=True, plant_frac=0.01, slots=32),
}
# Selection-policy variants of the 128k workloads: the paper's DeepSeek preset
# (512 sinks, 512 selected, 31744 recent, pool kernel 13) on the latent shape;
# a SAGE-KV-like choice (the last query only, no pooling) and StreamingLLM
# alone (no selected rows) on the Llama batch.
WORKLOADS["mla-deepseek-preset-61layer-b16-128k"] = replace(
    WORKLOADS["mla-8head-61layer-b16-128k"], name="mla-deepseek-preset-61layer-b16-128k", sink=512, recent=31744,
    topk=512, pool_kernel=13)
WORKLOADS["llama8b-sagekv-32layer-b8-128k"] = replace(
    WORKLOADS["llama8b-32layer-b8-128k"], name="llama8b-sagekv-32layer-b8-128k", obs_window=1, pool_kernel=1)
WORKLOADS["llama8b-streamingllm-32layer-b8-128k"] = replace(
    WORKLOADS["llama8b-32layer-b8-128k"], name="llama8b-streamingllm-32layer-b8-128k", topk=0)


def seed_of(cfg: int, layer: int, slot: int, purpose: int, step: int = 0) -> int:
    return (((cfg * 1000 + layer) * 1000 + slot) * 16 + purpose) * 100003 + step


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed & 0x7FFFFFFFFFFFFFFF)
    return g


def _randn(shape, seed: int, device) -> torch.Tensor:
    return torch.randn(shape, generator=_gen(seed, device), device=device, dtype=torch.float32)


def rope_(x: torch.Tensor, positions: torch.Tensor, theta: float) -> torch.Tensor:
    """Rotate-half rotary encoding in fp32, in place; x [..., n_pos, D], positions [n_pos]."""
    D = x.shape[-1]
    half = D // 2
    inv = theta ** (-torch.arange(0, half, device=x.device, dtype=torch.float64) * 2.0 / D)
    ang = positions.to(torch.float64)[:, None] * inv[None, :]
    cos = torch.cos(ang).to(torch.float32)
    sin = torch.sin(ang).to(torch.float32)
    x1 = x[..., :half].clone()
    x2 = x[..., half:].clone()
    x[..., :half] = x1 * cos - x2 * sin
    x[..., half:] = x2 * cos + x1 * sin
    return x


def cast(x: torch.Tensor, dtype: str) -> torch.Tensor:
    return x.to(torch.float32 if dtype == "f32" else torch.bfloat16)


def draw_lengths(wl: Workload, layer: int, n: int, device="cpu", salt: int = 0) -> list[int]:
    if wl.length is not None:
        return [wl.length] * n
    lo, hi = wl.length_range
    g = _gen(seed_of(wl.cfg_id, layer, 999, P_LEN, salt), "cpu")
    return [int(x) for x in torch.randint(lo, hi + 1, (n,), generator=g)]


def plant_positions(wl: Workload, layer: int, slot: int, L: int, salt: int = 0) -> torch.Tensor:
    """Heavy-hitter token positions, uniform without replacement among the
    tokens that are neither sinks nor recent."""
    lo, hi = wl.sink, L - wl.recent
    n_avail = max(hi - lo, 0)
    if wl.plant_count is not None:
        n = wl.plant_count
    elif wl.plant_frac is not None:
        n = int(wl.plant_frac * L)
    else:
        n = 0
    n = min(n, n_avail)
    if n == 0:
        return torch.zeros(0, dtype=torch.int64)
    g = _gen(seed_of(wl.cfg_id, layer, slot, P_PLANT_POS, salt), "cpu")
    return lo + torch.randperm(n_avail, generator=g)[:n]


def plant_direction(wl: Workload, layer: int, kv_head: int) -> torch.Tensor:
    g = _gen(seed_of(wl.cfg_id, layer, 900 + kv_head, P_PLANT_DIR), "cpu")
    u = torch.randn(wl.d_qk, generator=g, dtype=torch.float64)
    return (u / u.norm()).to(torch.float32)


def obs_queries(wl: Workload, layer: int, slot: int, L: int, device="cpu", salt: int = 0) -> torch.Tensor:
    """The observation-window queries of one prompt alone, q_obs [Hq][w][dqk]:
    the same tensor prefill() returns for these arguments."""
    w = wl.obs_window
    q = _randn((wl.n_q_heads, w, wl.d_qk), seed_of(wl.cfg_id, layer, slot, P_Q, salt), device)
    if wl.rope:
        rope_(q, torch.arange(L - w, L, device=device), wl.rope_theta)
    return cast(q, wl.in_dtype)


def prefill(wl: Workload, layer: int, slot: int, L: int, device="cpu", salt: int = 0,
            max_len: int | None = None, pad_value: float = 0.0):
    """Inputs of one sequence: q_obs [Hq][w][dqk], k [Hkv][Lpad][k_width], v [Hkv][Lpad][dv]
    (None for a latent cache), in the workload's input dtype; rows >= L hold pad_value."""
    Lpad = max_len or L
    w = wl.obs_window
    sd = lambda p: seed_of(wl.cfg_id, layer, slot, p, salt)
    k = _randn((wl.n_kv_heads, L, wl.k_width), sd(P_K), device)
    q = _randn((wl.n_q_heads, w, wl.d_qk), sd(P_Q), device)
    v = None if wl.v_in_k else _randn((wl.n_kv_heads, L, wl.d_v), sd(P_V), device)
    if wl.rope:
        rope_(k, torch.arange(L, device=device), wl.rope_theta)
        rope_(q, torch.arange(L - w, L, device=device), wl.rope_theta)
    pos = plant_positions(wl, layer, slot, L, salt).to(device)
    if pos.numel():
        for g in range(wl.n_kv_heads):
            u = plant_direction(wl, layer, g).to(device)
            k[g, pos] += wl.plant_gain * math.sqrt(wl.d_qk) * u
    kk = torch.full((wl.n_kv_heads, Lpad, wl.k_width), pad_value, dtype=torch.float32, device=device)
    kk[:, :L] = k
    vv = None
    if v is not None:
        vv = torch.full((wl.n_kv_heads, Lpad, wl.d_v), pad_value, dtype=torch.float32, device=device)
        vv[:, :L] = v
    return cast(q, wl.in_dtype), cast(kk, wl.in_dtype), None if vv is None else cast(vv, wl.in_dtype)


def prefill_batch(wl: Workload, layer: int, lengths, device="cpu", salt: int = 0,
                  max_len: int | None = None, pad_value: float = 0.0, slots=None):
    """Padded batch: q_obs [n][Hq][w][dqk], k [n][Hkv][max_len][k_width], v or None."""
    n = len(lengths)
    Lmax = max_len or max(lengths)
    slots = list(range(n)) if slots is None else list(slots)
    dt = torch.float32 if wl.in_dtype == "f32" else torch.bfloat16
    q = torch.empty((n, wl.n_q_heads, wl.obs_window, wl.d_qk), dtype=dt, device=device)
    k = torch.empty((n, wl.n_kv_heads, Lmax, wl.k_width), dtype=dt, device=device)
    v = None if wl.v_in_k else torch.empty((n, wl.n_kv_heads, Lmax, wl.d_v), dtype=dt, device=device)
    for b, L in enumerate(lengths):
        qb, kb, vb = prefill(wl, layer, slots[b], int(L), device, salt, Lmax, pad_value)
        q[b] = qb
        k[b] = kb
        if v is not None:
            v[b] = vb
    return q, k, v


def prompt_queries(wl: Workload, layer: int, slot: int, L: int, device="cpu", salt: int = 0,
                   max_len: int | None = None, pad_value: float = 0.0) -> torch.Tensor:
    """The queries of every prompt position, q [Hq][Lpad][dqk] (the input of the
    prefill attention; its last w rows are that prompt's observation window),
    Gaussian with the rotary encoding of positions 0..L-1; rows >= L hold
    pad_value."""
    Lpad = max_len or L
    q = _randn((wl.n_q_heads, L, wl.d_qk), seed_of(wl.cfg_id, layer, slot, P_Q_ALL, salt), device)
    if wl.rope:
        rope_(q, torch.arange(L, device=device), wl.rope_theta)
    qq = torch.full((wl.n_q_heads, Lpad, wl.d_qk), pad_value, dtype=torch.float32, device=device)
    qq[:, :L] = q
    return cast(qq, wl.in_dtype)


def prompt_batch(wl: Workload, layer: int, lengths, device="cpu", salt: int = 0,
                 max_len: int | None = None, pad_value: float = 0.0, slots=None):
    """Padded batch for the prefill attention: q [n][Hq][max_len][dqk] (every
    position), k [n][Hkv][max_len][dqk], v [n][Hkv][max_len][dv]; k and v as
    prefill_batch draws them."""
    n = len(lengths)
    Lmax = max_len or max(lengths)
    slots = list(range(n)) if slots is None else list(slots)
    _, k, v = prefill_batch(wl, layer, lengths, device, salt, Lmax, pad_value, slots)
    dt = torch.float32 if wl.in_dtype == "f32" else torch.bfloat16
    q = torch.empty((n, wl.n_q_heads, Lmax, wl.d_qk), dtype=dt, device=device)
    for b, L in enumerate(lengths):
        q[b] = prompt_queries(wl, layer, slots[b], int(L), device, salt, Lmax, pad_value)
    return q, k, v


def decode_inputs(wl: Workload, layer: int, step: int, positions, device="cpu", salt: int = 0):
    """One decode step for n sequences at absolute positions `positions`:
    q [n][Hq][dqk], k_new [n][Hkv][k_width], v_new [n][Hkv][dv] (None for latent)."""
    n = len(positions)
    sd = lambda p: seed_of(wl.cfg_id, layer, 0, p, salt * 1000003 + step)
    q = _randn((n, wl.n_q_heads, 1, wl.d_qk), sd(P_DEC_Q), device)
    k = _randn((n, wl.n_kv_heads, 1, wl.k_width), sd(P_DEC_K), device)
    v = None if wl.v_in_k else _randn((n, wl.n_kv_heads, wl.d_v), sd(P_DEC_V), device)
    if wl.rope:
        for b, p in enumerate(positions):
            pt = torch.tensor([int(p)], device=device)
            rope_(q[b], pt, wl.rope_theta)
            rope_(k[b], pt, wl.rope_theta)
    q = q[:, :, 0]
    k = k[:, :, 0]
    return cast(q, wl.in_dtype), cast(k, wl.in_dtype), None if v is None else cast(v, wl.in_dtype)


def decode_inputs_all(wl: Workload, layer: int, steps: int, start_positions, device="cpu", salt: int = 0):
    """Decode inputs of `steps` consecutive steps at once (one random draw per
    tensor): q [steps][n][Hq][dqk], k [steps][n][Hkv][k_width], v or None.
    Step t of sequence b sits at position start_positions[b] + t."""
    n = len(start_positions)
    sd = lambda p: seed_of(wl.cfg_id, layer, 0, p, salt * 1000003 + 777777)
    q = _randn((steps, n, wl.n_q_heads, wl.d_qk), sd(P_DEC_Q), device)
    k = _randn((steps, n, wl.n_kv_heads, wl.k_width), sd(P_DEC_K), device)
    v = None if wl.v_in_k else _randn((steps, n, wl.n_kv_heads, wl.d_v), sd(P_DEC_V), device)
    if wl.rope:
        start = torch.as_tensor(start_positions, device=device)
        pos = (start[None, :] + torch.arange(steps, device=device)[:, None]).reshape(-1)
        qq = q.reshape(steps * n, wl.n_q_heads, wl.d_qk).transpose(0, 1)   # [H][steps*n][D]
        kk = k.reshape(steps * n, wl.n_kv_heads, wl.k_width).transpose(0, 1)
        qq = rope_(qq.contiguous(), pos, wl.rope_theta)
        kk = rope_(kk.contiguous(), pos, wl.rope_theta)
        q = qq.transpose(0, 1).reshape(steps, n, wl.n_q_heads, wl.d_qk)
        k = kk.transpose(0, 1).reshape(steps, n, wl.n_kv_heads, wl.k_width)
    return cast(q, wl.in_dtype).contiguous(), cast(k, wl.in_dtype).contiguous(), \
        None if v is None else cast(v, wl.in_dtype).contiguous()


def small(wl: Workload, **kw) -> Workload:
    """A copy with some fields replaced (for scaled-down test cases)."""
    return replace(wl, **kw)
