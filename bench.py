#!/usr/bin/env python3
"""Benchmark of the SnapStream hot path on one MI355X.

One step = one pass of the whole hot path over one batch: snap_compress of
every (layer, sequence) from prompts resident in HBM, then `decode_steps`
decode steps, each running snap_decode_step (append + attention; or, with
--two-calls, snap_cache_append + snap_decode_attn) for every layer and one
snap_advance.  Inputs (prompts and every decode step's q/k/v) are generated
before the timed region.

Prints ONE JSON line.  `value` is decoded tokens per second of the whole step
(compression included); the decode-only rate, the per-layer decode-step HBM
GB/s and the per-(sequence, layer) snap_compress latency are reported beside
it.

--prefill measures the other end of the path instead: one step is one
snap_prefill call per layer (causal attention over every prompt position,
then the compression with the window statistics taken from the attention
pass).  `value` is prompt tokens per second per layer; the roofline is the
attention kernel's bf16 MFMA rate, timed through snap_prefill_attn (the same
attention without the compression), and the cost of the fused compression is
reported beside the unfused snap_compress on the same window queries.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import subprocess
import sys
import time

DEFAULT_WORKLOAD = "mla-8head-61layer-b16-128k"
KV_REUSE = {"auto": 0, "stream": 1, "keep": 2}  # snap_kv_reuse
DEFAULT_PREFILL_WORKLOAD = "llama8b-1layer-32k"
HERE = os.path.dirname(os.path.abspath(__file__))


def _elf_section(d: bytes, want: bytes):
    """Contents of the section named `want` of a 64-bit ELF image, or None."""
    import struct
    if d[:5] != b"\x7fELF\x02":
        return None
    shoff = struct.unpack_from("<Q", d, 0x28)[0]
    shentsize, shnum, shstrndx = struct.unpack_from("<HHH", d, 0x3A)
    sh = lambda i: struct.unpack_from("<IIQQQQ", d, shoff + i * shentsize)  # noqa: E731
    stroff = sh(shstrndx)[4]
    for i in range(shnum):
        name, _, _, _, off, size = sh(i)
        if d[stroff + name:d.index(b"\0", stroff + name)] == want:
            return d[off:off + size]
    return None


def _kernel_code(code: bytes, pattern: str):
    """Machine code of the functions of an ELF code object whose symbol names
    match `pattern` (a regular expression), concatenated in name order."""
    import re
    import struct
    if code[:5] != b"\x7fELF\x02":
        return None
    shoff = struct.unpack_from("<Q", code, 0x28)[0]
    shentsize, shnum = struct.unpack_from("<HH", code, 0x3A)
    secs = [struct.unpack_from("<IIQQQQIIQQ", code, shoff + i * shentsize) for i in range(shnum)]
    out = []
    for _, type_, _, _, off, size, link, _, _, entsize in secs:
        if type_ != 2:  # SHT_SYMTAB
            continue
        stroff = secs[link][4]
        for j in range(size // entsize):
            st_name, st_info, _, st_shndx, st_value, st_size = struct.unpack_from("<IBBHQQ", code, off + j * entsize)
            nm = code[stroff + st_name:code.index(b"\0", stroff + st_name)].decode()
            if (st_info & 0xF) == 2 and st_size and re.search(pattern, nm):  # STT_FUNC
                sec = secs[st_shndx]
                start = sec[4] + (st_value - sec[3])
                out.append((nm, code[start:start + st_size]))
    if not out:
        return None
    return b"".join(c for _, c in sorted(out))


def device_code_sha256(lib_path: str, kernels: str):
    """sha256 of the machine code of the kernels whose symbol names match
    `kernels` (a regular expression), in the gfx950 code objects of a built
    library's .hip_fatbin section: it changes when one of those kernels
    changes, and not when only comments, host code or other kernels do."""
    import hashlib
    import struct
    try:
        d = open(lib_path, "rb").read()
    except OSError:
        return None
    fat = _elf_section(d, b".hip_fatbin")
    if fat is None:
        return None
    # offload bundles: magic, entry count, then (offset, size, triple length,
    # triple) per entry, offsets from the bundle's start
    magic = b"__CLANG_OFFLOAD_BUNDLE__"
    parts = []
    b = fat.find(magic)
    while b >= 0:
        n = struct.unpack_from("<Q", fat, b + len(magic))[0]
        o = b + len(magic) + 8
        for _ in range(n):
            off, size, tl = struct.unpack_from("<QQQ", fat, o)
            triple = fat[o + 24:o + 24 + tl]
            o += 24 + tl
            if triple.endswith(b"gfx950"):
                k = _kernel_code(fat[b + off:b + off + size], kernels)
                if k:
                    parts.append(k)
        b = fat.find(magic, b + 1)
    return hashlib.sha256(b"".join(parts)).hexdigest() if parts else None


def seed_rule(wl):
    """How every synthetic input of the run is seeded (all are drawn from
    these counters alone, so a run is reproducible from the workload name)."""
    return {"cfg_id": wl.cfg_id, "rule": "synth.seed_of(cfg_id, layer, slot, purpose, step)"}


def measured_traffic(workload: str):
    """HBM bytes per launch of the roofline kernel from the committed counter
    runs (profiles/traffic.json, keyed by workload; the prefill attention's
    records by "prefill:" + workload), or None when no record exists or the
    machine code of the record's kernels (its "kernels" pattern) has changed
    since the counters were taken."""
    try:
        rec = json.load(open(os.path.join(HERE, "profiles", "traffic.json")))[workload]
    except (OSError, KeyError, ValueError):
        return None
    code = device_code_sha256(os.path.join(HERE, "paper_2511_03092_amd", "libsnapstream.so"), rec["kernels"])
    if code is None or code != rec.get("device_code_sha256"):
        return None
    return rec["traffic_bytes_per_launch"]


def measured_mfma(workload: str):
    """MFMA utilisation of the workload's score kernels (or the prefill
    attention, records keyed "prefill:" + workload) from the committed counter
    runs (profiles/mfma.json: MfmaUtil = MFMA-busy cycles over active cycles of
    every SIMD, per kernel), or None when no record exists or the kernels'
    machine code has changed since the counters were taken."""
    try:
        rec = json.load(open(os.path.join(HERE, "profiles", "mfma.json")))[workload]
    except (OSError, KeyError, ValueError):
        return None
    code = device_code_sha256(os.path.join(HERE, "paper_2511_03092_amd", "libsnapstream.so"), rec["kernels"])
    if code is None or code != rec.get("device_code_sha256"):
        return None
    return {"mfma_util": rec["mfma_util"], "mfma_bf16_flops_per_launch": rec["mfma_bf16_flops_per_launch"],
            "source": "rocprofv3 counters, profiles/mfma.json"}


def copy_calibration(torch, nbytes, dev):
    """One device-to-device copy of nbytes: the reference that scales the HBM
    byte counters (FETCH_SIZE / WRITE_SIZE) of a counter run."""
    src = torch.empty(nbytes // 4, dtype=torch.float32, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


# continuous batching: the new prompt's per-layer compressions run on this many
# streams (measured 3405 tok/s with 1, 4250 with 2, 4070 with 4, 4337 with 8)
DEFAULT_COMPRESS_STREAMS = 2

PEAK_HBM_GBPS = 8000.0
PEAK_BF16_TFLOPS = 2500.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed steps (default 3; 64 for the continuous-batching workload)")
    ap.add_argument("--warmup", type=int, default=None,
                    help="untimed steps first (default 1; 32 for the continuous-batching workload)")
    ap.add_argument("--workload", default=None)
    ap.add_argument("--prefill", action="store_true",
                    help="time snap_prefill (prefill attention + fused compression) instead of the decode step")
    ap.add_argument("--decode-steps", type=int, default=None, help="override the workload's decode steps")
    ap.add_argument("--layers", type=int, default=None, help="override the layer count (profiling only)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--two-calls", action="store_true",
                    help="decode with snap_cache_append + snap_decode_attn instead of snap_decode_step")
    ap.add_argument("--graph", action="store_true",
                    help="run each step's decode phase as one captured HIP graph (replayed every step)")
    ap.add_argument("--fp8-scales-from-data", action="store_true",
                    help="continuous batching: snap_compress sets the fp8 scales (amax / 448 of the kept rows)")
    ap.add_argument("--fp8-qk", action="store_true",
                    help="fp8 caches: quantise each decode query head to E4M3 and run Q K^T on the fp8 MFMA "
                         "(snap_params.fp8_qk)")
    ap.add_argument("--overlap", action="store_true",
                    help="continuous batching: run each step's compression and decode on two streams at once")
    ap.add_argument("--compress-streams", type=int, default=None, metavar="K",
                    help="continuous batching: the new prompt's per-layer compress calls over K streams "
                         f"(default {DEFAULT_COMPRESS_STREAMS}; layers are independent; each stream has its own "
                         "workspace; 1 runs them in order on the step's stream)")
    ap.add_argument("--kv-reuse", choices=["auto", "stream", "keep"], default="auto",
                    help="decode load hint (snap_params.kv_reuse): auto streams calls of 128 MiB and more")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="before the run, copy BYTES device-to-device once (a reference for HBM counters)")
    ap.add_argument("--no-others", action="store_true",
                    help="the default run: skip the short runs of the other workloads after the headline one")
    return ap.parse_args()


def main(args):
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU: this build has no multi-GPU path (the hot path shards by "
              "KV head or by slot with no exchange; see the design notes). Run with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)
    import torch

    import paper_2511_03092_amd as snap
    import synth

    if args.workload is None:
        args.workload = DEFAULT_PREFILL_WORKLOAD if args.prefill else DEFAULT_WORKLOAD
    wl = synth.WORKLOADS[args.workload]
    if args.prefill:
        return run_prefill(args, wl)
    if wl.slots is not None:
        return run_cb(args, wl)
    if args.steps is None:
        args.steps = 3
    if args.warmup is None:
        args.warmup = 1
    layers = args.layers or wl.layers
    dsteps = wl.decode_steps if args.decode_steps is None else args.decode_steps
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    DT = {"f32": snap.SNAP_F32, "bf16": snap.SNAP_BF16, "fp8": snap.SNAP_FP8_E4M3}
    p = snap.Params(wl.n_q_heads, wl.n_kv_heads, wl.d_qk, wl.d_v, wl.sink, wl.recent, wl.topk, wl.obs_window,
                    wl.pool_kernel, wl.pool, wl.norm, wl.v_in_k, DT[wl.in_dtype], DT[wl.kv_dtype],
                    kv_reuse=KV_REUSE[args.kv_reuse])
    n = wl.batch
    lengths = synth.draw_lengths(wl, 0, n)
    max_len = max(lengths)
    B = p.budget
    kvt = {"f32": torch.float32, "bf16": torch.bfloat16, "fp8": torch.uint8}[wl.kv_dtype]

    # ---- resident inputs and caches (untimed)
    t_setup = time.time()
    prompts, caches, dec = [], [], []
    for l in range(layers):
        q, k, v = synth.prefill_batch(wl, l, lengths, device=dev, max_len=max_len)
        prompts.append((q, k, v))
        ck = torch.zeros((n, wl.n_kv_heads, B, wl.d_qk), dtype=kvt, device=dev)
        cv = None if wl.v_in_k else torch.zeros((n, wl.n_kv_heads, B, wl.d_v), dtype=kvt, device=dev)
        caches.append((ck, cv, snap.cache_struct(ck, cv)))
        dec.append(synth.decode_inputs_all(wl, l, max(dsteps, 1), lengths, device=dev))
    pos = torch.zeros((n,), dtype=torch.int32, device=dev)
    ntop = torch.zeros((n,), dtype=torch.int32, device=dev)
    slots = torch.arange(n, dtype=torch.int32, device=dev)
    lens = torch.tensor(lengths, dtype=torch.int32, device=dev)
    wsc = snap.workspace(snap.snap_compress_workspace(p, n, max_len), dev)
    wsd = snap.workspace(snap.snap_decode_workspace(p, n), dev)
    out = torch.empty((n, wl.n_q_heads, wl.d_v), dtype=torch.bfloat16, device=dev)
    torch.cuda.synchronize()
    t_setup = time.time() - t_setup
    stream = torch.cuda.current_stream()
    sptr = stream.cuda_stream

    if args.copy_calibration:
        copy_calibration(torch, args.copy_calibration, dev)

    # ---- one step.  Events bracket whole phases (every layer's compress; the
    # whole decode loop), never single calls: an event record costs device
    # time of its own, which would be charged to the call it brackets.
    def ev():
        e = torch.cuda.Event(enable_timing=True)
        e.record(stream)
        return e

    def decode_phase(sp):
        for t in range(dsteps):
            for l in range(layers):
                qd, kd, vd = dec[l]
                if args.two_calls:
                    snap.snap_cache_append(p, caches[l][2], pos, slots, kd[t], None if vd is None else vd[t],
                                           stream=sp)
                    snap.snap_decode_attn(p, caches[l][2], pos, ntop, slots, qd[t], out, wsd, stream=sp)
                else:
                    snap.snap_decode_step(p, caches[l][2], pos, ntop, slots, qd[t], kd[t],
                                          None if vd is None else vd[t], out, wsd, stream=sp)
            snap.snap_advance(pos, slots, stream=sp)

    graph = []

    def step(timing):
        if timing is not None:
            c0 = ev()
        for l in range(layers):
            q, k, v = prompts[l]
            snap.snap_compress(p, caches[l][2], pos, ntop, slots, lens, q, k, v, wsc, stream=sptr)
        if timing is not None:
            timing["compress"].append((c0, ev()))
        if graph:
            graph[0].replay()
        else:
            decode_phase(sptr)
        if timing is not None:
            timing["decode"].append((timing["compress"][-1][1], ev()))

    for _ in range(args.warmup):
        step(None)
    torch.cuda.synchronize()
    if args.graph:
        # the whole decode phase of a step (every layer's decode calls and the
        # advances) captured once; every timed step compresses eagerly, then
        # replays it on the same stream
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            decode_phase(torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        graph.append(g)
    timing = {"compress": [], "decode": []}
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record(stream)
    for _ in range(args.steps):
        step(timing)
    t1.record(stream)
    torch.cuda.synchronize()
    ms_total = t0.elapsed_time(t1)
    ms_step = ms_total / args.steps
    # per layer call: phase time / calls (the decode phase includes one
    # snap_advance per step, shared by that step's layer calls)
    comp_ms = sum(a.elapsed_time(b) for a, b in timing["compress"]) / (args.steps * layers)
    dec_ms = (sum(a.elapsed_time(b) for a, b in timing["decode"]) / (args.steps * dsteps * layers)
              if dsteps else 0.0)

    # ---- algorithmic bytes of one layer's decode step: valid rows + q + out, plus
    # the appended token (read from the input, written to its cache row)
    s_r = wl.sink + wl.recent
    elt = {"f32": 4, "bf16": 2, "fp8": 1}[wl.kv_dtype]
    row_bytes = wl.d_qk * elt + (0 if wl.v_in_k else wl.d_v * elt)
    valid = 0
    for L in lengths:
        ncand = max(L - s_r, 0)
        # rows valid while decoding: sinks+ring (full once L >= s+r) plus the kept rows
        valid += min(L + 1, s_r) + min(ncand, wl.topk)
    q_bytes = n * wl.n_q_heads * wl.d_qk * 2
    o_bytes = n * wl.n_q_heads * wl.d_v * 2
    in_elt = 2 if wl.in_dtype == "bf16" else 4
    new_bytes = n * wl.n_kv_heads * (wl.d_qk + (0 if wl.v_in_k else wl.d_v)) * in_elt + n * wl.n_kv_heads * row_bytes
    dec_bytes = valid * wl.n_kv_heads * row_bytes + q_bytes + o_bytes + new_bytes
    dec_gbps = dec_bytes / (dec_ms * 1e-3) / 1e9 if dec_ms > 0 else 0.0
    # ---- score GEMM (Q_obs x K^T of both compress passes) against the bf16 MFMA
    # peak: useful flops over the whole compress call, a lower bound on the
    # score kernels' own utilisation (the call also pools, selects and gathers)
    G = wl.n_q_heads // wl.n_kv_heads
    score_flop = 0
    for L in lengths:
        keys = max(L - s_r, 0) if wl.topk > 0 else 0  # candidates: the normaliser domain of both passes
        score_flop += wl.n_kv_heads * 2 * G * min(wl.obs_window, L) * wl.d_qk * keys
    score_tflops = 2 * score_flop / (comp_ms * 1e-3) / 1e12 if comp_ms > 0 else 0.0
    tokens = n * dsteps
    value = tokens / (ms_step * 1e-3)
    decode_ms_per_token_step = dec_ms * layers  # attention only, per decode step (all layers)

    res = {
        "metric": "compressed-KV decode tok/s/GPU + HBM GB/s at 128k; snap_compress latency",
        "value": round(value, 2),
        "unit": "tok/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.in_dtype == "bf16" else "f32",
        "data": "synthetic",
        "launch": "hip_graph" if args.graph else "eager",
        "config": {"workload": wl.name, "seeds": seed_rule(wl), "layers": layers, "sequences": n, "prompt_lengths": lengths,
                   "budget": B, "sink": wl.sink, "recent": wl.recent, "topk": wl.topk,
                   "obs_window": wl.obs_window, "pool_kernel": wl.pool_kernel, "decode_steps": dsteps,
                   "q_heads": wl.n_q_heads, "kv_heads": wl.n_kv_heads, "d_qk": wl.d_qk, "d_v": wl.d_v,
                   "kv_dtype": wl.kv_dtype, "kv_reuse": args.kv_reuse},
        "decode_step_ms_per_call": round(dec_ms, 4),
        "decode_step_hbm_gbps": round(dec_gbps, 1),
        "decode_only_tok_s": round(n / (decode_ms_per_token_step * 1e-3), 1) if dec_ms > 0 else 0.0,
        "compress_ms_per_layer_call": round(comp_ms, 4),
        "compress_ms_per_seq_layer": round(comp_ms / n, 4),
        "score_gemm": {"gflop_per_layer_call_one_pass": round(score_flop / 1e9, 2), "passes": 2,
                       "tflops_over_compress_call": round(score_tflops, 1), "peak_tflops": PEAK_BF16_TFLOPS,
                       "mfma_util_lower_bound": round(score_tflops / PEAK_BF16_TFLOPS, 4),
                       "counters": measured_mfma(wl.name)},
        "roofline": {"bound": "hbm",
                     "kernel": ("snap_cache_append + snap_decode_attn" if args.two_calls else
                                "snap_decode_step (append + split-K attention, one launch) + chunk merge"),
                     "achieved": round(dec_gbps, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                     "frac": round(dec_gbps / PEAK_HBM_GBPS, 4), "traffic": measured_traffic(wl.name),
                     "algorithmic_bytes_per_launch": dec_bytes},
        "setup_s": round(t_setup, 1),
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(wl, p, lengths, n, layers, dsteps, n * dsteps, value)
    return res


def run_cb(args, wl):
    """Continuous batching over wl.slots static cache slots (every layer has
    its own caches; slot metadata is shared).  All slots are filled first
    (untimed).  Step t then retires slot t mod slots: snap_compress of a new
    prompt into it for every layer, and one decode step (snap_decode_step per
    layer, snap_advance) over the other slots, one after the other (with
    --overlap, on two streams at once: they touch disjoint slots).
    Prompts are prefixes, of a
    seeded length in the workload's range, of one 128k-token K/V bank per
    layer resident in HBM, each with its own observation-window queries.  fp8
    cache scales are per (slot, KV head) amax / 448, set by this harness: the
    amax is taken over the layer's whole bank (an upper bound for every
    prefix), once, before the timed region."""
    import torch

    import paper_2511_03092_amd as snap
    import synth

    if args.steps is None:
        args.steps = 64
    if args.warmup is None:
        args.warmup = wl.slots
    S = wl.slots
    layers = args.layers or wl.layers
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    DT = {"f32": snap.SNAP_F32, "bf16": snap.SNAP_BF16, "fp8": snap.SNAP_FP8_E4M3}
    p = snap.Params(wl.n_q_heads, wl.n_kv_heads, wl.d_qk, wl.d_v, wl.sink, wl.recent, wl.topk, wl.obs_window,
                    wl.pool_kernel, wl.pool, wl.norm, wl.v_in_k, DT[wl.in_dtype], DT[wl.kv_dtype],
                    fp8_scales=snap.SNAP_FP8_SCALES_AMAX if args.fp8_scales_from_data else snap.SNAP_FP8_SCALES_GIVEN,
                    fp8_qk=1 if args.fp8_qk else 0, kv_reuse=KV_REUSE[args.kv_reuse])
    B = p.budget
    Lmax = wl.max_len
    n_steps = args.warmup + args.steps
    nd = S - 1  # sequences decoded per step
    lengths = synth.draw_lengths(wl, 0, S + n_steps)  # the initial fill, then one prompt per step
    kvt = {"f32": torch.float32, "bf16": torch.bfloat16, "fp8": torch.uint8}[wl.kv_dtype]

    t_setup = time.time()
    banks, caches, obsq, dec = [], [], [], []
    for l in range(layers):
        _, kb, vb = synth.prefill(wl, l, 0, Lmax, device=dev)
        kb, vb = kb.unsqueeze(0), vb.unsqueeze(0)  # [1][Hkv][Lmax][d]
        banks.append((kb, vb))
        ck = torch.zeros((S, wl.n_kv_heads, B, wl.d_qk), dtype=kvt, device=dev)
        cv = torch.zeros((S, wl.n_kv_heads, B, wl.d_v), dtype=kvt, device=dev)
        ks = (kb[0].float().abs().amax(dim=(1, 2)).clamp_min(1e-6) / 448.0).repeat(S, 1).contiguous()
        vs = (vb[0].float().abs().amax(dim=(1, 2)).clamp_min(1e-6) / 448.0).repeat(S, 1).contiguous()
        caches.append((ck, cv, ks, vs, snap.cache_struct(ck, cv, ks, vs)))
        # observation-window queries of every prompt (initial fill, then one per step)
        obsq.append(torch.stack([synth.obs_queries(wl, l, 1000 + i, lengths[i], device=dev)
                                 for i in range(S + n_steps)]).contiguous())
        dec.append(synth.decode_inputs_all(wl, l, n_steps, lengths[1:S], device=dev))
    pos = torch.full((S,), -1, dtype=torch.int32, device=dev)
    ntop = torch.zeros((S,), dtype=torch.int32, device=dev)
    slot_ids = torch.arange(S, dtype=torch.int32, device=dev)
    lens = torch.tensor(lengths, dtype=torch.int32, device=dev)
    # the decoded slots of the step that retires slot r: every slot but r
    live = [torch.tensor([x for x in range(S) if x != r], dtype=torch.int32, device=dev) for r in range(S)]
    KC = max(1, DEFAULT_COMPRESS_STREAMS if args.compress_streams is None else args.compress_streams)
    wscs = [snap.workspace(snap.snap_compress_workspace(p, 1, Lmax), dev) for _ in range(KC)]
    wsd = snap.workspace(snap.snap_decode_workspace(p, nd), dev)
    out = torch.empty((nd, wl.n_q_heads, wl.d_v), dtype=torch.bfloat16, device=dev)
    stream = torch.cuda.current_stream()
    sptr = stream.cuda_stream
    side = [torch.cuda.Stream() for _ in range(KC)] if KC > 1 else []

    def compress(i, slot, st):
        # one prompt into `slot` for every layer, ordered on stream st (with
        # --compress-streams K the layers run on K side streams that start
        # after, and end before, st's work at this point)
        if KC > 1:
            e = torch.cuda.Event()
            e.record(st)
            for x in side:
                x.wait_event(e)
        for l in range(layers):
            kb, vb = banks[l]
            sp = side[l % KC].cuda_stream if KC > 1 else st.cuda_stream
            snap.snap_compress(p, caches[l][4], pos, ntop, slot_ids[slot:slot + 1], lens[i:i + 1],
                               obsq[l][i:i + 1], kb, vb, wscs[l % KC], stream=sp)
        if KC > 1:
            for x in side:
                e = torch.cuda.Event()
                e.record(x)
                st.wait_event(e)

    def decode(t, retired, sp):
        for l in range(layers):
            qd, kd, vd = dec[l]
            snap.snap_decode_step(p, caches[l][4], pos, ntop, live[retired], qd[t], kd[t], vd[t], out, wsd,
                                  stream=sp)
        snap.snap_advance(pos, live[retired], stream=sp)

    for r in range(S):  # fill every slot
        compress(r, r, stream)
    torch.cuda.synchronize()
    t_setup = time.time() - t_setup
    if args.copy_calibration:
        copy_calibration(torch, args.copy_calibration, dev)

    def ev(st):
        e = torch.cuda.Event(enable_timing=True)
        e.record(st)
        return e

    # The new prompt's compression and the other slots' decode step touch
    # disjoint slots, so with --overlap they run on two streams at once.
    # Across steps: the compression of step t rewrites a slot the decode of
    # step t-1 used, and the decode of step t attends the slot compressed in
    # step t-1.
    overlap = args.overlap
    s_c = torch.cuda.Stream() if overlap else stream
    s_d = torch.cuda.Stream() if overlap else stream
    # host mirror of each slot's prompt length and position, for the bytes count
    slot_len = list(lengths[:S])
    slot_pos = list(lengths[:S])
    s_r, row_bytes = wl.sink + wl.recent, (wl.d_qk + wl.d_v) * (1 if wl.kv_dtype == "fp8" else 2)
    timing = {"compress": [], "decode": []}
    dec_bytes, timed_lengths = 0, []
    t0 = t1 = prev_c = prev_d = None
    for t in range(n_steps):
        timed = t >= args.warmup
        if t == args.warmup:
            torch.cuda.synchronize()
            t0 = ev(stream)
            if overlap:
                s_c.wait_event(t0)
                s_d.wait_event(t0)
        r = t % S
        i = S + t
        if overlap and prev_d is not None:
            s_c.wait_event(prev_d)
        c0 = ev(s_c)
        compress(i, r, s_c)
        prev_c_next = ev(s_c)
        if overlap and prev_c is not None:
            s_d.wait_event(prev_c)
        d0 = ev(s_d)
        decode(t, r, s_d.cuda_stream)
        prev_d = ev(s_d)
        prev_c = prev_c_next
        if timed:
            timing["compress"].append((c0, prev_c))
            timing["decode"].append((d0, prev_d))
            timed_lengths.append(lengths[i])
        slot_len[r] = slot_pos[r] = lengths[i]
        for x in range(S):
            if x == r:
                continue
            if timed:
                ncand = max(slot_len[x] - s_r, 0)
                dec_bytes += layers * (wl.n_kv_heads * (min(slot_pos[x] + 1, s_r) + min(ncand, wl.topk)) * row_bytes
                                       + wl.n_kv_heads * 2 * 4)  # rows + the two scales
            slot_pos[x] += 1
    if overlap:
        stream.wait_event(prev_c)
        stream.wait_event(prev_d)
    t1 = ev(stream)
    torch.cuda.synchronize()
    K = args.steps
    ms_step = t0.elapsed_time(t1) / K
    comp_ms = sum(a.elapsed_time(b) for a, b in timing["compress"]) / (K * layers)
    dec_ms = sum(a.elapsed_time(b) for a, b in timing["decode"]) / (K * layers)
    # per decode call: q and out (bf16), the new token read (bf16) and written (fp8)
    io = nd * (wl.n_q_heads * (wl.d_qk + wl.d_v) * 2 + wl.n_kv_heads * (wl.d_qk + wl.d_v) * (2 + 1))
    dec_bytes_call = dec_bytes / (K * layers) + io
    dec_gbps = dec_bytes_call / (dec_ms * 1e-3) / 1e9
    G = wl.n_q_heads // wl.n_kv_heads
    score_flop = sum(wl.n_kv_heads * 2 * G * min(wl.obs_window, L) * wl.d_qk * max(L - s_r, 0)
                     for L in timed_lengths) / K
    score_tflops = 2 * score_flop / (comp_ms * 1e-3) / 1e12 if comp_ms > 0 else 0.0
    value = nd * K / (t0.elapsed_time(t1) * 1e-3)
    res = {
        "metric": "compressed-KV decode tok/s/GPU + HBM GB/s at 128k; snap_compress latency",
        "value": round(value, 2),
        "unit": "tok/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "launch": ("eager, compression and decode on two streams" if overlap else
                   "eager, one stream" if KC == 1 else
                   f"eager, the layers' compressions over {KC} streams, then the decode step"),
        "config": {"workload": wl.name, "seeds": seed_rule(wl), "layers": layers, "slots": S, "decoded_per_step": nd,
                   "prompt_length_range": list(wl.length_range), "prompt_bank_tokens": Lmax,
                   "budget": B, "sink": wl.sink, "recent": wl.recent, "topk": wl.topk,
                   "obs_window": wl.obs_window, "pool_kernel": wl.pool_kernel, "q_heads": wl.n_q_heads,
                   "kv_heads": wl.n_kv_heads, "d_qk": wl.d_qk, "d_v": wl.d_v, "kv_dtype": wl.kv_dtype,
                   "step": "compress one new prompt into the retired slot (every layer), then one decode "
                           "step of the other slots",
                   "fp8_scales": "amax/448 of the kept rows, set by snap_compress" if args.fp8_scales_from_data
                   else "amax/448 of the layer's prompt bank, set by the harness",
                   "fp8_qk": bool(args.fp8_qk), "kv_reuse": args.kv_reuse, "compress_streams": KC},
        "decode_step_ms_per_call": round(dec_ms, 4),
        "decode_step_hbm_gbps": round(dec_gbps, 1),
        "decode_only_tok_s": round(nd / (dec_ms * layers * 1e-3), 1) if dec_ms > 0 else 0.0,
        "compress_ms_per_layer_call": round(comp_ms, 4),
        "compress_ms_per_seq_layer": round(comp_ms, 4),
        "score_gemm": {"gflop_per_layer_call_one_pass": round(score_flop / 1e9, 2), "passes": 2,
                       "tflops_over_compress_call": round(score_tflops, 1), "peak_tflops": PEAK_BF16_TFLOPS,
                       "mfma_util_lower_bound": round(score_tflops / PEAK_BF16_TFLOPS, 4),
                       "counters": measured_mfma(wl.name)},
        "roofline": {"bound": "hbm",
                     "kernel": "snap_decode_step (fp8 cache: append + split-K attention, one launch) + chunk merge"
                               + (", fp8 Q K^T" if args.fp8_qk else ""),
                     "achieved": round(dec_gbps, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                     "frac": round(dec_gbps / PEAK_HBM_GBPS, 4),
                     "traffic": None if args.fp8_qk else measured_traffic(wl.name),
                     "algorithmic_bytes_per_launch": round(dec_bytes_call)},
        "setup_s": round(t_setup, 1),
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(wl, p, timed_lengths, nd, layers, K, nd * K, value)
    print(json.dumps(res), flush=True)


def run_prefill(args, wl):
    """snap_prefill of one batch of prompts per layer (every sequence of the
    workload, its lengths), prompts resident in HBM."""
    import torch

    import paper_2511_03092_amd as snap
    import synth

    if wl.in_dtype != "bf16" or wl.v_in_k:
        sys.exit(f"--prefill needs a bf16 workload with separate K and V (got {wl.name})")
    layers = args.layers or 1
    n = wl.batch if wl.slots is None else 8
    lengths = synth.draw_lengths(wl, 0, n)
    max_len = max(lengths)
    if args.steps is None:
        args.steps = 10 if max_len * n <= 65536 else 2
    if args.warmup is None:
        args.warmup = 2 if max_len * n <= 65536 else 1
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    DT = {"f32": snap.SNAP_F32, "bf16": snap.SNAP_BF16, "fp8": snap.SNAP_FP8_E4M3}
    p = snap.Params(wl.n_q_heads, wl.n_kv_heads, wl.d_qk, wl.d_v, wl.sink, wl.recent, wl.topk, wl.obs_window,
                    wl.pool_kernel, wl.pool, wl.norm, wl.v_in_k, DT[wl.in_dtype], DT[wl.kv_dtype])
    kvt = {"bf16": torch.bfloat16, "fp8": torch.uint8}[wl.kv_dtype]
    B = p.budget
    t_setup = time.time()
    prompts, caches = [], []
    for l in range(layers):
        prompts.append(synth.prompt_batch(wl, l, lengths, device=dev, max_len=max_len))
        ck = torch.zeros((n, wl.n_kv_heads, B, wl.d_qk), dtype=kvt, device=dev)
        cv = torch.zeros((n, wl.n_kv_heads, B, wl.d_v), dtype=kvt, device=dev)
        ks = vs = None
        if wl.kv_dtype == "fp8":
            k_, v_ = prompts[-1][1], prompts[-1][2]
            ks = torch.stack([k_[b, :, :lengths[b]].float().abs().amax(dim=(1, 2)) for b in range(n)]) / 448.0
            vs = torch.stack([v_[b, :, :lengths[b]].float().abs().amax(dim=(1, 2)) for b in range(n)]) / 448.0
            ks, vs = ks.clamp_min(1e-12).contiguous(), vs.clamp_min(1e-12).contiguous()
        caches.append((ck, cv, ks, vs, snap.cache_struct(ck, cv, ks, vs)))
    # the window queries for the unfused comparison (snap_compress), gathered untimed
    qobs = []
    for l in range(layers):
        q = prompts[l][0]
        qo = torch.zeros((n, wl.n_q_heads, wl.obs_window, wl.d_qk), dtype=q.dtype, device=dev)
        for b, L in enumerate(lengths):
            w = min(wl.obs_window, L)
            qo[b, :, wl.obs_window - w:] = q[b, :, L - w:L]
        qobs.append(qo)
    pos = torch.zeros((n,), dtype=torch.int32, device=dev)
    ntop = torch.zeros((n,), dtype=torch.int32, device=dev)
    slots = torch.arange(n, dtype=torch.int32, device=dev)
    lens = torch.tensor(lengths, dtype=torch.int32, device=dev)
    ws = snap.workspace(snap.snap_prefill_workspace(p, n, max_len), dev)
    wsc = snap.workspace(snap.snap_compress_workspace(p, n, max_len), dev)
    out = torch.empty((n, wl.n_q_heads, max_len, wl.d_v), dtype=torch.bfloat16, device=dev)
    torch.cuda.synchronize()
    t_setup = time.time() - t_setup
    stream = torch.cuda.current_stream()
    sptr = stream.cuda_stream
    if args.copy_calibration:
        copy_calibration(torch, args.copy_calibration, dev)

    def fused():
        for l in range(layers):
            q, k, v = prompts[l]
            snap.snap_prefill(p, caches[l][4], pos, ntop, slots, lens, q, k, v, out, ws, stream=sptr)

    def attn_only():
        for l in range(layers):
            q, k, v = prompts[l]
            snap.snap_prefill_attn(p, lens, q, k, v, out, ws, stream=sptr)

    def unfused_compress():
        for l in range(layers):
            _, k, v = prompts[l]
            snap.snap_compress(p, caches[l][4], pos, ntop, slots, lens, qobs[l], k, v, wsc, stream=sptr)

    for _ in range(args.warmup):
        fused()
        attn_only()
        unfused_compress()
    torch.cuda.synchronize()
    # the three are interleaved step by step (clock drift over the run falls
    # on all three alike); events bracket whole calls only
    evs = []
    torch.cuda.synchronize()
    for _ in range(args.steps):
        e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        e[0].record(stream)
        fused()          # the reported step: snap_prefill, every layer
        e[1].record(stream)
        attn_only()      # the attention launch alone
        e[2].record(stream)
        unfused_compress()
        e[3].record(stream)
        evs.append(e)
    torch.cuda.synchronize()
    ms_step = sum(e[0].elapsed_time(e[1]) for e in evs) / args.steps
    ms_attn = sum(e[1].elapsed_time(e[2]) for e in evs) / args.steps / layers
    ms_comp = sum(e[2].elapsed_time(e[3]) for e in evs) / args.steps / layers
    ms_layer = ms_step / layers
    tokens = sum(lengths)
    # algorithmic flops of the causal attention: per row i, (i+1) keys x (2*d_qk + 2*d_v)
    flop = sum(wl.n_q_heads * L * (L + 1) / 2 * (2 * wl.d_qk + 2 * wl.d_v) for L in lengths)
    tflops = flop / (ms_attn * 1e-3) / 1e12
    value = tokens * layers / (ms_step * 1e-3) / layers
    res = {
        "metric": "prefill attention + SnapKV compression (snap_prefill): prompt tok/s per layer",
        "value": round(value, 1),
        "unit": "tok/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "launch": "eager",
        "config": {"workload": wl.name, "seeds": seed_rule(wl), "layers": layers, "sequences": n, "prompt_lengths": lengths,
                   "q_heads": wl.n_q_heads, "kv_heads": wl.n_kv_heads, "d_qk": wl.d_qk, "d_v": wl.d_v,
                   "sink": wl.sink, "recent": wl.recent, "topk": wl.topk, "obs_window": wl.obs_window,
                   "pool_kernel": wl.pool_kernel, "kv_dtype": wl.kv_dtype},
        "prefill_ms_per_layer_call": round(ms_layer, 4),
        "attention_ms_per_layer_call": round(ms_attn, 4),
        # the compression inside snap_prefill is about 1% of the call: this
        # difference of two whole-call timings carries their spread as well
        "prefill_minus_attention_ms_per_layer_call": round(ms_layer - ms_attn, 4),
        "unfused_compress_ms_per_layer_call": round(ms_comp, 4),
        "roofline": {"bound": "mfma", "kernel": "prefill_attn (+ vt_transpose), timed as snap_prefill_attn",
                     "achieved": round(tflops, 1), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(tflops / PEAK_BF16_TFLOPS, 4),
                     "traffic": measured_traffic("prefill:" + wl.name),
                     "algorithmic_flops_per_launch": flop,
                     "mfma_counters": measured_mfma("prefill:" + wl.name)},
        "setup_s": round(t_setup, 1),
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline_prefill(wl, p, lengths, layers, value)
    print(json.dumps(res), flush=True)


def cpu_model():
    """The host CPU's model name (/proc/cpuinfo), or None where it is not readable."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_threads():
    """Threads for the oracle baseline: the CPUs this process may run on, at
    most 16 (a GPU's CPU share on the machines this runs on), and the counts
    behind that choice for the report."""
    try:
        avail = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        avail = os.cpu_count() or 1
    T = max(1, min(avail, 16))
    return T, {"host_logical_cpus": os.cpu_count(), "affinity_cpus": avail, "threads_used": T,
               "thread_cap": "16: one GPU's CPU share"}


def cpu_baseline_prefill(wl, p, lengths, layers, gpu_value, budget_s=10.0):
    """The fp64 oracle's causal attention on the host's cores, on a bounded
    sample: the last rows of one query head at the longest prompt (each row
    needs all of its keys), rows added until about budget_s of one-thread
    work; then the same rows of T heads on T threads at once.  Extrapolated
    by flops to the attention of every head and position of every prompt and
    layer; `value` is the T-thread rate in prompt tokens per second per
    layer."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    import oracle
    import synth

    T, cpus = cpu_threads()
    op = oracle.Params(p.n_q_heads, p.n_kv_heads, p.d_qk, p.d_v, p.sink, p.recent, p.topk, p.obs_window,
                       p.pool_kernel, p.pool, p.norm, bool(p.v_in_k), p.sm_scale)
    L = max(lengths)
    q, k, v = synth.prompt_batch(wl, 0, [L], device="cpu")
    kc, vc = oracle.f64(k[0, 0]), oracle.f64(v[0, 0])
    qh = [oracle.f64(q[0, h]) for h in range(min(T, p.n_q_heads))]

    def rows(h, i0, i1):
        qq = np.zeros((1, L, p.d_qk))
        qq[0, i0:i1] = qh[h % len(qh)][i0:i1]
        oracle.prefill_attn_group(op, L, qq, kc, vc, rows=(i0, i1))

    nrow, t1 = 8, 0.0
    while True:
        t = time.time()
        rows(0, L - nrow, L)
        t1 = time.time() - t
        if t1 >= budget_s / 4 or nrow >= L:
            break
        nrow = min(L, nrow * 4)
    with ThreadPoolExecutor(T) as ex:
        t = time.time()
        list(ex.map(lambda h: rows(h, L - nrow, L), range(T)))
        tT = time.time() - t
    macs_row = lambda i: (i + 1) * (p.d_qk + p.d_v)
    sample_macs = sum(macs_row(i) for i in range(L - nrow, L))
    total_macs = sum(p.n_q_heads * Lb * (Lb + 1) / 2 * (p.d_qk + p.d_v) for Lb in lengths)
    rate1 = sample_macs / t1
    rateT = T * sample_macs / tT
    tokens = sum(lengths)
    val1 = tokens / (total_macs / rate1)
    valT = tokens / (total_macs / rateT)
    return {"value": float(f"{valT:.6g}"), "unit": "tok/s", "cores": T, "kind": "oracle",
            "cpu_model": cpu_model(), "cpus": cpus, "single_thread_value": float(f"{val1:.6g}"),
            "sample": (f"causal attention rows {L - nrow}..{L - 1} of one head at L={L} (fp64 oracle): "
                       f"{t1:.2f} s on one thread, the same rows of {T} heads on {T} threads in {tT:.2f} s; "
                       f"extrapolated by multiply-adds to every head and position of {len(lengths)} prompt(s), "
                       f"per layer (the compression's oracle cost is not included)"),
            "gpu_over_cpu": float(f"{gpu_value / valT:.4g}")}


def cpu_baseline(wl, p, comp_lengths, dec_seqs, layers, dsteps, tokens, gpu_value, dec_budget_s=1.0):
    """The fp64 oracle on the host's cores, on a bounded sample of the same
    workload: compress units (one sequence x one KV head) at the longest
    prompt and decode units (one sequence x one KV head x one step) over the
    cache one of them built, first on one thread, then on T threads at once
    (T = the cores available, at most 16; independent units, the oracle's C
    calls run in parallel).  Extrapolated by unit counts to the timed work:
    every prompt in comp_lengths compressed (scaled by its length) and dsteps
    decode steps of dec_seqs sequences, every layer, for `tokens` decoded
    tokens.  `value` is the T-thread rate; the one-thread rate is beside it."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    import oracle
    import synth

    T, cpus = cpu_threads()
    op = oracle.Params(p.n_q_heads, p.n_kv_heads, p.d_qk, p.d_v, p.sink, p.recent, p.topk, p.obs_window,
                       p.pool_kernel, p.pool, p.norm, bool(p.v_in_k), p.sm_scale)
    L = max(comp_lengths)
    q, k, v = synth.prefill(wl, 0, 0, L, device="cpu")
    G = op.group
    heads = [(oracle.f64(q[g * G:(g + 1) * G]), oracle.f64(k[g]), None if v is None else oracle.f64(v[g]))
             for g in range(p.n_kv_heads)]

    def comp_unit(i):
        qg, kg, vg = heads[i % p.n_kv_heads]
        return oracle.compress_group(op, L, qg, kg, vg)

    t = time.time()
    res = comp_unit(0)
    t_comp1 = time.time() - t
    qd = np.random.default_rng(0).normal(size=(G, p.d_qk))

    def dec_units(n):
        for _ in range(n):
            oracle.decode_attn_group(op, L, len(res.sel), qd, res.cache_k, res.cache_v)

    n_dec, t_all = 0, 0.0
    while t_all < dec_budget_s and n_dec < 4096:
        t = time.time()
        dec_units(1)
        t_all += time.time() - t
        n_dec += 1
    t_dec1 = t_all / n_dec
    with ThreadPoolExecutor(T) as ex:
        t = time.time()
        list(ex.map(comp_unit, range(T)))
        t_compT = (time.time() - t) / T
        per = max(1, n_dec // 2)
        t = time.time()
        list(ex.map(dec_units, [per] * T))
        t_decT = (time.time() - t) / (T * per)
    units_comp = layers * len(comp_lengths) * p.n_kv_heads
    units_dec = layers * dec_seqs * p.n_kv_heads * dsteps
    scale = sum(Lb / L for Lb in comp_lengths) * layers * p.n_kv_heads
    val1 = tokens / (t_comp1 * scale + t_dec1 * units_dec)
    valT = tokens / (t_compT * scale + t_decT * units_dec)
    return {"value": float(f"{valT:.6g}"), "unit": "tok/s", "cores": T, "kind": "oracle",
            "cpu_model": cpu_model(), "cpus": cpus, "single_thread_value": float(f"{val1:.6g}"),
            "sample": (f"compress units (1 sequence x 1 KV head, L={L}): 1 alone at {t_comp1:.2f} s, then {T} "
                       f"on {T} threads at {t_compT:.2f} s each; decode units (1 sequence x 1 KV head x 1 "
                       f"step): {n_dec} alone at {t_dec1 * 1e3:.1f} ms, then {T * per} on {T} threads at "
                       f"{t_decT * 1e3:.2f} ms each; extrapolated to {units_comp} compress units (scaled by "
                       f"length) and {units_dec} decode units for {tokens} tokens"),
            "gpu_over_cpu": float(f"{gpu_value / valT:.4g}")}


# The other workloads, timed after the headline one by the default run (each
# in a child process of its own, once the headline run's memory is freed), so
# that one plain `python3 bench.py` measures every configuration: the GQA
# batch, continuous batching, the launch-bound one-layer decode (as a HIP
# graph) and the prefill attention + fused compression.
OTHER_RUNS = [
    ["--workload", "llama8b-32layer-b8-128k", "--steps", "1", "--warmup", "1"],
    ["--workload", "cb-fp8-llama8b-32slot"],
    ["--workload", "llama8b-1layer-32k", "--graph"],
    ["--prefill"],
]
OTHER_KEYS = ["value", "unit", "ms_per_step", "steps", "warmup", "launch", "decode_step_ms_per_call",
              "decode_step_hbm_gbps", "compress_ms_per_layer_call", "compress_ms_per_seq_layer",
              "attention_ms_per_layer_call", "prefill_ms_per_layer_call"]


def wants_others(args) -> bool:
    return (args.workload is None and not args.prefill and not args.no_others and args.layers is None
            and args.decode_steps is None and not args.copy_calibration)


def run_others(timeout_s: float = 300.0):
    out = []
    for extra in OTHER_RUNS:
        cmd = [sys.executable, os.path.abspath(__file__), "--no-cpu-baseline", "--no-others"] + extra
        print("[bench] other workload:", " ".join(extra), file=sys.stderr, flush=True)
        t0 = time.time()
        rec = {"args": " ".join(extra)}
        try:
            r = subprocess.run(cmd, capture_output=True, text=True, timeout=timeout_s)
            lines = [x for x in r.stdout.splitlines() if x.startswith("{")]
            if r.returncode != 0 or not lines:
                rec["error"] = f"exit status {r.returncode}"
                rec["stderr_tail"] = r.stderr[-400:]
            else:
                d = json.loads(lines[-1])
                rec["workload"] = d["config"]["workload"]
                rec.update({k: d[k] for k in OTHER_KEYS if k in d})
                rf = d.get("roofline") or {}
                rec["roofline"] = {k: rf[k] for k in ("bound", "achieved", "peak", "unit", "frac") if k in rf}
        except subprocess.TimeoutExpired:
            rec["error"] = f"no result within {timeout_s:.0f} s"
        rec["wall_s"] = round(time.time() - t0, 1)
        out.append(rec)
    return out


if __name__ == "__main__":
    args = parse()
    others = wants_others(args)  # before main() fills in the default workload
    res = main(args)
    if res is not None:  # the decode driver's line (the other drivers print their own)
        if others:
            import gc

            import torch
            gc.collect()
            torch.cuda.synchronize()
            torch.cuda.empty_cache()
            res["other_workloads"] = run_others()
        print(json.dumps(res), flush=True)
