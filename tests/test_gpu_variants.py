"""GPU parity for every kernel configuration the C ABI accepts beyond the
benchmark workloads: each case compresses a ragged batch into some slots of a
canary-filled cache, checks selection, pooled scores and cache bytes against
the fp64 oracle (untouched slots must keep the canary), refills every row
decode must not read with the canary, then decodes across ring wraps with
the two-call path (snap_cache_append + snap_decode_attn) on even steps and
snap_decode_step on odd ones, each checked against the oracle on the GPU's
cache and end to end against the oracle's own cache.

Which kernels each case reaches (csrc names):
  d64 bf16 / fp8 caches      score_pass<bf16, D=64> (both passes),
                             decode_generic<bf16 / fp8>, append<bf16, fp8>
  latent-style caches at     assemble without a V input, decode_generic with
  d 64 / 128 (v_in_k)        values read from the key rows, fp32 and fp8
  wide windows (G*w > 128)   the eight-wave score passes at D = 64 and 128
  G = 1, G = 3               score rows that leave waves empty or ragged
  latent 576, w = 16         the four-wave 576-wide score passes
  latent fp8                 fp8 latent assembly (given and data scales),
                             decode_mla<fp8>
  *-stream                   kv_reuse = SNAP_KV_STREAM: the streaming-load
                             instantiations of decode_mfma (bf16, fp8),
                             decode_mla_lds and decode_mla<fp8>, which the
                             default hint picks only for calls of 128 MiB and
                             more (the full-size tests)

Every case prints what names it before touching the GPU.
"""
import pytest
import torch

import paper_2511_03092_amd as snap
import synth
from snaphelp import TOL, params_of, run_case

pytestmark = pytest.mark.gpu

_G4 = synth.Workload("var-gqa", 14, 8, 2, 64, 64, False, 4, 16, 200, 32, 7, "bf16", "bf16", layers=1, batch=2,
                     length=None, length_range=(500, 4000), decode_steps=40, rope=True, plant_frac=0.01)
# Latent-style caches hold each token's values inside its key row, so they
# follow the latent workload's input recipe (N(0, 1) rows, no planted heavy
# hitters, no rotary encoding): a planted key, of norm 4*sqrt(d), would also
# be a value of that norm, and outputs that large are not what the absolute
# decode bound is set for.
_G4_LATENT = synth.small(_G4, v_in_k=True, rope=False, plant_frac=None)
_LAT = synth.small(synth.WORKLOADS["mla-8head-61layer-b16-128k"], name="var-latent", cfg_id=15, recent=64, topk=512)

# name: (workload, params overrides, lengths, slots, n_slots, steps, check_every, out dtype)
CASES = {
    "d64-bf16": (_G4, {}, [3001, 777], [1, 3], 4, 40, 1, torch.bfloat16),
    "d64-fp8-given": (synth.small(_G4, kv_dtype="fp8"), {}, [3001, 777], [2, 0], 4, 40, 1, torch.bfloat16),
    "d64-fp8-amax": (synth.small(_G4, kv_dtype="fp8"), {"fp8_scales": snap.SNAP_FP8_SCALES_AMAX},
                     [2500, 1200], [0, 3], 4, 40, 1, torch.float32),
    "d128-latent-style-bf16": (synth.small(_G4_LATENT, d_qk=128, d_v=128), {}, [3001, 900], [1, 2], 3, 40, 1,
                               torch.bfloat16),
    "d64-latent-style-fp8": (synth.small(_G4_LATENT, kv_dtype="fp8"), {}, [2000, 1500], [0, 2], 3, 40, 1,
                             torch.bfloat16),
    "d128-latent-style-f32": (synth.small(_G4_LATENT, d_qk=128, d_v=128, in_dtype="f32", kv_dtype="f32"), {},
                              [2100, 333], [1, 0], 2, 40, 1, torch.float32),
    "wide-d64-g8": (synth.small(_G4, n_q_heads=16), {}, [3001, 1000], [3, 1], 4, 24, 2, torch.bfloat16),
    "wide-d128-g8-row-avg": (synth.small(_G4, n_q_heads=16, d_qk=128, d_v=128, norm=synth.NORM_ROW,
                                         pool=synth.POOL_AVG), {}, [3001, 1000], [0, 1], 2, 24, 2, torch.bfloat16),
    "wide-d128-g16-w16": (synth.small(_G4, n_q_heads=32, d_qk=128, d_v=128, obs_window=16), {}, [2600, 1700],
                          [1, 0], 2, 24, 2, torch.bfloat16),
    "mha-g1-d128": (synth.small(_G4, n_q_heads=2, d_qk=128, d_v=128), {}, [3001, 800], [0, 1], 2, 24, 2,
                    torch.bfloat16),
    "g3-60-rows-d128": (synth.small(_G4, n_q_heads=6, d_qk=128, d_v=128, obs_window=20), {}, [3001, 800], [1, 0],
                        2, 24, 2, torch.bfloat16),
    "latent-576-w16": (synth.small(_LAT, obs_window=16), {}, [5000, 2100], [0, 1], 2, 80, 8, torch.bfloat16),
    "latent-fp8-given": (synth.small(_LAT, kv_dtype="fp8"), {}, [6000, 2500], [2, 0], 3, 80, 8, torch.bfloat16),
    "latent-fp8-amax": (synth.small(_LAT, kv_dtype="fp8"), {"fp8_scales": snap.SNAP_FP8_SCALES_AMAX},
                        [5000, 700], [1, 2], 3, 80, 8, torch.bfloat16),
    "gqa-d128-bf16-stream": (synth.small(_G4, d_qk=128, d_v=128), {"kv_reuse": snap.SNAP_KV_STREAM},
                             [3001, 800], [1, 0], 2, 40, 2, torch.bfloat16),
    "gqa-d128-fp8-stream": (synth.small(_G4, d_qk=128, d_v=128, kv_dtype="fp8"), {"kv_reuse": snap.SNAP_KV_STREAM},
                            [2700, 1300], [0, 2], 3, 40, 2, torch.bfloat16),
    "latent-576-stream": (_LAT, {"kv_reuse": snap.SNAP_KV_STREAM}, [5000, 2100], [1, 0], 2, 80, 8, torch.bfloat16),
    "latent-fp8-stream": (synth.small(_LAT, kv_dtype="fp8"), {"kv_reuse": snap.SNAP_KV_STREAM}, [6000, 2500],
                          [0, 2], 3, 80, 8, torch.bfloat16),
}


@pytest.mark.parametrize("name", list(CASES))
def test_abi_variant(name):
    wl, over, lengths, slots, n_slots, steps, every, out_dtype = CASES[name]
    p = params_of(wl, **over)
    tol = TOL[wl.kv_dtype]
    given = wl.kv_dtype == "fp8" and p.fp8_scales == snap.SNAP_FP8_SCALES_GIVEN
    print(f"\n[case] {name}: Hq {p.n_q_heads} Hkv {p.n_kv_heads} d ({p.d_qk},{p.d_v}) v_in_k {int(p.v_in_k)} "
          f"in {wl.in_dtype} cache {wl.kv_dtype} fp8_scales {p.fp8_scales} window {p.obs_window} "
          f"norm {p.norm} pool {p.pool} lengths {lengths} -> slots {slots} of {n_slots}, {steps} steps",
          flush=True)
    run_case(wl, p, lengths, slots, n_slots, steps, out_dtype, tol, check_every=every, fp8_scales=given,
             fused="alt")
