// abi.hip -- the extern "C" entry points of libsnapstream: host-side argument
// validation, workspace sizing and dispatch to the kernel launchers.  Nothing
// here allocates device memory or synchronises, and every validation runs
// before anything touches the device (the one device query, of
// snap_decode_step_noalloc's scratch address, follows its checks), so every
// validation path can run on a host without a GPU.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>

#include "snap_internal.h"

namespace snap {

static thread_local char g_err[512];

void set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
}

static snap_status fail(snap_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return s;
}

static bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Largest second launch-grid dimension (workgroups along y): per-(sequence,
// KV head) and per-(sequence, query head) grids must fit it.
constexpr int kMaxGridY = 65535;

// Parameter checks shared by every call.
static snap_status check_params(const snap_params* p) {
  if (!p) return fail(SNAP_ERR_INVALID_ARG, "params is NULL");
  if (p->n_q_heads < 1 || p->n_kv_heads < 1 || p->n_q_heads % p->n_kv_heads)
    return fail(SNAP_ERR_INVALID_ARG, "n_q_heads (%d) must be a positive multiple of n_kv_heads (%d)",
                p->n_q_heads, p->n_kv_heads);
  const int G = p->n_q_heads / p->n_kv_heads;
  if (G > 16) return fail(SNAP_ERR_UNSUPPORTED, "at most 16 query heads per KV head (got %d)", G);
  if (p->sink < 0 || p->recent < 1 || p->topk < 0)
    return fail(SNAP_ERR_INVALID_ARG, "need sink >= 0, recent >= 1, topk >= 0 (got %d, %d, %d)", p->sink,
                p->recent, p->topk);
  if ((long long)p->sink + p->recent + p->topk > (1 << 24))
    return fail(SNAP_ERR_INVALID_ARG, "budget sink+recent+topk exceeds 2^24 rows");
  if (p->obs_window < 1) return fail(SNAP_ERR_INVALID_ARG, "obs_window must be >= 1");
  if (p->pool_kernel < 1 || p->pool_kernel > 63 || (p->pool_kernel & 1) == 0)
    return fail(SNAP_ERR_INVALID_ARG, "pool_kernel must be odd in [1, 63] (got %d)", p->pool_kernel);
  if (p->pool != SNAP_POOL_MAX && p->pool != SNAP_POOL_AVG) return fail(SNAP_ERR_INVALID_ARG, "unknown pool type");
  if (p->norm != SNAP_NORM_CAND && p->norm != SNAP_NORM_ROW) return fail(SNAP_ERR_INVALID_ARG, "unknown norm");
  if (!isfinite(p->sm_scale)) return fail(SNAP_ERR_INVALID_ARG, "sm_scale must be finite");
  // a positive scale must keep scale * log2(e) a normal fp32 value: the score
  // kernels form every logit from it and its remainder
  if (p->sm_scale > 0.f && p->sm_scale < 1e-30f)
    return fail(SNAP_ERR_INVALID_ARG, "sm_scale must be <= 0 (the default) or at least 1e-30");
  if (p->fp8_scales != SNAP_FP8_SCALES_GIVEN && p->fp8_scales != SNAP_FP8_SCALES_AMAX)
    return fail(SNAP_ERR_INVALID_ARG, "unknown fp8_scales mode");
  if (p->fp8_qk != 0 && p->fp8_qk != 1) return fail(SNAP_ERR_INVALID_ARG, "fp8_qk must be 0 or 1");
  if (p->kv_reuse != SNAP_KV_AUTO && p->kv_reuse != SNAP_KV_STREAM && p->kv_reuse != SNAP_KV_KEEP)
    return fail(SNAP_ERR_INVALID_ARG, "unknown kv_reuse hint");
  if (p->fp8_qk && !(p->kv_dtype == SNAP_FP8_E4M3 && p->in_dtype == SNAP_BF16 && !p->v_in_k && p->d_qk == 128 &&
                     p->d_v == 128))
    return fail(SNAP_ERR_UNSUPPORTED, "fp8_qk needs bf16 inputs, a GQA fp8 cache and d_qk = d_v = 128");
  const bool dims_ok = (p->d_qk == 64 && p->d_v == 64) || (p->d_qk == 128 && p->d_v == 128) ||
                       (p->d_qk == 576 && p->d_v == 512);
  if (!dims_ok) return fail(SNAP_ERR_UNSUPPORTED, "(d_qk, d_v) must be (64,64), (128,128) or (576,512)");
  if (p->v_in_k != 0 && p->v_in_k != 1) return fail(SNAP_ERR_INVALID_ARG, "v_in_k must be 0 or 1");
  if (p->d_qk == 576 && !p->v_in_k) return fail(SNAP_ERR_UNSUPPORTED, "576/512 is supported as a latent (v_in_k) cache");
  if (p->in_dtype == SNAP_F32) {
    if (p->kv_dtype != SNAP_F32) return fail(SNAP_ERR_UNSUPPORTED, "fp32 inputs need an fp32 cache");
    if (p->d_qk > 128) return fail(SNAP_ERR_UNSUPPORTED, "fp32 inputs support d_qk <= 128");
  } else if (p->in_dtype == SNAP_BF16) {
    if (p->kv_dtype != SNAP_BF16 && p->kv_dtype != SNAP_FP8_E4M3)
      return fail(SNAP_ERR_UNSUPPORTED, "bf16 inputs need a bf16 or fp8 cache");
  } else {
    return fail(SNAP_ERR_INVALID_ARG, "in_dtype must be SNAP_F32 or SNAP_BF16");
  }
  const long rows = (long)G * p->obs_window;
  const long rows_max = p->in_dtype == SNAP_F32 ? 128 : 256;
  if (rows > rows_max)
    return fail(SNAP_ERR_UNSUPPORTED, "G * obs_window = %ld exceeds %ld score rows per KV head", rows, rows_max);
  return SNAP_OK;
}

static snap_status check_cache(const snap_params* p, const snap_cache* c) {
  if (!c) return fail(SNAP_ERR_INVALID_ARG, "cache is NULL");
  if (c->n_slots < 1) return fail(SNAP_ERR_INVALID_ARG, "cache n_slots must be >= 1");
  if (!c->k || !aligned16(c->k)) return fail(SNAP_ERR_INVALID_ARG, "cache k is NULL or not 16-byte aligned");
  if (!p->v_in_k && (!c->v || !aligned16(c->v)))
    return fail(SNAP_ERR_INVALID_ARG, "cache v is NULL or not 16-byte aligned");
  if (p->kv_dtype == SNAP_FP8_E4M3 && (!c->k_scale || (!p->v_in_k && !c->v_scale)))
    return fail(SNAP_ERR_INVALID_ARG, "an fp8 cache needs k_scale and v_scale");
  return SNAP_OK;
}

}  // namespace snap

using namespace snap;

extern "C" {

const char* snap_status_str(snap_status s) {
  switch (s) {
    case SNAP_OK: return "ok";
    case SNAP_ERR_INVALID_ARG: return "invalid argument";
    case SNAP_ERR_UNSUPPORTED: return "unsupported configuration";
    case SNAP_ERR_WORKSPACE: return "workspace missing or too small";
    case SNAP_ERR_HIP: return "HIP launch error";
  }
  return "unknown status";
}

const char* snap_last_error(void) { return g_err; }

size_t snap_compress_workspace(const snap_params* p, int32_t n_seq, int32_t max_len) {
  if (check_params(p) != SNAP_OK || n_seq < 0 || max_len < 1) return 0;
  return compress_geometry(*p, n_seq, max_len).compress_bytes;
}

size_t snap_decode_workspace(const snap_params* p, int32_t n) {
  if (check_params(p) != SNAP_OK || n < 0) return 0;
  return decode_geometry(*p, n).decode_bytes;
}

snap_status snap_compress(const snap_params* p, const snap_cache* cache, int32_t* pos, int32_t* n_topk,
                          int32_t n_seq, const int32_t* slot_ids, const int32_t* lengths, int32_t max_len,
                          const void* q_obs, const void* k, const void* v, int32_t* sel_out, float* pooled_out,
                          void* workspace, size_t ws_bytes, void* stream) {
  g_err[0] = 0;
  snap_status st = check_params(p);
  if (st != SNAP_OK) return st;
  if ((st = check_cache(p, cache)) != SNAP_OK) return st;
  if (n_seq < 0) return fail(SNAP_ERR_INVALID_ARG, "n_seq must be >= 0");
  if (n_seq == 0) return SNAP_OK;
  if (max_len < 1 || max_len > (1 << 28)) return fail(SNAP_ERR_INVALID_ARG, "max_len must be in [1, 2^28]");
  if ((long long)n_seq * p->n_kv_heads > kMaxGridY)
    return fail(SNAP_ERR_UNSUPPORTED, "n_seq * n_kv_heads must be at most %d", kMaxGridY);
  if (!pos || !n_topk || !slot_ids || !lengths) return fail(SNAP_ERR_INVALID_ARG, "pos/n_topk/slot_ids/lengths NULL");
  if (!q_obs || !aligned16(q_obs)) return fail(SNAP_ERR_INVALID_ARG, "q_obs is NULL or not 16-byte aligned");
  if (!k || !aligned16(k)) return fail(SNAP_ERR_INVALID_ARG, "k is NULL or not 16-byte aligned");
  if (!p->v_in_k && (!v || !aligned16(v))) return fail(SNAP_ERR_INVALID_ARG, "v is NULL or not 16-byte aligned");
  if (p->v_in_k && v) return fail(SNAP_ERR_INVALID_ARG, "v must be NULL for a latent (v_in_k) cache");
  if ((sel_out && !aligned16(sel_out)) || (pooled_out && !aligned16(pooled_out)))
    return fail(SNAP_ERR_INVALID_ARG, "sel_out/pooled_out must be 16-byte aligned");
  const size_t need = compress_geometry(*p, n_seq, max_len).compress_bytes;
  if (!workspace || ((uintptr_t)workspace & 255u) || ws_bytes < need)
    return fail(SNAP_ERR_WORKSPACE, "workspace needs %zu bytes, 256-byte aligned (got %zu)", need, ws_bytes);
  st = launch_compress(*p, *cache, pos, n_topk, n_seq, slot_ids, lengths, max_len, q_obs, k, v, sel_out, pooled_out,
                       workspace, (hipStream_t)stream);
  if (st == SNAP_ERR_HIP) set_error("kernel launch failed: %s", hipGetErrorString(hipGetLastError()));
  return st;
}

size_t snap_prefill_workspace(const snap_params* p, int32_t n_seq, int32_t max_len) {
  if (check_params(p) != SNAP_OK || n_seq < 0 || max_len < 1) return 0;
  return prefill_geometry(*p, n_seq, max_len).prefill_bytes;
}

// Checks shared by snap_prefill and snap_prefill_attn.
static snap_status check_prefill(const snap_params* p, int32_t n_seq, const int32_t* lengths, int32_t max_len,
                                 const void* q, const void* k, const void* v, void* out, void* workspace,
                                 size_t ws_bytes) {
  if (p->in_dtype != SNAP_BF16) return fail(SNAP_ERR_UNSUPPORTED, "snap_prefill takes bf16 inputs");
  if (p->v_in_k || p->d_qk != p->d_v || (p->d_qk != 64 && p->d_qk != 128))
    return fail(SNAP_ERR_UNSUPPORTED, "snap_prefill supports d_qk == d_v in {64, 128} with a separate V");
  const int G = p->n_q_heads / p->n_kv_heads;
  if (G != 1 && G != 2 && G != 4 && G != 8 && G != 16)
    return fail(SNAP_ERR_UNSUPPORTED, "snap_prefill supports 1, 2, 4, 8 or 16 query heads per KV head (got %d)", G);
  if (n_seq < 0) return fail(SNAP_ERR_INVALID_ARG, "n_seq must be >= 0");
  if (n_seq == 0) return SNAP_OK;
  if (max_len < 1 || max_len > (1 << 28)) return fail(SNAP_ERR_INVALID_ARG, "max_len must be in [1, 2^28]");
  const long long groups = (long long)n_seq * p->n_kv_heads;
  const long long positions = 256 / G;  // query positions per attention workgroup
  if (groups > kMaxGridY || 8 * ((groups + 7) / 8) * ((max_len + positions - 1) / positions) > 0x7fffffffLL)
    return fail(SNAP_ERR_UNSUPPORTED, "n_seq * n_kv_heads (%lld) and max_len (%d) exceed the launch grid", groups,
                max_len);
  if (!lengths) return fail(SNAP_ERR_INVALID_ARG, "lengths is NULL");
  if (!q || !aligned16(q) || !k || !aligned16(k) || !v || !aligned16(v))
    return fail(SNAP_ERR_INVALID_ARG, "q, k and v must be non-NULL and 16-byte aligned");
  if (!out || !aligned16(out)) return fail(SNAP_ERR_INVALID_ARG, "out is NULL or not 16-byte aligned");
  const size_t need = prefill_geometry(*p, n_seq, max_len).prefill_bytes;
  if (!workspace || ((uintptr_t)workspace & 255u) || ws_bytes < need)
    return fail(SNAP_ERR_WORKSPACE, "workspace needs %zu bytes, 256-byte aligned (got %zu)", need, ws_bytes);
  return SNAP_OK;
}

snap_status snap_prefill_attn(const snap_params* p, int32_t n_seq, const int32_t* lengths, int32_t max_len,
                              const void* q, const void* k, const void* v, void* out, void* workspace,
                              size_t ws_bytes, void* stream) {
  g_err[0] = 0;
  snap_status st = check_params(p);
  if (st != SNAP_OK) return st;
  if ((st = check_prefill(p, n_seq, lengths, max_len, q, k, v, out, workspace, ws_bytes)) != SNAP_OK) return st;
  if (n_seq == 0) return SNAP_OK;
  st = launch_prefill_attn(*p, n_seq, lengths, max_len, q, k, v, out, false, workspace, (hipStream_t)stream);
  if (st == SNAP_ERR_HIP) set_error("kernel launch failed: %s", hipGetErrorString(hipGetLastError()));
  return st;
}

snap_status snap_prefill(const snap_params* p, const snap_cache* cache, int32_t* pos, int32_t* n_topk, int32_t n_seq,
                         const int32_t* slot_ids, const int32_t* lengths, int32_t max_len, const void* q, const void* k,
                         const void* v, void* out, int32_t* sel_out, float* pooled_out, void* workspace,
                         size_t ws_bytes, void* stream) {
  g_err[0] = 0;
  snap_status st = check_params(p);
  if (st != SNAP_OK) return st;
  if ((st = check_cache(p, cache)) != SNAP_OK) return st;
  if ((st = check_prefill(p, n_seq, lengths, max_len, q, k, v, out, workspace, ws_bytes)) != SNAP_OK) return st;
  if (n_seq == 0) return SNAP_OK;
  if (!pos || !n_topk || !slot_ids) return fail(SNAP_ERR_INVALID_ARG, "pos/n_topk/slot_ids NULL");
  if ((sel_out && !aligned16(sel_out)) || (pooled_out && !aligned16(pooled_out)))
    return fail(SNAP_ERR_INVALID_ARG, "sel_out/pooled_out must be 16-byte aligned");
  st = launch_prefill(*p, *cache, pos, n_topk, n_seq, slot_ids, lengths, max_len, q, k, v, out, sel_out, pooled_out,
                      workspace, (hipStream_t)stream);
  if (st == SNAP_ERR_HIP) set_error("kernel launch failed: %s", hipGetErrorString(hipGetLastError()));
  return st;
}

snap_status snap_cache_append(const snap_params* p, const snap_cache* cache, const int32_t* pos, int32_t n,
                              const int32_t* slot_ids, const void* k_new, const void* v_new, void* stream) {
  g_err[0] = 0;
  snap_status st = check_params(p);
  if (st != SNAP_OK) return st;
  if ((st = check_cache(p, cache)) != SNAP_OK) return st;
  if (n < 0) return fail(SNAP_ERR_INVALID_ARG, "n must be >= 0");
  if (n == 0) return SNAP_OK;
  if (!pos || !slot_ids) return fail(SNAP_ERR_INVALID_ARG, "pos/slot_ids NULL");
  if (!k_new || !aligned16(k_new)) return fail(SNAP_ERR_INVALID_ARG, "k_new is NULL or not 16-byte aligned");
  if (!p->v_in_k && (!v_new || !aligned16(v_new)))
    return fail(SNAP_ERR_INVALID_ARG, "v_new is NULL or not 16-byte aligned");
  st = launch_append(*p, *cache, pos, n, slot_ids, k_new, v_new, (hipStream_t)stream);
  if (st == SNAP_ERR_HIP) set_error("kernel launch failed: %s", hipGetErrorString(hipGetLastError()));
  return st;
}

snap_status snap_decode_attn(const snap_params* p, const snap_cache* cache, const int32_t* pos,
                             const int32_t* n_topk, int32_t n, const int32_t* slot_ids, const void* q, void* out,
                             int32_t out_dtype, void* workspace, size_t ws_bytes, void* stream) {
  g_err[0] = 0;
  snap_status st = check_params(p);
  if (st != SNAP_OK) return st;
  if ((st = check_cache(p, cache)) != SNAP_OK) return st;
  if (n < 0) return fail(SNAP_ERR_INVALID_ARG, "n must be >= 0");
  if (n == 0) return SNAP_OK;
  if ((long long)n * p->n_q_heads > kMaxGridY)
    return fail(SNAP_ERR_UNSUPPORTED, "n * n_q_heads must be at most %d", kMaxGridY);
  if (!pos || !n_topk || !slot_ids) return fail(SNAP_ERR_INVALID_ARG, "pos/n_topk/slot_ids NULL");
  if (!q || !aligned16(q)) return fail(SNAP_ERR_INVALID_ARG, "q is NULL or not 16-byte aligned");
  if (!out || !aligned16(out)) return fail(SNAP_ERR_INVALID_ARG, "out is NULL or not 16-byte aligned");
  if (out_dtype != SNAP_F32 && out_dtype != SNAP_BF16) return fail(SNAP_ERR_INVALID_ARG, "out_dtype must be F32 or BF16");
  const size_t need = decode_geometry(*p, n).decode_bytes;
  if (!workspace || ((uintptr_t)workspace & 255u) || ws_bytes < need)
    return fail(SNAP_ERR_WORKSPACE, "workspace needs %zu bytes, 256-byte aligned (got %zu)", need, ws_bytes);
  st = launch_decode(*p, *cache, pos, n_topk, n, slot_ids, q, nullptr, nullptr, out, out_dtype, workspace,
                     (hipStream_t)stream);
  if (st == SNAP_ERR_HIP) set_error("kernel launch failed: %s", hipGetErrorString(hipGetLastError()));
  return st;
}

// Checks of snap_decode_step and snap_decode_step_noalloc except the
// workspace.
static snap_status check_decode_step(const snap_params* p, const snap_cache* cache, const int32_t* pos,
                                     const int32_t* n_topk, int32_t n, const int32_t* slot_ids, const void* q,
                                     const void* k_new, const void* v_new, void* out, int32_t out_dtype) {
  snap_status st = check_params(p);
  if (st != SNAP_OK) return st;
  if ((st = check_cache(p, cache)) != SNAP_OK) return st;
  if (n < 0) return fail(SNAP_ERR_INVALID_ARG, "n must be >= 0");
  if (n == 0) return SNAP_OK;
  if ((long long)n * p->n_q_heads > kMaxGridY)
    return fail(SNAP_ERR_UNSUPPORTED, "n * n_q_heads must be at most %d", kMaxGridY);
  if (!pos || !n_topk || !slot_ids) return fail(SNAP_ERR_INVALID_ARG, "pos/n_topk/slot_ids NULL");
  if (!q || !aligned16(q)) return fail(SNAP_ERR_INVALID_ARG, "q is NULL or not 16-byte aligned");
  if (!k_new || !aligned16(k_new)) return fail(SNAP_ERR_INVALID_ARG, "k_new is NULL or not 16-byte aligned");
  if (!p->v_in_k && (!v_new || !aligned16(v_new)))
    return fail(SNAP_ERR_INVALID_ARG, "v_new is NULL or not 16-byte aligned");
  if (!out || !aligned16(out)) return fail(SNAP_ERR_INVALID_ARG, "out is NULL or not 16-byte aligned");
  if (out_dtype != SNAP_F32 && out_dtype != SNAP_BF16) return fail(SNAP_ERR_INVALID_ARG, "out_dtype must be F32 or BF16");
  return SNAP_OK;
}

snap_status snap_decode_step(const snap_params* p, const snap_cache* cache, const int32_t* pos,
                             const int32_t* n_topk, int32_t n, const int32_t* slot_ids, const void* q,
                             const void* k_new, const void* v_new, void* out, int32_t out_dtype, void* workspace,
                             size_t ws_bytes, void* stream) {
  g_err[0] = 0;
  snap_status st = check_decode_step(p, cache, pos, n_topk, n, slot_ids, q, k_new, v_new, out, out_dtype);
  if (st != SNAP_OK || n == 0) return st;
  const size_t need = decode_geometry(*p, n).decode_bytes;
  if (!workspace || ((uintptr_t)workspace & 255u) || ws_bytes < need)
    return fail(SNAP_ERR_WORKSPACE, "workspace needs %zu bytes, 256-byte aligned (got %zu)", need, ws_bytes);
  st = launch_decode(*p, *cache, pos, n_topk, n, slot_ids, q, k_new, p->v_in_k ? nullptr : v_new, out, out_dtype,
                     workspace, (hipStream_t)stream);
  if (st == SNAP_ERR_HIP) set_error("kernel launch failed: %s", hipGetErrorString(hipGetLastError()));
  return st;
}

snap_status snap_decode_step_noalloc(const snap_params* p, const snap_cache* cache, const int32_t* pos,
                                     const int32_t* n_topk, int32_t n, const int32_t* slot_ids, const void* q,
                                     const void* k_new, const void* v_new, void* out, int32_t out_dtype,
                                     void* stream) {
  g_err[0] = 0;
  snap_status st = check_decode_step(p, cache, pos, n_topk, n, slot_ids, q, k_new, v_new, out, out_dtype);
  if (st != SNAP_OK || n == 0) return st;
  const size_t need = decode_geometry(*p, n).decode_bytes;
  if (need > (size_t)SNAP_NOALLOC_SCRATCH_BYTES)
    return fail(SNAP_ERR_WORKSPACE, "this call needs %zu bytes of scratch; the library's array holds %zu (split the batch)",
                need, (size_t)SNAP_NOALLOC_SCRATCH_BYTES);
  void* scratch = nullptr;
  if ((st = noalloc_scratch(&scratch)) != SNAP_OK) return st;
  st = launch_decode(*p, *cache, pos, n_topk, n, slot_ids, q, k_new, p->v_in_k ? nullptr : v_new, out, out_dtype,
                     scratch, (hipStream_t)stream);
  if (st == SNAP_ERR_HIP) set_error("kernel launch failed: %s", hipGetErrorString(hipGetLastError()));
  return st;
}

snap_status snap_debug_checks(uint32_t* flags, int32_t reset) {
  g_err[0] = 0;
  if (!flags) return fail(SNAP_ERR_INVALID_ARG, "flags is NULL");
  *flags = 0;
#ifdef SNAP_DEBUG_CHECKS
  if (hipDeviceSynchronize() != hipSuccess) return fail(SNAP_ERR_HIP, "hipDeviceSynchronize failed");
  const uint32_t c = debug_flags_compress(reset != 0), d = debug_flags_decode(reset != 0),
                 f = debug_flags_prefill(reset != 0);
  if (c == 0xffffffffu || d == 0xffffffffu || f == 0xffffffffu)
    return fail(SNAP_ERR_HIP, "reading the check words failed");
  *flags = c | d | f;
  return SNAP_OK;
#else
  (void)reset;
  return fail(SNAP_ERR_UNSUPPORTED, "a release build: no device-side checks (build with --debug)");
#endif
}

snap_status snap_advance(int32_t* pos, int32_t n_slots, int32_t n, const int32_t* slot_ids, void* stream) {
  g_err[0] = 0;
  if (n < 0 || n_slots < 1) return fail(SNAP_ERR_INVALID_ARG, "need n >= 0 and n_slots >= 1");
  if (n == 0) return SNAP_OK;
  if (!pos || !slot_ids) return fail(SNAP_ERR_INVALID_ARG, "pos/slot_ids NULL");
  snap_status st = launch_advance(pos, n_slots, n, slot_ids, (hipStream_t)stream);
  if (st == SNAP_ERR_HIP) set_error("kernel launch failed: %s", hipGetErrorString(hipGetLastError()));
  return st;
}

}  // extern "C"
