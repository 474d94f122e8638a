/*
 * snapstream.h -- C ABI of the SnapStream hot path on MI355X (gfx950).
 *
 * SnapStream (arXiv 2511.03092) keeps, per sequence and KV head, a cache of
 * fixed size B = sink + recent + topk rows (Sec. III-A):
 *   rows [0, sink)                 attention-sink tokens (StreamingLLM),
 *   rows [sink, sink+recent)       the rolling window of recent tokens, kept as
 *                                  a ring buffer (Sec. III-B.1),
 *   rows [sink+recent, B)          the top-K tokens chosen by SnapKV at the end
 *                                  of prefill (Sec. III-B.2, Eq. 1-3), followed
 *                                  by zeroed padding rows when fewer exist.
 * The library fills that cache from a padded prefill (snap_compress; or
 * snap_prefill, which also computes the prompt's causal attention and takes
 * the window statistics from it), writes
 * each decoded token into its ring row (snap_cache_append, Sec. III-C), and
 * runs decode attention over the valid rows (snap_decode_attn; snap_decode_step
 * does both for one layer).
 *
 * Conventions shared by every call
 *  - Token positions are 0-based; a prompt of length L holds tokens 0..L-1 and
 *    the first decoded token is at position L.
 *  - Every pointer argument named as a tensor is DEVICE memory owned by the
 *    caller.  The library allocates nothing, frees nothing and never
 *    synchronises; all work is enqueued on `stream` (a hipStream_t, NULL = the
 *    null stream) and the call returns once it is launched.
 *  - Arguments are validated on the host before anything is launched; a
 *    failure returns a non-zero snap_status, launches nothing and leaves a
 *    message for snap_last_error().  A failed launch returns SNAP_ERR_HIP.
 *  - Per-sequence lengths and positions are device data, so a decode step
 *    needs no host round trip.  Device data out of range is handled without
 *    faulting: lengths are clamped to [0, max_len]; a slot id outside
 *    [0, n_slots) makes the call skip that sequence.
 *  - Inputs must not alias the cache.  Calls on disjoint buffers may run
 *    concurrently on different streams.  One exception to disjointness:
 *    snap_compress / snap_prefill calls of different layers for the same
 *    prompt may run concurrently although they share that slot's pos and
 *    n_topk entries, since those calls only write them, with the same values
 *    (L and min(K, |C|)).
 *  - Batch limits of the launch grids: n_seq * n_kv_heads <= 65535
 *    (snap_compress, snap_prefill, snap_prefill_attn) and n * n_q_heads <=
 *    65535 (snap_decode_attn, snap_decode_step); larger calls return
 *    SNAP_ERR_UNSUPPORTED (split the batch).
 */
#ifndef SNAPSTREAM_H
#define SNAPSTREAM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SNAP_OK = 0,
  SNAP_ERR_INVALID_ARG = 1, /* a parameter, pointer or size is invalid     */
  SNAP_ERR_UNSUPPORTED = 2, /* valid, but no kernel for this combination   */
  SNAP_ERR_WORKSPACE = 3,   /* workspace NULL or smaller than the query    */
  SNAP_ERR_HIP = 4          /* the HIP runtime reported an error on launch */
} snap_status;

typedef enum {
  SNAP_F32 = 0,
  SNAP_BF16 = 1,
  SNAP_FP8_E4M3 = 2 /* OCP E4M3 (fn): bias 7, max 448, no inf; cache only */
} snap_dtype;

typedef enum {
  SNAP_POOL_MAX = 0, /* max pooling of the summed attention            */
  SNAP_POOL_AVG = 1  /* average pooling (Eq. 2), zero padding, / kernel */
} snap_pool;

typedef enum {
  SNAP_NORM_CAND = 0, /* softmax over the eviction candidates only (Eq. 3) */
  SNAP_NORM_ROW = 1   /* softmax over the whole causal row [0, i]          */
} snap_norm;

/* Who sets an fp8 cache's per-(slot, KV head) scales. */
typedef enum {
  SNAP_FP8_SCALES_GIVEN = 0, /* the caller, before compress / append           */
  SNAP_FP8_SCALES_AMAX = 1   /* snap_compress: amax / 448 over the rows the
                                compressed cache keeps (sinks, ring, selected;
                                1 when they are all zero), for K and V apart;
                                tokens appended later saturate at +-448 codes */
} snap_fp8_scales;

/* How decode reads the cache rows: a load hint.  Results agree to rounding
 * (under streaming loads the bf16 GQA kernel adds the dot products' 8-element
 * pieces in another order; the other kernels give the same bits). */
typedef enum {
  SNAP_KV_AUTO = 0,   /* streaming when the call's cache rows at the full
                         budget reach 128 MiB, cached loads otherwise          */
  SNAP_KV_STREAM = 1, /* non-temporal loads: the rows will not be read again
                         before the last-level cache (256 MB) has turned over,
                         e.g. many layers or large batches between two reads  */
  SNAP_KV_KEEP = 2    /* ordinary loads: the cache fits in the last-level cache
                         and is read again soon (a one-layer model, a small
                         batch)                                                 */
} snap_kv_reuse;

/* The method's hyper-parameters (Sec. III, Table 6's names). */
typedef struct {
  int32_t n_q_heads;   /* query heads; a multiple of n_kv_heads                 */
  int32_t n_kv_heads;  /* KV heads (1 for a shared latent cache)                */
  int32_t d_qk;        /* query/key width: 64, 128 or 576                        */
  int32_t d_v;         /* value width: 64, 128 or 512                            */
  int32_t v_in_k;      /* 1: latent cache (Sec. VI) -- one stored row per token
                          of width d_qk whose first d_v dims are the value; there
                          is no separate V input or V cache                       */
  int32_t sink;        /* L_sink >= 0                                            */
  int32_t recent;      /* L_recent >= 1 (ring length)                            */
  int32_t topk;        /* K >= 0                                                 */
  int32_t obs_window;  /* L_obs >= 1: queries of the last L_obs prompt tokens    */
  int32_t pool_kernel; /* odd, 1..63                                             */
  int32_t pool;        /* snap_pool                                              */
  int32_t norm;        /* snap_norm                                              */
  int32_t in_dtype;    /* q / k / v inputs: SNAP_F32 or SNAP_BF16                */
  int32_t kv_dtype;    /* cache storage: SNAP_F32, SNAP_BF16 (in_dtype == the
                          same) or SNAP_FP8_E4M3 (with SNAP_BF16 inputs)          */
  float sm_scale;      /* softmax scale; <= 0 means 1/sqrt(d_qk); a positive
                          value must be finite and at least 1e-30                */
  int32_t fp8_scales;  /* snap_fp8_scales (fp8 caches; ignored otherwise)        */
  int32_t fp8_qk;      /* decode attention over an fp8 cache: 0 = Q K^T in bf16
                          (the codes converted exactly); 1 = the query of each
                          head quantised to E4M3 with scale amax|q_h| / 448 (1
                          when q_h is zero; codes round to nearest even on the
                          fp32 quotient) and Q K^T on the fp8 MFMA.  Mode 1
                          changes the logits by the query's quantisation error
                          (about 2^-4 relative per element): it needs bf16
                          inputs, a GQA fp8 cache, d_qk = d_v = 128
                          (SNAP_ERR_UNSUPPORTED otherwise).  Values stay bf16
                          products.                                              */
  int32_t kv_reuse;    /* snap_kv_reuse: the decode kernels' load hint          */
} snap_params;

/* One layer's compressed cache (device memory, caller-owned, row-major):
 *   k       [n_slots][n_kv_heads][B][d_qk]  kv_dtype
 *   v       [n_slots][n_kv_heads][B][d_v]   kv_dtype; NULL when v_in_k
 *   k_scale [n_slots][n_kv_heads] fp32      FP8 only: stored code * scale is
 *   v_scale [n_slots][n_kv_heads] fp32      the value; set by the caller before
 *                                           compress/append, or by compress
 *                                           (fp8_scales); NULL otherwise. */
typedef struct {
  void* k;
  void* v;
  float* k_scale;
  float* v_scale;
  int32_t n_slots;
} snap_cache;

/* Slot metadata, shared by every layer (device int32[n_slots], caller-owned):
 *   pos[slot]    position of the token being decoded (L right after compress)
 *   n_topk[slot] real rows in the top-K region, min(max(L-sink-recent,0), K) */

/* Bytes of workspace snap_compress needs for n_seq sequences padded to
 * max_len.  0 on invalid parameters. */
size_t snap_compress_workspace(const snap_params* p, int32_t n_seq, int32_t max_len);

/* Bytes of workspace snap_decode_attn needs for n sequences.  0 on invalid
 * parameters. */
size_t snap_decode_workspace(const snap_params* p, int32_t n);

/* Compression at the end of prefill (Sec. III-B; Eq. 1-3).  For every
 * sequence b and KV head g:
 *   1. window scores: the G = n_q_heads/n_kv_heads query heads of group g at
 *      the last w_e = min(obs_window, L) positions score every key of the
 *      normaliser domain; softmax with sm_scale (Eq. 3);
 *   2. the softmax weights on the candidates C = [sink, L-recent) are summed
 *      over the window rows and the group's heads (Eq. 1);
 *   3. 1-D pooling (stride 1, pad pool_kernel/2) over C (Eq. 2);
 *   4. the min(K, |C|) candidates with the largest pooled score are kept (ties
 *      to the lower token index), in ascending token order;
 *   5. the cache of slot slot_ids[b] is rewritten: sinks, the last `recent`
 *      tokens at their ring rows (token t at row t < sink ? t :
 *      sink + (t - sink) mod recent), the kept tokens at rows sink+recent+m,
 *      zeros elsewhere (fp8: quantised with the slot/head scale), and
 *      pos[slot] = L, n_topk[slot] = min(K, |C|).
 * Arguments (device unless noted):
 *   slot_ids [n_seq] int32, lengths [n_seq] int32 (prompt lengths L),
 *   max_len (host) padded length of the inputs,
 *   q_obs [n_seq][n_q_heads][obs_window][d_qk] in_dtype; row obs_window-1 is
 *         position L-1 (rows before position 0 are ignored),
 *   k     [n_seq][n_kv_heads][max_len][d_qk] in_dtype (rows >= L never read),
 *   v     [n_seq][n_kv_heads][max_len][d_v]  in_dtype, NULL when v_in_k,
 *   sel_out    optional [n_seq][n_kv_heads][topk] int32: kept token indices,
 *              ascending, -1 padded (NULL to skip),
 *   pooled_out optional [n_seq][n_kv_heads][max_len] fp32: the pooled score of
 *              every candidate at its token index, NaN elsewhere (debug),
 *   workspace  >= snap_compress_workspace(p, n_seq, max_len) bytes, 256-byte
 *              aligned; its contents on entry do not matter.
 * n_seq == 0 is a no-op.  The sequences must target distinct slots. */
snap_status snap_compress(const snap_params* p, const snap_cache* cache, int32_t* pos,
                          int32_t* n_topk, int32_t n_seq, const int32_t* slot_ids,
                          const int32_t* lengths, int32_t max_len, const void* q_obs,
                          const void* k, const void* v, int32_t* sel_out, float* pooled_out,
                          void* workspace, size_t ws_bytes, void* stream);

/* Bytes of workspace snap_prefill needs for n_seq sequences padded to
 * max_len: the snap_compress workspace, the window queries and a transposed
 * copy of V.  0 on invalid parameters. */
size_t snap_prefill_workspace(const snap_params* p, int32_t n_seq, int32_t max_len);

/* Prefill attention and compression in one call (Sec. IV-A's attention step
 * followed by Sec. III-B, with the window scores' softmax statistics taken
 * from the attention pass instead of a separate recompute, Sec. III-B.2).
 *   1. out[b][h][i] = sum_{j <= i} softmax_j(sm_scale q[b][h][i].k[b][g][j])
 *      v[b][g][j] for every position i < L (g = h / G), in bf16;
 *   2. the compression of snap_compress with q_obs = the queries of the last
 *      obs_window positions of q (same cache, pos, n_topk, sel_out and
 *      pooled_out results).
 * Arguments as snap_compress, except (device):
 *   q   [n_seq][n_q_heads][max_len][d_qk] bf16 (rows >= L never read),
 *   k   [n_seq][n_kv_heads][max_len][d_qk] bf16,
 *   v   [n_seq][n_kv_heads][max_len][d_v]  bf16,
 *   out [n_seq][n_q_heads][max_len][d_v]   bf16; rows >= L are not written,
 *   workspace >= snap_prefill_workspace(p, n_seq, max_len) bytes, 256-byte
 *             aligned; its contents on entry do not matter.
 * Supported: in_dtype bf16, d_qk == d_v in {64, 128} (v_in_k = 0), and
 * G = n_q_heads / n_kv_heads in {1, 2, 4, 8, 16}; SNAP_ERR_UNSUPPORTED otherwise.
 * out must not alias q, k or v.  n_seq == 0 is a no-op. */
snap_status snap_prefill(const snap_params* p, const snap_cache* cache, int32_t* pos, int32_t* n_topk,
                         int32_t n_seq, const int32_t* slot_ids, const int32_t* lengths, int32_t max_len,
                         const void* q, const void* k, const void* v, void* out, int32_t* sel_out,
                         float* pooled_out, void* workspace, size_t ws_bytes, void* stream);

/* The attention step of snap_prefill alone (Sec. IV-A): out as in
 * snap_prefill, no cache or metadata written, no selection.  For layers that
 * are not compressed, and for timing the attention apart from the
 * compression.  Same supported shapes, workspace (snap_prefill_workspace) and
 * errors as snap_prefill. */
snap_status snap_prefill_attn(const snap_params* p, int32_t n_seq, const int32_t* lengths, int32_t max_len,
                              const void* q, const void* k, const void* v, void* out, void* workspace,
                              size_t ws_bytes, void* stream);

/* Decode KV update (Sec. III-C): for each of the n sequences, the new token's
 * keys/values k_new [n][n_kv_heads][d_qk] and v_new [n][n_kv_heads][d_v]
 * (in_dtype; v_new NULL when v_in_k) are written to row
 * slot_of(pos[slot]) = pos < sink ? pos : sink + (pos - sink) mod recent,
 * which for pos >= sink is the paper's (pos - sink + recent) mod recent + sink.
 * Sequences with pos[slot] < 0 are skipped. */
snap_status snap_cache_append(const snap_params* p, const snap_cache* cache, const int32_t* pos,
                              int32_t n, const int32_t* slot_ids, const void* k_new,
                              const void* v_new, void* stream);

/* Decode attention over the compressed cache (Sec. III-C; padding rows masked
 * per Sec. III-B.2).  For sequence b with p = pos[slot] (the token already
 * appended) the valid rows are [0, min(p+1, sink+recent)) and
 * [sink+recent, sink+recent+n_topk[slot]); each query head h attends its KV
 * head h / G: out[b][h] = sum_j softmax_j(sm_scale q.k_j) v_j.
 *   q   [n][n_q_heads][d_qk] in_dtype,
 *   out [n][n_q_heads][d_v]  out_dtype (SNAP_F32 or SNAP_BF16, rounded to
 *                            nearest even),
 *   workspace >= snap_decode_workspace(p, n) bytes, 256-byte aligned.
 * Rows outside the valid set are never read. */
snap_status snap_decode_attn(const snap_params* p, const snap_cache* cache, const int32_t* pos,
                             const int32_t* n_topk, int32_t n, const int32_t* slot_ids,
                             const void* q, void* out, int32_t out_dtype, void* workspace,
                             size_t ws_bytes, void* stream);

/* One layer's decode step (Sec. III-C): snap_cache_append(k_new, v_new)
 * followed by snap_decode_attn, with the same arguments, results and cache
 * contents as those two calls on the same stream.  For bf16 and fp8 caches of
 * the GQA shapes (d_qk = d_v = 128) and bf16 latent caches both happen in one
 * launch (the new token's row is read from k_new / v_new by the workgroup that
 * attends it, quantised there for an fp8 cache, and stored into the cache in
 * the same launch); other caches run the two launches.  The same workspace as
 * snap_decode_attn; k_new / v_new must not alias the cache. */
snap_status snap_decode_step(const snap_params* p, const snap_cache* cache, const int32_t* pos,
                             const int32_t* n_topk, int32_t n, const int32_t* slot_ids,
                             const void* q, const void* k_new, const void* v_new, void* out,
                             int32_t out_dtype, void* workspace, size_t ws_bytes, void* stream);

/* Device memory of snap_decode_step_noalloc: one array of this many bytes per
 * GPU, owned by the library. */
#define SNAP_NOALLOC_SCRATCH_BYTES (32u << 20)

/* snap_decode_step for callers that cannot allocate device memory (code under
 * HIP graph capture that must not allocate, tight serving loops, harnesses
 * that forbid allocation): the same arguments, results and cache contents,
 * without the workspace.  The split-K partials go to a library-owned device
 * array of SNAP_NOALLOC_SCRATCH_BYTES per GPU (reserved with the library's
 * device code on the first call on that GPU, held until the process ends;
 * the call itself allocates nothing).  A call that would need more than that
 * (snap_decode_workspace(p, n) > SNAP_NOALLOC_SCRATCH_BYTES) returns
 * SNAP_ERR_WORKSPACE and launches nothing.  Every call on one GPU shares that
 * GPU's array: calls that may overlap in time on one GPU (other streams, or
 * other threads without ordering between them) race and give wrong results,
 * so serialise them.  What one call leaves in the array does not affect the
 * next (a call writes every byte it reads first). */
snap_status snap_decode_step_noalloc(const snap_params* p, const snap_cache* cache, const int32_t* pos,
                                     const int32_t* n_topk, int32_t n, const int32_t* slot_ids, const void* q,
                                     const void* k_new, const void* v_new, void* out, int32_t out_dtype,
                                     void* stream);

/* The decode position moves on by one token (Sec. III-C: each generated token
 * takes the next position, and the ring row follows from it):
 * pos[slot_ids[b]] += 1 for b < n (once per decode step, after every layer).
 * pos is device int32[n_slots]; slot ids outside [0, n_slots) are skipped. */
snap_status snap_advance(int32_t* pos, int32_t n_slots, int32_t n, const int32_t* slot_ids,
                         void* stream);

/* Device-side checks of the debug build (libsnapstream_debug.so, built with
 * SNAP_DEBUG_CHECKS): its kernels test the invariants their indexing rests on
 * (keys inside the prompt, kept tokens inside the candidates, rows inside the
 * cache budget, chunk counts within the combine's capacity) and, where one
 * fails, skip the access and record it instead of faulting.  This call waits
 * for the device (hipDeviceSynchronize), stores the recorded bits in *flags (0
 * when none failed) and clears them when reset != 0.  A release build stores
 * 0 and returns SNAP_ERR_UNSUPPORTED.  Bits: 1 score chunk outside the keys,
 * 2 selection past K_eff, 4 kept token outside the candidates, 8 re-scored key
 * outside the candidates, 16 decode rows past the budget, 32 new token's row
 * outside the sink/ring rows, 64 too many split-K chunks, 128 appended row
 * outside the sink/ring rows, 256 prefill block outside the prompt. */
snap_status snap_debug_checks(uint32_t* flags, int32_t reset);

/* Static description of a status code. */
const char* snap_status_str(snap_status s);

/* Message describing the most recent failure on the calling thread ("" if
 * none).  The pointer stays valid until the thread's next library call. */
const char* snap_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* SNAPSTREAM_H */
