// snap_internal.h -- device helpers and the launcher interface shared by the
// HIP translation units of libsnapstream.  gfx950 (CDNA4) only: 64-lane
// wavefronts, bf16 MFMA 16x16x32, OCP fp8.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "snapstream.h"

namespace snap {

constexpr int kWave = 64;
constexpr uint32_t kQuietNaN = 0x7fc00000u;  // written as bits: kernels build without NaN semantics

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------- numerics
__device__ __forceinline__ float bf16_bits_to_f32(uint32_t h) { return __uint_as_float(h << 16); }

// fp32 -> bf16, round to nearest even (NaN stays NaN).
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

// Two fp32 -> packed bf16 pair (lo in the low half), round to nearest even:
// one v_cvt_pk_bf16_f32 on gfx950.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

// Work-item and workgroup indices straight from the hardware.  HIP's
// threadIdx / blockIdx / blockDim are device-library functions that cannot be
// inlined into kernels built without packed fp32 ops and IEEE mode (their
// target attributes differ), so they would become real calls whose results
// the compiler must treat as divergent.
__device__ __forceinline__ int tid() { return (int)__builtin_amdgcn_workitem_id_x(); }
__device__ __forceinline__ int bid_x() { return (int)__builtin_amdgcn_workgroup_id_x(); }
__device__ __forceinline__ int bid_y() { return (int)__builtin_amdgcn_workgroup_id_y(); }
__device__ __forceinline__ int nthreads() { return (int)__builtin_amdgcn_workgroup_size_x(); }

// A workgroup-uniform value read from global memory.  Kernels that also write
// global memory read their metadata with vector loads (the scalar cache is not
// coherent with those writes), which leaves the value in a vector register and
// makes the compiler treat control flow that depends on it as divergent;
// readfirstlane moves it back to a scalar register.
__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

// true when pred holds in any lane of the wave (wave-uniform)
__device__ __forceinline__ bool wave_any(bool pred) { return __builtin_amdgcn_ballot_w64(pred) != 0; }

// fp32 -> OCP E4M3 code: round to nearest even, saturate at +-448, NaN -> 0x7F.
__device__ __forceinline__ uint32_t f32_to_e4m3(float v) {
  uint32_t u = __float_as_uint(v);
  uint32_t sign = (u >> 24) & 0x80u;
  uint32_t a = u & 0x7fffffffu;
  if (a > 0x7f800000u) return 0x7fu;
  if (a >= 0x43e00000u) return sign | 0x7eu;  // |v| >= 448
  if (a >= 0x3c800000u) {                       // |v| >= 2^-6: normal code
    uint32_t r = a + 0x7ffffu + ((a >> 20) & 1u);
    uint32_t e = (r >> 23) - 120u;
    uint32_t m = (r >> 20) & 7u;
    return sign | (e << 3) | m;
  }
  // subnormal codes m * 2^-9 (m = 8 is the smallest normal, code 0x08)
  float q = __builtin_rintf(__uint_as_float(a) * 512.0f);
  return sign | (uint32_t)q;
}

// Four values -> four OCP E4M3 codes (low byte first) by the gfx950
// conversion instruction, two values per instruction (scale 1, round to
// nearest even).  The values are clamped to +-448 first and NaN is mapped to
// 0x7F afterwards, which makes every code equal to f32_to_e4m3's (checked
// over all 2^32 fp32 bit patterns by tests/native/fp8_cvt_check.hip).
typedef short e4m3_v2i16 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t e4m3x4_hw(float v0, float v1, float v2, float v3) {
  const float f[4] = {v0, v1, v2, v3};
  float c[4];
  uint32_t nan_mask = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    // NaN by its bits: the build lets float compares assume no NaN
    if ((__float_as_uint(f[i]) & 0x7fffffffu) > 0x7f800000u) nan_mask |= 0xffu << (8 * i);
    c[i] = __builtin_fminf(__builtin_fmaxf(f[i], -448.f), 448.f);
  }
  e4m3_v2i16 r = {0, 0};
  r = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(r, c[0], c[1], 1.0f, false);
  r = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(r, c[2], c[3], 1.0f, true);
  const uint32_t w = (uint32_t)(uint16_t)r[0] | ((uint32_t)(uint16_t)r[1] << 16);
  return (w & ~nan_mask) | (0x7f7f7f7fu & nan_mask);
}

// OCP E4M3 code -> fp32 (exact).
__device__ __forceinline__ float e4m3_to_f32(uint32_t c) {
  uint32_t cm = c & 0x7fu;
  float mag = (cm < 8u) ? (float)cm * (1.0f / 512.0f) : __uint_as_float((cm << 20) + (120u << 23));
  if (cm == 0x7fu) mag = __uint_as_float(0x7fc00000u);  // the E4M3 NaN code
  return (c & 0x80u) ? -mag : mag;
}

// 2^x by the hardware instruction (about 1 ulp).  Results below 2^-126 flush
// to zero; every caller exponentiates a value relative to a running maximum,
// where such terms are negligible.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ float warp_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// ---------------------------------------------------------------- debug checks
// Built with SNAP_DEBUG_CHECKS (libsnapstream_debug.so), kernels test the
// invariants their indexing rests on and record a violated one as a bit of a
// device word (one per source file), skipping the access the check guards,
// instead of faulting; snap_debug_checks() reads the words.  Release builds
// compile the checks away.
enum : uint32_t {
  kDbgScoreRange = 1u << 0,  // a score chunk's keys outside [0, max_len)
  kDbgSelWrite = 1u << 1,    // the ordered compaction would write past K_eff
  kDbgAsmSource = 1u << 2,   // a kept row's token outside the candidates
  kDbgBand = 1u << 3,        // a re-scored key outside the candidates
  kDbgDecodeSpan = 1u << 4,  // decode rows past sink + recent + topk
  kDbgDecodeNew = 1u << 5,   // the new token's row outside the sink / ring rows
  kDbgCombine = 1u << 6,     // more split-K chunks than the combine holds
  kDbgAppend = 1u << 7,      // an appended row outside the sink / ring rows
  kDbgPrefill = 1u << 8,     // a prefill block's positions outside the prompt
};
#ifdef SNAP_DEBUG_CHECKS
static __device__ uint32_t g_debug_flags;  // one per translation unit
__device__ __forceinline__ bool debug_check(bool ok, uint32_t bit) {
  if (!ok) atomicOr(&g_debug_flags, bit);
  return ok;
}
// host side: this file's word (and clear it)
#define SNAP_DEBUG_READER(name)                                                     \
  uint32_t name(bool reset) {                                                      \
    uint32_t v = 0;                                                                \
    if (hipMemcpyFromSymbol(&v, HIP_SYMBOL(g_debug_flags), sizeof(v)) != hipSuccess) \
      return 0xffffffffu;                                                          \
    if (reset) {                                                                   \
      const uint32_t z = 0;                                                        \
      if (hipMemcpyToSymbol(HIP_SYMBOL(g_debug_flags), &z, sizeof(z)) != hipSuccess) \
        return 0xffffffffu;                                                        \
    }                                                                              \
    return v;                                                                      \
  }
#else
__device__ __forceinline__ bool debug_check(bool, uint32_t) { return true; }
#define SNAP_DEBUG_READER(name) \
  uint32_t name(bool) { return 0; }
#endif
uint32_t debug_flags_compress(bool reset);
uint32_t debug_flags_decode(bool reset);
uint32_t debug_flags_prefill(bool reset);

// ---------------------------------------------------------------- launch context
struct Geometry {
  // compress
  int rows;         // G * obs_window
  int rows_pad;     // rows rounded up to 32 (one wave per 32 rows)
  int key_chunk;    // keys per workgroup in the score passes
  int n_kchunks;    // score-pass chunks per (sequence, KV head)
  int n_splits;     // candidate splits per group in pool/select
  int n_rowblocks;   // assemble row blocks per group
  size_t off_stats, off_rowref, off_A, off_P, off_hist, off_state, off_counts, off_sel, off_amax;
  // fp64 re-score of the candidates next to the selection threshold
  size_t off_rowz, off_band_n, off_band_idx, off_band_p, off_band_above, off_A64;
  size_t compress_bytes;
  // prefill (compress workspace followed by the window queries and V^T)
  int ld_vt;        // keys per V^T row (max_len rounded up to the key tile)
  size_t off_qobs, off_vt;
  size_t prefill_bytes;
  // decode
  int n_chunks;     // split-K chunks per (sequence, KV head)
  bool merge_many;  // the chunks are merged by merge_chunks (more than the combine keeps in registers)
  size_t off_part, off_ml;
  size_t decode_bytes;
};

constexpr int kKeyTile = 64;      // key chunks of the score passes are multiples of this
constexpr int kCandChunk = 2048;  // candidates per pool/select workgroup
constexpr int kSelThreads = 256;
constexpr int kRadixBins = 2048;
// Candidates whose pooled score lies within a factor 1 +- 2^-17 of the K-th
// largest are re-scored in fp64 before the final selection, up to this many
// per (sequence, KV head); a group with more keeps its fp32 selection.
constexpr int kBandCap = 512;

struct RadixState {
  uint32_t prefix;  // decided high bits of the threshold
  uint32_t mask;    // which bits are decided
  int32_t krem;     // how many elements equal to the threshold prefix still to take
  int32_t keff;     // how many candidates are kept in total
  int32_t mode;     // 0: nothing kept, 1: all candidates kept, 2: radix select
  int32_t pad[3];
};

// scale * log2(e) split as hi + lo (hi: fp32 rounded toward zero; lo > 0)
void split_scale2(float scale, float& hi, float& lo);

Geometry compress_geometry(const snap_params& p, int n_seq, int max_len);
Geometry decode_geometry(const snap_params& p, int n);
Geometry prefill_geometry(const snap_params& p, int n_seq, int max_len);

snap_status launch_compress(const snap_params& p, const snap_cache& c, int32_t* pos,
                            int32_t* n_topk, int n_seq, const int32_t* slot_ids,
                            const int32_t* lengths, int max_len, const void* q_obs, const void* k,
                            const void* v, int32_t* sel_out, float* pooled_out, void* ws,
                            hipStream_t stream, bool stats_given = false);
// causal attention of the whole prompt into out, then the compression with
// the window statistics taken from the attention pass
snap_status launch_prefill(const snap_params& p, const snap_cache& c, int32_t* pos, int32_t* n_topk, int n_seq,
                           const int32_t* slot_ids, const int32_t* lengths, int max_len, const void* q, const void* k,
                           const void* v, void* out, int32_t* sel_out, float* pooled_out, void* ws,
                           hipStream_t stream);
// the attention part of launch_prefill; want_stats: also the window rows'
// statistics and queries (into the compress part of the workspace)
snap_status launch_prefill_attn(const snap_params& p, int n_seq, const int32_t* lengths, int max_len, const void* q,
                                const void* k, const void* v, void* out, bool want_stats, void* ws,
                                hipStream_t stream);
snap_status launch_append(const snap_params& p, const snap_cache& c, const int32_t* pos, int n,
                          const int32_t* slot_ids, const void* k_new, const void* v_new,
                          hipStream_t stream);
// k_new / v_new non-NULL: append the token at pos first (fused into the
// attention launch for bf16 caches), as snap_cache_append would
snap_status launch_decode(const snap_params& p, const snap_cache& c, const int32_t* pos,
                          const int32_t* n_topk, int n, const int32_t* slot_ids, const void* q,
                          const void* k_new, const void* v_new, void* out, int out_dtype, void* ws,
                          hipStream_t stream);
snap_status launch_advance(int32_t* pos, int n_slots, int n, const int32_t* slot_ids, hipStream_t stream);

// device address of the current GPU's snap_decode_step_noalloc scratch array
snap_status noalloc_scratch(void** addr);

void set_error(const char* fmt, ...);

}  // namespace snap
