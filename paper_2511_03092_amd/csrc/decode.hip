// decode.hip -- decoding over the SnapStream cache (arXiv 2511.03092,
// Sec. III-C): the in-place ring update at row L_rb, and split-K attention
// over the valid rows (sinks + ring rows filled so far + the real top-K rows;
// padding rows are never read, Sec. III-B.2).
//
//   append         one workgroup per sequence writes k/v of token pos to its row
//   decode_mfma    per (chunk, sequence, KV head), one wave: bf16 MFMA
//                  K x q^T for the G heads of the group (padded to 16 columns),
//                  online softmax in the exp2 domain, MFMA V^T x P^T; bf16 or
//                  fp8 E4M3 rows (converted to bf16 in registers)
//   decode_mla_lds bf16 latent rows (576 wide, values = first 512 dims): four
//                  waves per (chunk, sequence) streaming 32-row blocks through
//                  a 4-stage LDS ring
//   decode_mla     fp8 latent rows, register-streamed
//   decode_generic one wave per (chunk, sequence, query head); any dtype
//   combine        log-sum-exp merge of the chunk partials -> out
// decode_mfma (bf16 and fp8 caches) and decode_mla_lds (bf16) also take the
// new token (snap_decode_step): the append happens in the same launch.
#include <math.h>

#include "snap_internal.h"

namespace snap {

constexpr float kLog2e = 1.4426950408889634f;
// Online softmax with a stale reference max: a head's reference moves only
// when a block's max exceeds it by more than this (log2 units), so the
// accumulators are rescaled on few blocks; probabilities stay <= 2^8.  Any
// reference gives the same softmax (the combine merges chunks by their own
// reference), only the rounding differs.
constexpr float kStaleMax = 8.f;

struct DecodeArgs {
  const void* q;         // [n][Hq][dk] (bf16 or fp32)
  const void* ck;        // [n_slots][Hkv][B][dk]
  const void* cv;        // [n_slots][Hkv][B][dv] or NULL (values = first dv dims of ck)
  const float* k_scale;  // fp8 only
  const float* v_scale;
  const int32_t* pos;
  const int32_t* n_topk;
  const int32_t* slot_ids;
  float* part;           // [n][Hq][n_chunks][dv]
  float2* ml;            // [n][Hq][n_chunks]  (max in log2 units, sum)
  // fused append (bf16 caches only): the token at pos, [n][Hkv][dk] / [n][Hkv][dv];
  // NULL when the launch only attends
  const void* k_new;
  const void* v_new;
  int Hq, Hkv, G, dk, dv, sink, recent, topk, n_slots, n_chunks, q_f32;
  float scale;
};

struct RowSpan {
  int n1, v0, v1, nv;  // first-run length, this chunk's [v0, v1), all valid rows
};

// Virtual row v in [0, n1 + n_topk) -> cache row: the first n1 are sinks and
// ring rows [0, n1), the rest the real top-K rows.
__device__ __forceinline__ int virt_row(int v, int n1, int sr) { return v < n1 ? v : sr + (v - n1); }

// Slot metadata is read with vector loads (the kernels also write global
// memory, so the compiler cannot use the scalar cache); readfirstlane puts the
// workgroup-uniform values back in scalar registers, which keeps the row loop
// and its waits scalar control flow.
__device__ __forceinline__ bool span_of(const DecodeArgs& a, int b, int chunk, int& slot, RowSpan& sp) {
  slot = __builtin_amdgcn_readfirstlane(a.slot_ids[b]);
  if (slot < 0 || slot >= a.n_slots) return false;
  const int sr = a.sink + a.recent;
  const int p = __builtin_amdgcn_readfirstlane(a.pos[slot]);
  int nt = __builtin_amdgcn_readfirstlane(a.n_topk[slot]);
  nt = nt < 0 ? 0 : (nt > a.topk ? a.topk : nt);
  const int n1 = p < 0 ? 0 : (p >= sr ? sr : p + 1);
  const int nv = n1 + nt;
  int cs = (nv + a.n_chunks - 1) / a.n_chunks;
  cs = (cs + 31) & ~31;
  sp.n1 = n1;
  sp.nv = nv;
  sp.v0 = chunk * cs;
  sp.v1 = min(sp.v0 + cs, nv);
  return debug_check(nv <= sr + a.topk, kDbgDecodeSpan);
}

// ---------------------------------------------------------------- fp8 -> bf16
// 8 E4M3 codes -> 8 bf16 (exact: every E4M3 value is a bf16 value), two codes
// per conversion instruction (scale 1; the cache scale is applied after the
// products).
__device__ __forceinline__ u32x4 e4m3x8_to_bf16x8(u32x2 c) {
  u32x4 o;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    o[2 * h] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(c[h], 1.0f, false));
    o[2 * h + 1] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(c[h], 1.0f, true));
  }
  return o;
}

// Raw 8-element loads: bf16 rows stay as 16 bytes, fp8 rows as 8 bytes of codes
// until they are used, so a prefetch does not wait on a conversion.  NT: the
// non-temporal (streaming) hint, for calls whose cache rows are too many to
// stay in the 256 MB last-level cache until the next call (launch_decode
// picks it): measured 13% faster for the fp8 GQA decode of 31 slots and,
// with the bf16 K chunk order of decode_mfma (kchunk), 7% for the bf16 one;
// on a one-layer 32k call (17 MB, re-read from that cache every step) it
// was slower, so small calls load without it.
template <bool FP8>
struct Raw8 {
  typedef u32x4 T;
};
template <>
struct Raw8<true> {
  typedef u32x2 T;
};

template <bool FP8, bool NT>
__device__ __forceinline__ typename Raw8<FP8>::T load_raw8(const void* base, size_t elem, bool ok) {
  typedef typename Raw8<FP8>::T T;
  T z = {};
  if (!ok) return z;
  const T* p = FP8 ? (const T*)((const uint8_t*)base + elem) : (const T*)((const uint16_t*)base + elem);
  if constexpr (NT)
    return __builtin_nontemporal_load(p);
  else
    return *p;
}

template <bool FP8>
__device__ __forceinline__ u32x4 bf16x8_of(typename Raw8<FP8>::T r) {
  if constexpr (FP8)
    return e4m3x8_to_bf16x8(r);
  else
    return r;
}

// 8 bf16 values (low half of each word first) -> the 8 E4M3 codes of
// value / scale: the quantisation snap_cache_append stores.
__device__ __forceinline__ u32x2 bf16x8_to_e4m3x8(u32x4 raw, float scale) {
  u32x2 o;
#pragma unroll
  for (int h2 = 0; h2 < 2; ++h2) {
    uint32_t w = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = h2 * 4 + i;
      const uint32_t bits = (j & 1) ? raw[j >> 1] >> 16 : raw[j >> 1] & 0xffffu;
      w |= f32_to_e4m3(bf16_bits_to_f32(bits) / scale) << (8 * i);
    }
    o[h2] = w;
  }
  return o;
}

// The new token's 8 elements at `elem` of its bf16 input row, in the cache's
// raw form: bf16 as is, fp8 quantised with the slot's scale (the bytes the
// append writes, so attending them equals attending the appended row).
template <bool FP8>
__device__ __forceinline__ typename Raw8<FP8>::T new_raw8(const void* src, size_t elem, float scale) {
  const u32x4 raw = *(const u32x4*)((const uint16_t*)src + elem);
  if constexpr (FP8)
    return bf16x8_to_e4m3x8(raw, scale);
  else
    return raw;
}

// Fused append: the cache row of the token at pos[slot] (the ring update of
// Sec. III-C; sinks are filled in place while pos < sink), or -1 when the
// launch carries no new token.  The row lies in the first run of valid rows,
// so its virtual index equals its cache row.  The workgroup that owns it reads
// it from k_new/v_new, chunk 0 stores it into the cache (fp8 caches: the
// owning workgroup quantises it and stores the codes), and nothing else in the
// launch touches that row: no ordering between workgroups is needed.
__device__ __forceinline__ int new_row(const DecodeArgs& a, int slot) {
  if (!a.k_new) return -1;
  const int p = __builtin_amdgcn_readfirstlane(a.pos[slot]);
  if (p < 0) return -1;
  const int row = p < a.sink ? p : a.sink + (p - a.sink) % a.recent;
  return debug_check(row < a.sink + a.recent, kDbgDecodeNew) ? row : -1;
}

// Chunk 0 of (slot, KV head g) stores the new k (and v) row, one 16-byte
// piece per thread (dk/8 + dv/8 pieces, at most the workgroup size).  The
// piece is fetched with the query and stored once that load has landed, so
// the store adds no memory round trip of its own.
__device__ __forceinline__ bool new_piece_load(const DecodeArgs& a, int b, int g, int i, u32x4& x) {
  const int kc = a.dk / 8, vc = a.cv ? a.dv / 8 : 0;
  if (i >= kc + vc) return false;
  if (i < kc)
    x = *((const u32x4*)a.k_new + ((size_t)b * a.Hkv + g) * kc + i);
  else
    x = *((const u32x4*)a.v_new + ((size_t)b * a.Hkv + g) * vc + (i - kc));
  return true;
}
__device__ __forceinline__ void new_piece_store(const DecodeArgs& a, int g, int slot, int row, int i, u32x4 x) {
  const int B = a.sink + a.recent + a.topk;
  const size_t crow = ((size_t)slot * a.Hkv + g) * (size_t)B + row;
  const int kc = a.dk / 8, vc = a.cv ? a.dv / 8 : 0;
  if (i < kc)
    *((u32x4*)const_cast<void*>(a.ck) + crow * kc + i) = x;
  else
    *((u32x4*)const_cast<void*>(a.cv) + crow * vc + (i - kc)) = x;
}

// ---------------------------------------------------------------- MFMA decode
// KSTEPS = dk / 32, VPASS = dv / 128.  Lane l owns head l%16 of the group and,
// per 16-row set, the output rows 4*(l/16)+e; P never leaves the lane between
// the two products because the V operand is loaded in the matching row order.
typedef int i32x8 __attribute__((ext_vector_type(8)));

// The 8-element chunk of a 32 * KSTEPS-wide row that lane group lg feeds to
// k-step t (q and K use the same map, so the dot products are unchanged).
// bf16 with streaming loads: chunk 4t + lg, so one load instruction reads 64
// contiguous bytes of each of its 16 rows (chunk KSTEPS*lg + t, where the four
// instructions each read 16 bytes of every 64, re-fetched lines under the
// streaming hint and was 15% slower).  Otherwise chunk KSTEPS*lg + t: with
// ordinary loads it measured 1.5% faster on the one-layer 32k call, and fp8
// keeps lane group lg on the 32 contiguous codes 32lg..32lg+31 that the fp8
// MFMA of the fp8_qk path takes per lane.
template <int KSTEPS, bool FP8, bool NT>
__device__ __forceinline__ int kchunk(int t, int lg) { return (FP8 || !NT) ? KSTEPS * lg + t : 4 * t + lg; }

template <int KSTEPS, int VPASS, bool FP8, bool QK8, bool NT>
__global__ __launch_bounds__(64) void decode_mfma(DecodeArgs a) {
  static_assert(!QK8 || (FP8 && KSTEPS == 4), "fp8 products need an fp8 cache of 128-wide rows");
  constexpr int D = KSTEPS * 32;
  typedef typename Raw8<FP8>::T RawT;
  const int lane = tid(), l16 = lane & 15, lg = lane >> 4;
  const int chunk = bid_x(), bg = bid_y(), b = bg / a.Hkv, g = bg % a.Hkv;
  int slot;
  RowSpan sp;
  if (!span_of(a, b, chunk, slot, sp)) return;
  const int sr = a.sink + a.recent;
  const int B = sr + a.topk;
  const int h = l16;
  const bool hval = h < a.G;
  const int qh = g * a.G + (hval ? h : 0);

  bf16x8 qf[KSTEPS];
  {
    const uint16_t* qp = (const uint16_t*)a.q + ((size_t)b * a.Hq + qh) * D;
#pragma unroll
    for (int t = 0; t < KSTEPS; ++t) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (hval) v = *(const u32x4*)(qp + 8 * kchunk<KSTEPS, FP8, NT>(t, lg));
      qf[t] = __builtin_bit_cast(bf16x8, v);
    }
  }
  const size_t row0 = ((size_t)slot * a.Hkv + g) * (size_t)B;
  const float ksc = FP8 ? a.k_scale[(size_t)slot * a.Hkv + g] : 1.f;
  const float vsc = FP8 ? (a.cv ? a.v_scale : a.k_scale)[(size_t)slot * a.Hkv + g] : 1.f;
  // QK8: this lane's head (l16) quantised to E4M3 with scale amax|q| / 448
  // (the lane holds dims 32*lg .. 32*lg+31, the fp8 MFMA's k-slots for them)
  i32x8 q8 = {0, 0, 0, 0, 0, 0, 0, 0};
  float qsc = 1.f;
  if constexpr (QK8) {
    float amax = 0.f;
#pragma unroll
    for (int t = 0; t < KSTEPS; ++t) {
      const u32x4 w = __builtin_bit_cast(u32x4, qf[t]);
#pragma unroll
      for (int i = 0; i < 4; ++i)
        amax = fmaxf(amax, fmaxf(fabsf(bf16_bits_to_f32(w[i] & 0xffffu)), fabsf(bf16_bits_to_f32(w[i] >> 16))));
    }
    amax = fmaxf(amax, __shfl_xor(amax, 16));
    amax = fmaxf(amax, __shfl_xor(amax, 32));
    qsc = amax > 0.f ? amax / 448.f : 1.f;
#pragma unroll
    for (int t = 0; t < KSTEPS; ++t) {
      const u32x2 c = bf16x8_to_e4m3x8(__builtin_bit_cast(u32x4, qf[t]), qsc);
      q8[2 * t] = (int)c[0];
      q8[2 * t + 1] = (int)c[1];
    }
  }
  const float xs = a.scale * kLog2e * ksc * qsc;
  const void* vbase = a.cv ? a.cv : a.ck;
  const int vstride = a.cv ? a.dv : a.dk;
  // fused append: row vnew comes from k_new / v_new (quantised for fp8 caches)
  const int vnew = new_row(a, slot);
  const size_t knew_off = ((size_t)b * a.Hkv + g) * D, vnew_off = ((size_t)b * a.Hkv + g) * a.dv;
  u32x4 newp = {0u, 0u, 0u, 0u};
  const bool has_newp = !FP8 && vnew >= 0 && chunk == 0 && new_piece_load(a, b, g, lane, newp);
  // fp8: the chunk that attends the new row quantises it once into LDS (K
  // codes in pieces [0, D/8), V codes after them, 8 codes per piece) and
  // stores those codes into the cache at its end
  __shared__ u32x2 newq[FP8 ? (D + 128 * VPASS) / 8 : 1];
  const bool owns_new = FP8 && vnew >= sp.v0 && vnew < sp.v1;
  if constexpr (FP8) {
    if (owns_new) {
      constexpr int kc = D / 8;
      if (lane < kc)
        newq[lane] = new_raw8<true>(a.k_new, knew_off + 8 * lane, ksc);
      else if (lane < kc + 16 * VPASS)
        newq[lane] = new_raw8<true>(a.v_new, vnew_off + 8 * (lane - kc), vsc);
      __syncthreads();
    }
  }

  float m = -INFINITY, mref = 0.f, lsum = 0.f;  // reference max (log2 units), its finite stand-in, sum
  f32x4 acc[VPASS][8];
#pragma unroll
  for (int pp = 0; pp < VPASS; ++pp)
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[pp][c] = f32x4{0.f, 0.f, 0.f, 0.f};

  // a whole block inside one run of the row map, without the new token: 32
  // consecutive cache rows from a uniform base (wave-uniform test)
  auto plain = [&](int vb) {
    return vb + 32 <= sp.v1 && (vb + 32 <= sp.n1 || vb >= sp.n1) && !(vnew >= vb && vnew < vb + 32);
  };
  // K of block vb: lane's rows vb+l16 and vb+16+l16, k-slot group lg
  auto load_k = [&](int vb, RawT* ka, RawT* kb) {
    if (plain(vb)) {
      const size_t e0 = (row0 + virt_row(vb, sp.n1, sr)) * D + (size_t)l16 * D;
#pragma unroll
      for (int t = 0; t < KSTEPS; ++t) {
        const int col = 8 * kchunk<KSTEPS, FP8, NT>(t, lg);
        ka[t] = load_raw8<FP8, NT>(a.ck, e0 + col, true);
        kb[t] = load_raw8<FP8, NT>(a.ck, e0 + 16 * D + col, true);
      }
      return;
    }
    const int va = vb + l16, vb2 = vb + 16 + l16;
    const size_t ea = (row0 + virt_row(va, sp.n1, sr)) * D;
    const size_t eb = (row0 + virt_row(vb2, sp.n1, sr)) * D;
#pragma unroll
    for (int t = 0; t < KSTEPS; ++t) {
      const int col = 8 * kchunk<KSTEPS, FP8, NT>(t, lg);
      if constexpr (FP8) {
        ka[t] = va == vnew ? newq[col / 8] : load_raw8<FP8, NT>(a.ck, ea + col, va < sp.v1);
        kb[t] = vb2 == vnew ? newq[col / 8] : load_raw8<FP8, NT>(a.ck, eb + col, vb2 < sp.v1);
      } else {
        ka[t] = load_raw8<FP8, NT>(va == vnew ? a.k_new : a.ck, va == vnew ? knew_off + col : ea + col, va < sp.v1);
        kb[t] = load_raw8<FP8, NT>(vb2 == vnew ? a.k_new : a.ck, vb2 == vnew ? knew_off + col : eb + col, vb2 < sp.v1);
      }
    }
  };
  RawT ka[KSTEPS], kb[KSTEPS];
  if (sp.v0 < sp.v1) load_k(sp.v0, ka, kb);

  for (int vb = sp.v0; vb < sp.v1; vb += 32) {
    // V of this block (eight rows per lane, in the order of the score layout),
    // then K of the next block: the value product waits only for V.
    RawT vv[VPASS][8];
    if (plain(vb)) {
      const size_t e0 = (row0 + virt_row(vb, sp.n1, sr)) * vstride + 8 * l16;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int r = i < 4 ? 4 * lg + i : 16 + 4 * lg + (i - 4);
#pragma unroll
        for (int pp = 0; pp < VPASS; ++pp) vv[pp][i] = load_raw8<FP8, NT>(vbase, e0 + (size_t)r * vstride + 128 * pp, true);
      }
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int vi = vb + (i < 4 ? 4 * lg + i : 16 + 4 * lg + (i - 4));
        const size_t ev = (row0 + virt_row(vi, sp.n1, sr)) * vstride;
#pragma unroll
        for (int pp = 0; pp < VPASS; ++pp)
          if constexpr (FP8)
            vv[pp][i] = vi == vnew ? newq[D / 8 + 16 * pp + l16]
                                   : load_raw8<FP8, NT>(vbase, ev + 128 * pp + 8 * l16, vi < sp.v1);
          else
            vv[pp][i] = load_raw8<FP8, NT>(vi == vnew ? a.v_new : vbase,
                                       (vi == vnew ? vnew_off : ev) + 128 * pp + 8 * l16, vi < sp.v1);
      }
    }
    RawT kn[KSTEPS], kn2[KSTEPS];
    if (vb + 32 < sp.v1) load_k(vb + 32, kn, kn2);

    f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
    if constexpr (QK8) {
      // one fp8 MFMA per 16 rows: the lane's 32 codes of each row against the
      // head's 32 query codes (E4M3 both, unit block scales)
      i32x8 k8a, k8b;
#pragma unroll
      for (int t = 0; t < KSTEPS; ++t) {
        k8a[2 * t] = (int)ka[t][0];
        k8a[2 * t + 1] = (int)ka[t][1];
        k8b[2 * t] = (int)kb[t][0];
        k8b[2 * t + 1] = (int)kb[t][1];
      }
      s0 = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(k8a, q8, s0, 0, 0, 0, 127, 0, 127);
      s1 = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(k8b, q8, s1, 0, 0, 0, 127, 0, 127);
    } else {
#pragma unroll
      for (int t = 0; t < KSTEPS; ++t) {
        s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, bf16x8_of<FP8>(ka[t])), qf[t], s0, 0, 0, 0);
        s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, bf16x8_of<FP8>(kb[t])), qf[t], s1, 0, 0, 0);
      }
    }
    // raw dot products; the scale (> 0, fp8 key scale included) is applied to
    // the block max and folded into the exponent
    float x[8];
    if (vb + 32 <= sp.v1) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x[e] = s0[e];
        x[4 + e] = s1[e];
      }
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x[e] = (vb + 4 * lg + e < sp.v1) ? s0[e] : -INFINITY;
        x[4 + e] = (vb + 16 + 4 * lg + e < sp.v1) ? s1[e] : -INFINITY;
      }
    }
    float bm = fmaxf(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])), fmaxf(fmaxf(x[4], x[5]), fmaxf(x[6], x[7])));
    bm = fmaxf(bm, __shfl_xor(bm, 16));
    bm = fmaxf(bm, __shfl_xor(bm, 32));
    bm *= xs;
    const bool up = bm > m + kStaleMax;  // always true for the first valid block (m = -inf)
    if (wave_any(up)) {
      const float mnew = up ? bm : m;
      const float alpha = up ? fast_exp2(m - mnew) : 1.f;
#pragma unroll
      for (int pp = 0; pp < VPASS; ++pp)
#pragma unroll
        for (int c = 0; c < 8; ++c) acc[pp][c] *= alpha;
      lsum *= alpha;
      m = mnew;
      mref = m == -INFINITY ? 0.f : m;  // no valid row yet: every x is -inf, exp2 gives 0
    }
    float pe[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) pe[i] = fast_exp2(fmaf(x[i], xs, -mref));
    lsum += ((pe[0] + pe[1]) + (pe[2] + pe[3])) + ((pe[4] + pe[5]) + (pe[6] + pe[7]));
    u32x4 pw;
#pragma unroll
    for (int i = 0; i < 4; ++i) pw[i] = pack_bf16x2(pe[2 * i], pe[2 * i + 1]);
    const bf16x8 pb = __builtin_bit_cast(bf16x8, pw);
#pragma unroll
    for (int pp = 0; pp < VPASS; ++pp) {
      u32x4 vbf[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) vbf[i] = bf16x8_of<FP8>(vv[pp][i]);
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const int u = c >> 1;
        const uint32_t selb = (c & 1) ? 0x07060302u : 0x05040100u;
        u32x4 av;
#pragma unroll
        for (int i = 0; i < 4; ++i) av[i] = __builtin_amdgcn_perm(vbf[2 * i + 1][u], vbf[2 * i][u], selb);
        acc[pp][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, av), pb, acc[pp][c], 0, 0, 0);
      }
    }
#pragma unroll
    for (int t = 0; t < KSTEPS; ++t) {
      ka[t] = kn[t];
      kb[t] = kn2[t];
    }
  }
  lsum += __shfl_xor(lsum, 16);
  lsum += __shfl_xor(lsum, 32);
  if (has_newp) new_piece_store(a, g, slot, vnew, lane, newp);
  if constexpr (FP8) {
    if (owns_new && lane < D / 8 + 16 * VPASS) {
      const size_t crow = ((size_t)slot * a.Hkv + g) * (size_t)B + vnew;
      if (lane < D / 8)
        *((u32x2*)const_cast<void*>(a.ck) + crow * (D / 8) + lane) = newq[lane];
      else
        *((u32x2*)const_cast<void*>(a.cv) + crow * (a.dv / 8) + (lane - D / 8)) = newq[lane];
    }
  }
  if (!hval) return;
  const size_t pi = ((size_t)b * a.Hq + qh) * a.n_chunks + chunk;
  if (lg == 0) a.ml[pi] = make_float2(m, lsum);
  float* dst = a.part + pi * a.dv;
#pragma unroll
  for (int pp = 0; pp < VPASS; ++pp)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float4 lo = make_float4(acc[pp][0][e], acc[pp][1][e], acc[pp][2][e], acc[pp][3][e]);
      float4 hi = make_float4(acc[pp][4][e], acc[pp][5][e], acc[pp][6][e], acc[pp][7][e]);
      lo.x *= vsc; lo.y *= vsc; lo.z *= vsc; lo.w *= vsc;
      hi.x *= vsc; hi.y *= vsc; hi.z *= vsc; hi.w *= vsc;
      float* d = dst + 128 * pp + 8 * (4 * lg + e);
      *(float4*)d = lo;
      *(float4*)(d + 4) = hi;
    }
}

// ---------------------------------------------------------------- latent (MLA) decode
// One workgroup of 4 waves per (chunk, sequence) of a shared 576-wide latent
// cache (values = first 512 dims).  Per block of 32 rows, wave w computes the
// partial logits over its share of the 18 k-steps of 32 dims (5,5,4,4), the
// four partials are summed through LDS in a fixed order (so every wave holds
// identical logits), and wave w then runs the value product for dims
// [128w, 128w+128).  Heads beyond G (<= 16) are zero columns.
constexpr int kMlaKSteps = 18;
__device__ __forceinline__ int mla_kbeg(int w) { return w < 2 ? 5 * w : 10 + 4 * (w - 2); }
__device__ __forceinline__ int mla_kcnt(int w) { return w < 2 ? 5 : 4; }

template <bool FP8, bool NT>
__global__ __launch_bounds__(256) void decode_mla(DecodeArgs a) {
  constexpr int D = kMlaKSteps * 32;  // 576
  typedef typename Raw8<FP8>::T RawT;
  __shared__ f32x4 sbuf[2][4][2][64];  // [parity][wave][row set][lane]
  const int lane = tid() & 63, w = tid() >> 6;
  const int l16 = lane & 15, lg = lane >> 4;
  const int chunk = bid_x(), b = bid_y();  // one KV head
  int slot;
  RowSpan sp;
  if (!span_of(a, b, chunk, slot, sp)) return;
  const int sr = a.sink + a.recent;
  const int B = sr + a.topk;
  const int h = l16;
  const bool hval = h < a.G;
  const int kb = mla_kbeg(w), kc = mla_kcnt(w);

  bf16x8 qf[5];
  {
    const uint16_t* qp = (const uint16_t*)a.q + ((size_t)b * a.Hq + (hval ? h : 0)) * D;
#pragma unroll
    for (int t = 0; t < 5; ++t) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (hval && t < kc) v = *(const u32x4*)(qp + 32 * kb + 8 * (kc * lg + t));
      qf[t] = __builtin_bit_cast(bf16x8, v);
    }
  }
  const size_t row0 = (size_t)slot * B;
  const float ksc = FP8 ? a.k_scale[slot] : 1.f;
  const float xs = a.scale * kLog2e * ksc;

  float m = -INFINITY, mref = 0.f, lsum = 0.f;  // reference max (log2 units), its finite stand-in, sum
  f32x4 acc[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) acc[c] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto load_k = [&](int vb, RawT* ka, RawT* kbv) {
    const int va = vb + l16, vb2 = vb + 16 + l16;
    const size_t ra = row0 + virt_row(va, sp.n1, sr), rb = row0 + virt_row(vb2, sp.n1, sr);
#pragma unroll
    for (int t = 0; t < 5; ++t) {
      const int col = 32 * kb + 8 * (kc * lg + t);
      const bool tin = t < kc;
      ka[t] = load_raw8<FP8, NT>(a.ck, ra * D + col, va < sp.v1 && tin);
      kbv[t] = load_raw8<FP8, NT>(a.ck, rb * D + col, vb2 < sp.v1 && tin);
    }
  };
  RawT ka[5], kbv[5];
  if (sp.v0 < sp.v1) load_k(sp.v0, ka, kbv);

  int parity = 0;
  for (int vb = sp.v0; vb < sp.v1; vb += 32, parity ^= 1) {
    RawT vv[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int vi = vb + (i < 4 ? 4 * lg + i : 16 + 4 * lg + (i - 4));
      const size_t rr = row0 + virt_row(vi, sp.n1, sr);
      vv[i] = load_raw8<FP8, NT>(a.ck, rr * D + 128 * w + 8 * l16, vi < sp.v1);
    }
    RawT kn[5], kn2[5];
    if (vb + 32 < sp.v1) load_k(vb + 32, kn, kn2);

    f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int t = 0; t < 5; ++t) {
      if (t < kc) {
        s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, bf16x8_of<FP8>(ka[t])), qf[t], s0, 0, 0, 0);
        s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, bf16x8_of<FP8>(kbv[t])), qf[t], s1, 0, 0, 0);
      }
    }
    sbuf[parity][w][0][lane] = s0;
    sbuf[parity][w][1][lane] = s1;
    __syncthreads();
    s0 = ((sbuf[parity][0][0][lane] + sbuf[parity][1][0][lane]) + sbuf[parity][2][0][lane]) + sbuf[parity][3][0][lane];
    s1 = ((sbuf[parity][0][1][lane] + sbuf[parity][1][1][lane]) + sbuf[parity][2][1][lane]) + sbuf[parity][3][1][lane];
    // raw dot products; the scale (> 0, fp8 key scale included) is applied to
    // the block max and folded into the exponent
    float x[8];
    if (vb + 32 <= sp.v1) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x[e] = s0[e];
        x[4 + e] = s1[e];
      }
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x[e] = (vb + 4 * lg + e < sp.v1) ? s0[e] : -INFINITY;
        x[4 + e] = (vb + 16 + 4 * lg + e < sp.v1) ? s1[e] : -INFINITY;
      }
    }
    float bm = fmaxf(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])), fmaxf(fmaxf(x[4], x[5]), fmaxf(x[6], x[7])));
    bm = fmaxf(bm, __shfl_xor(bm, 16));
    bm = fmaxf(bm, __shfl_xor(bm, 32));
    bm *= xs;
    const bool up = bm > m + kStaleMax;  // always true for the first valid block (m = -inf)
    if (wave_any(up)) {
      const float mnew = up ? bm : m;
      const float alpha = up ? fast_exp2(m - mnew) : 1.f;
#pragma unroll
      for (int c = 0; c < 8; ++c) acc[c] *= alpha;
      lsum *= alpha;
      m = mnew;
      mref = m == -INFINITY ? 0.f : m;  // no valid row yet: every x is -inf, exp2 gives 0
    }
    float pe[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) pe[i] = fast_exp2(fmaf(x[i], xs, -mref));
    lsum += ((pe[0] + pe[1]) + (pe[2] + pe[3])) + ((pe[4] + pe[5]) + (pe[6] + pe[7]));
    u32x4 pw;
#pragma unroll
    for (int i = 0; i < 4; ++i) pw[i] = pack_bf16x2(pe[2 * i], pe[2 * i + 1]);
    const bf16x8 pb = __builtin_bit_cast(bf16x8, pw);
    u32x4 vbf[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) vbf[i] = bf16x8_of<FP8>(vv[i]);
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      const int u = c >> 1;
      const uint32_t selb = (c & 1) ? 0x07060302u : 0x05040100u;
      u32x4 av;
#pragma unroll
      for (int i = 0; i < 4; ++i) av[i] = __builtin_amdgcn_perm(vbf[2 * i + 1][u], vbf[2 * i][u], selb);
      acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, av), pb, acc[c], 0, 0, 0);
    }
#pragma unroll
    for (int t = 0; t < 5; ++t) {
      ka[t] = kn[t];
      kbv[t] = kn2[t];
    }
  }
  lsum += __shfl_xor(lsum, 16);
  lsum += __shfl_xor(lsum, 32);
  if (!hval) return;
  const size_t pi = ((size_t)b * a.Hq + h) * a.n_chunks + chunk;
  if (w == 0 && lg == 0) a.ml[pi] = make_float2(m, lsum);
  const float vsc = FP8 ? a.k_scale[slot] : 1.f;
  float* dst = a.part + pi * a.dv + 128 * w;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    float4 lo = make_float4(acc[0][e], acc[1][e], acc[2][e], acc[3][e]);
    float4 hi = make_float4(acc[4][e], acc[5][e], acc[6][e], acc[7][e]);
    lo.x *= vsc; lo.y *= vsc; lo.z *= vsc; lo.w *= vsc;
    hi.x *= vsc; hi.y *= vsc; hi.z *= vsc; hi.w *= vsc;
    float* d = dst + 8 * (4 * lg + e);
    *(float4*)d = lo;
    *(float4*)(d + 4) = hi;
  }
}

// ---------------------------------------------------------------- latent decode, LDS-staged
// bf16 latent caches (576-wide rows, values = first 512 dims).  One workgroup
// of 4 waves per (chunk, sequence) streams blocks of 32 rows through a ring
// of LDS stages with direct global->LDS loads, so three blocks (110 KB) are in
// flight per CU while one is consumed.  Every wave forms the block's logits
// over all 18 k-steps (the same sums in the same order in each wave: no
// exchange or barrier between the two products; measured 2% faster than
// splitting the k-steps over the waves and summing through LDS), and wave w
// computes the value product for dims [128w, 128w+128).
// LDS rows are 72 chunks of 16 bytes; chunk c of row r sits at slot
// r*72 + (c ^ lat_swz(r)).  The row swizzle spreads the key-fragment reads
// (one chunk of 16 consecutive rows) over the banks; the value reads
// (consecutive chunks of one row) stay within aligned groups of 8 chunks.  Of
// the swizzles measured with the LDS bank-conflict counter this one has the
// fewest conflicts.
// Four 36 KB stages (147 KB of the 160 KB LDS: one workgroup per CU); a
// stage is refilled once every wave has consumed it, so four blocks are in
// flight when block i is waited for.
constexpr int kLatStages = 4;
constexpr int kLatRowBytes = 576 * 2;
constexpr int kLatChunks = kLatRowBytes / 16;        // 72
constexpr int kLatBlockBytes = 32 * kLatRowBytes;    // 36864
constexpr int kLatLoadsPerWave = 32 * kLatChunks / 64 / 4;  // 9 wave-instructions per block per wave

__device__ __forceinline__ int lat_swz(int r) { return (r >> 1) & 7; }
__device__ __forceinline__ int lat_slot(int r, int c) { return r * kLatChunks + (c ^ lat_swz(r)); }

typedef __attribute__((address_space(3))) void* lds_void_ptr_t;
// One wave-instruction of global -> LDS copy (lane i's 16 bytes land at
// lds_wave_base + 16*i), issued through inline asm so that the only ordering
// with later LDS reads is the caller's explicit vmcnt wait and barrier.  M0
// (the DMA's LDS base) is saved and restored around it.  NT as for load_raw8
// (measured 3-7% faster on the 16 x 128k latent call).
template <bool NT>
__device__ __forceinline__ void dma16_lat(const void* g, const void* lds_wave_base) {
  // wave-uniform by construction; readfirstlane keeps it in a scalar register
  // whatever the compiler's uniformity analysis concludes
  const uint32_t la = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_void_ptr_t)lds_wave_base);
  uint32_t saved;
  if constexpr (NT)
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %1\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %2, off nt\n\t"
        "s_nop 0\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "s"(la), "v"(g)
        : "memory");
  else
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %1\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %2, off\n\t"
        "s_nop 0\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "s"(la), "v"(g)
        : "memory");
}

template <int N>
__device__ __forceinline__ void lat_wait_vm() {
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}
__device__ __forceinline__ void lat_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0) only
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

template <bool NT>
__global__ __launch_bounds__(256) void decode_mla_lds(DecodeArgs a) {
  constexpr int D = 576;
  __shared__ __align__(16) unsigned char stage[kLatStages][kLatBlockBytes];
  const int lane = tid() & 63, w = tid() >> 6;
  const int l16 = lane & 15, lg = lane >> 4;
  const int chunk = bid_x(), b = bid_y();
  int slot;
  RowSpan sp;
  if (!span_of(a, b, chunk, slot, sp)) return;
  const int sr = a.sink + a.recent;
  const int B = sr + a.topk;
  const int h = l16;
  const bool hval = h < a.G;
  const int wu = __builtin_amdgcn_readfirstlane(w);

  // every wave forms the block's logits over all 18 k-steps itself (the same
  // sums in the same order in each wave, so no exchange between waves);
  // lane group lg holds dims 8*(18*lg + t) of k-step t
  bf16x8 qf[kMlaKSteps];
  // this lane's share of every block load: (row, chunk) of its 9 slots
  int ld_r[kLatLoadsPerWave], ld_c[kLatLoadsPerWave], ld_off[kLatLoadsPerWave];
#pragma unroll
  for (int ii = 0; ii < kLatLoadsPerWave; ++ii) {
    const int q = (wu + 4 * ii) * 64 + lane;
    const int r = q / kLatChunks, cs = q % kLatChunks;
    ld_r[ii] = r;
    ld_c[ii] = cs ^ lat_swz(r);
    ld_off[ii] = r * kLatRowBytes + ld_c[ii] * 16;
  }
  const unsigned char* cache = (const unsigned char*)a.ck + (size_t)slot * B * kLatRowBytes;
  // fused append: row vnew comes from k_new
  const int vnew = new_row(a, slot);
  const unsigned char* knew = vnew >= 0 ? (const unsigned char*)a.k_new + (size_t)b * kLatRowBytes : nullptr;
  u32x4 newp = {0u, 0u, 0u, 0u};
  const bool has_newp = vnew >= 0 && chunk == 0 && new_piece_load(a, b, 0, tid(), newp);
  // The slot's 32-row blocks are interleaved over its chunks: block i of
  // this chunk is the slot's block chunk + i * n_chunks.  At any moment the
  // chunks of a slot read one window of neighbouring blocks, which spreads
  // the requests over the memory channels (measured 1% faster than
  // contiguous chunk ranges).
  const int nb_slot = (sp.nv + 31) / 32;
  const int nblk =
      __builtin_amdgcn_readfirstlane(chunk < nb_slot ? (nb_slot - chunk + a.n_chunks - 1) / a.n_chunks : 0);
  auto issue = [&](int blk) {
    const int vb = 32 * (chunk + blk * a.n_chunks);
    unsigned char* dst = &stage[blk % kLatStages][0];
    // a whole block inside one run of the row map, without the new token:
    // 32 consecutive cache rows from a uniform base
    const bool plain = vb + 32 <= sp.nv && (vb + 32 <= sp.n1 || vb >= sp.n1) && !(vnew >= vb && vnew < vb + 32);
    if (plain) {
      const unsigned char* base = cache + (size_t)virt_row(vb, sp.n1, sr) * kLatRowBytes;
#pragma unroll
      for (int ii = 0; ii < kLatLoadsPerWave; ++ii) dma16_lat<NT>(base + ld_off[ii], dst + (size_t)(wu + 4 * ii) * 1024);
    } else {
#pragma unroll
      for (int ii = 0; ii < kLatLoadsPerWave; ++ii) {
        int v = vb + ld_r[ii];
        v = v < sp.nv ? v : sp.nv - 1;
        const unsigned char* src =
            (v == vnew ? knew : cache + (size_t)virt_row(v, sp.n1, sr) * kLatRowBytes) + ld_c[ii] * 16;
        dma16_lat<NT>(src, dst + (size_t)(wu + 4 * ii) * 1024);
      }
    }
  };

  const float xs = a.scale * kLog2e;
  float m = -INFINITY, mref = 0.f, lsum = 0.f;  // reference max (log2 units), its finite stand-in, sum
  f32x4 acc[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) acc[c] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Prologue: the query rows (G x 1152 bytes) go straight to LDS in the last
  // stage, ahead of blocks 0..2, so one wait covers both and the first block
  // lands after a single memory latency.  Once every wave has copied its
  // query fragments out, the last stage takes block 3.
  if (nblk > 0) {
    const int qchunks = a.G * kLatChunks;
    const int nq = (qchunks + 63) / 64;  // wave-instructions (G <= 16: at most 18)
    const unsigned char* qsrc = (const unsigned char*)a.q + (size_t)b * a.Hq * kLatRowBytes;
    unsigned char* qdst = &stage[kLatStages - 1][0];
    for (int ii = wu; ii < nq; ii += 4) {
      int qc = ii * 64 + lane;
      qc = qc < qchunks ? qc : 0;  // the last instruction's spare lanes re-read chunk 0
      dma16_lat<NT>(qsrc + (size_t)qc * 16, qdst + (size_t)ii * 1024);
    }
    const int pro = min(nblk, kLatStages - 1);
    for (int s = 0; s < pro; ++s) issue(s);
    // block 0 (and every older load: the query) has landed
    if (pro == 3)
      lat_wait_vm<2 * kLatLoadsPerWave>();
    else if (pro == 2)
      lat_wait_vm<kLatLoadsPerWave>();
    else
      lat_wait_vm<0>();
    lat_barrier();
#pragma unroll
    for (int t = 0; t < kMlaKSteps; ++t) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (hval) v = *(const u32x4*)(qdst + (size_t)h * kLatRowBytes + 8 * (kMlaKSteps * lg + t) * 2);
      qf[t] = __builtin_bit_cast(bf16x8, v);
    }
    lat_barrier();  // every wave has its query fragments: the last stage is free
    if (nblk > kLatStages - 1) issue(kLatStages - 1);
  }

  for (int i = 0; i < nblk; ++i) {
    const int after = min(nblk - 1 - i, kLatStages - 1);  // block loads issued after block i
    if (after >= 3)
      lat_wait_vm<3 * kLatLoadsPerWave>();
    else if (after == 2)
      lat_wait_vm<2 * kLatLoadsPerWave>();
    else if (after == 1)
      lat_wait_vm<kLatLoadsPerWave>();
    else
      lat_wait_vm<0>();
    lat_barrier();  // block i is in LDS for every wave
    const unsigned char* st = &stage[i % kLatStages][0];
    const int vb = 32 * (chunk + i * a.n_chunks);

    f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int t = 0; t < kMlaKSteps; ++t) {
      const int c = kMlaKSteps * lg + t;
      const bf16x8 k0 = __builtin_bit_cast(bf16x8, *(const u32x4*)(st + (size_t)lat_slot(l16, c) * 16));
      const bf16x8 k1 = __builtin_bit_cast(bf16x8, *(const u32x4*)(st + (size_t)lat_slot(16 + l16, c) * 16));
      s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k0, qf[t], s0, 0, 0, 0);
      s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k1, qf[t], s1, 0, 0, 0);
    }
    // raw dot products; the scale (> 0) is applied to the block max and folded
    // into the exponent
    float x[8];
    if (vb + 32 <= sp.nv) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x[e] = s0[e];
        x[4 + e] = s1[e];
      }
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x[e] = (vb + 4 * lg + e < sp.nv) ? s0[e] : -INFINITY;
        x[4 + e] = (vb + 16 + 4 * lg + e < sp.nv) ? s1[e] : -INFINITY;
      }
    }
    float bm = fmaxf(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])), fmaxf(fmaxf(x[4], x[5]), fmaxf(x[6], x[7])));
    bm = fmaxf(bm, __shfl_xor(bm, 16));
    bm = fmaxf(bm, __shfl_xor(bm, 32));
    bm *= xs;
    const bool up = bm > m + kStaleMax;  // always true for the first valid block (m = -inf)
    if (wave_any(up)) {
      const float mnew = up ? bm : m;
      const float alpha = up ? fast_exp2(m - mnew) : 1.f;
#pragma unroll
      for (int c = 0; c < 8; ++c) acc[c] *= alpha;
      lsum *= alpha;
      m = mnew;
      mref = m == -INFINITY ? 0.f : m;  // no valid row yet: every x is -inf, exp2 gives 0
    }
    float pe[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) pe[k] = fast_exp2(fmaf(x[k], xs, -mref));
    lsum += ((pe[0] + pe[1]) + (pe[2] + pe[3])) + ((pe[4] + pe[5]) + (pe[6] + pe[7]));
    u32x4 pw;
#pragma unroll
    for (int k = 0; k < 4; ++k) pw[k] = pack_bf16x2(pe[2 * k], pe[2 * k + 1]);
    const bf16x8 pb = __builtin_bit_cast(bf16x8, pw);
    u32x4 vv[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int r = k < 4 ? 4 * lg + k : 16 + 4 * lg + (k - 4);
      vv[k] = *(const u32x4*)(st + (size_t)lat_slot(r, 16 * w + l16) * 16);
    }
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      const int u = c >> 1;
      const uint32_t selb = (c & 1) ? 0x07060302u : 0x05040100u;
      u32x4 av;
#pragma unroll
      for (int k = 0; k < 4; ++k) av[k] = __builtin_amdgcn_perm(vv[2 * k + 1][u], vv[2 * k][u], selb);
      acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, av), pb, acc[c], 0, 0, 0);
    }
    lat_barrier();  // every wave is done with this stage
    if (i + kLatStages < nblk) issue(i + kLatStages);
  }
  lsum += __shfl_xor(lsum, 16);
  lsum += __shfl_xor(lsum, 32);
  // the new row's store waits until here: its load is then long done, and no
  // other workgroup of this launch reads that row
  if (has_newp) new_piece_store(a, 0, slot, vnew, tid(), newp);
  if (!hval) return;
  const size_t pi = ((size_t)b * a.Hq + h) * a.n_chunks + chunk;
  if (w == 0 && lg == 0) a.ml[pi] = make_float2(m, lsum);
  float* dst = a.part + pi * a.dv + 128 * w;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    float4 lo = make_float4(acc[0][e], acc[1][e], acc[2][e], acc[3][e]);
    float4 hi = make_float4(acc[4][e], acc[5][e], acc[6][e], acc[7][e]);
    float* d = dst + 8 * (4 * lg + e);
    *(float4*)d = lo;
    *(float4*)(d + 4) = hi;
  }
}

// ---------------------------------------------------------------- generic decode
template <typename KV>
__device__ __forceinline__ float load_kv(const void* base, size_t i, float scale) {
  if constexpr (sizeof(KV) == 4) return ((const float*)base)[i];
  else if constexpr (sizeof(KV) == 2) return bf16_bits_to_f32(((const uint16_t*)base)[i]);
  else return e4m3_to_f32(((const uint8_t*)base)[i]) * scale;
}

// One wave per (chunk, sequence, query head); lane owns dims lane + 64*i.
template <typename KV>
__global__ __launch_bounds__(64) void decode_generic(DecodeArgs a) {
  constexpr int kMaxDk = 9, kMaxDv = 8;  // dk <= 576, dv <= 512
  const int lane = tid();
  const int chunk = bid_x(), bh = bid_y(), b = bh / a.Hq, qh = bh % a.Hq, g = qh / a.G;
  int slot;
  RowSpan sp;
  if (!span_of(a, b, chunk, slot, sp)) return;
  const int sr = a.sink + a.recent, B = sr + a.topk;
  const size_t row0 = ((size_t)slot * a.Hkv + g) * (size_t)B;
  const float ksc = sizeof(KV) == 1 ? a.k_scale[(size_t)slot * a.Hkv + g] : 1.f;
  const float vsc = sizeof(KV) == 1 ? (a.cv ? a.v_scale : a.k_scale)[(size_t)slot * a.Hkv + g] : 1.f;
  const void* vbase = a.cv ? a.cv : a.ck;
  const int vstride = a.cv ? a.dv : a.dk;
  float qv[kMaxDk];
#pragma unroll
  for (int i = 0; i < kMaxDk; ++i) {
    int d = lane + 64 * i;
    float x = 0.f;
    if (d < a.dk) {
      size_t qi = ((size_t)b * a.Hq + qh) * a.dk + d;
      x = a.q_f32 ? ((const float*)a.q)[qi] : bf16_bits_to_f32(((const uint16_t*)a.q)[qi]);
    }
    qv[i] = x;
  }
  float acc[kMaxDv];
#pragma unroll
  for (int i = 0; i < kMaxDv; ++i) acc[i] = 0.f;
  float m = -INFINITY, lsum = 0.f;
  const float xs = a.scale * kLog2e;
  for (int v = sp.v0; v < sp.v1; ++v) {
    const size_t row = row0 + virt_row(v, sp.n1, sr);
    float dot = 0.f;
#pragma unroll
    for (int i = 0; i < kMaxDk; ++i) {
      int d = lane + 64 * i;
      if (d < a.dk) dot = fmaf(qv[i], load_kv<KV>(a.ck, row * a.dk + d, ksc), dot);
    }
    dot = warp_sum(dot);
    const float x = dot * xs;
    const float mn = fmaxf(m, x);
    const float alpha = fast_exp2(m - mn);
    const float pe = fast_exp2(x - mn);
    lsum = lsum * alpha + pe;
    m = mn;
#pragma unroll
    for (int i = 0; i < kMaxDv; ++i) {
      int d = lane + 64 * i;
      float vx = d < a.dv ? load_kv<KV>(vbase, row * vstride + d, vsc) : 0.f;
      acc[i] = fmaf(pe, vx, acc[i] * alpha);
    }
  }
  const size_t pi = ((size_t)b * a.Hq + qh) * a.n_chunks + chunk;
  if (lane == 0) a.ml[pi] = make_float2(m, lsum);
  float* dst = a.part + pi * a.dv;
#pragma unroll
  for (int i = 0; i < kMaxDv; ++i) {
    int d = lane + 64 * i;
    if (d < a.dv) dst[d] = acc[i];
  }
}

// ---------------------------------------------------------------- combine
struct CombineArgs {
  const float* part;
  const float2* ml;
  const int32_t* slot_ids;
  void* out;  // [n][Hq][dv]
  int Hq, dv, n_chunks, n_slots, out_bf16;
};

constexpr int kMaxChunks = 512;
constexpr int kCombineThreads = 128;
constexpr int kCombineRegChunks = 32;  // partials loaded ahead into registers
// grid (n * Hq, ceil(dv / 128)): the chunk weights exp2(m_c - M) are formed
// once per workgroup in LDS, then each thread sums its value dim over chunks.
// The thread's first 32 partials are loaded before the weights are formed, so
// their latency overlaps the (m, l) loads and reductions instead of following
// them.
__global__ __launch_bounds__(kCombineThreads) void combine(CombineArgs a) {
  __shared__ float wts[kMaxChunks];
  __shared__ float red[kCombineThreads / 64];
  const int bh = bid_x(), b = bh / a.Hq;
  const int slot = a.slot_ids[b];
  if (slot < 0 || slot >= a.n_slots) return;
  if (!debug_check(a.n_chunks <= kMaxChunks, kDbgCombine)) return;
  const int lane = tid() & 63, wave = tid() >> 6;
  const int d = bid_y() * kCombineThreads + tid();
  const float* part = a.part + (size_t)bh * a.n_chunks * a.dv + d;
  const int nreg = d < a.dv ? min(a.n_chunks, kCombineRegChunks) : 0;
  float pr[kCombineRegChunks];
#pragma unroll
  for (int c = 0; c < kCombineRegChunks; ++c) pr[c] = c < nreg ? part[(size_t)c * a.dv] : 0.f;
  // the (m, l) of this thread's chunks tid, tid + 128, ... are loaded once
  const float2* ml = a.ml + (size_t)bh * a.n_chunks;
  constexpr int kMlPerThread = kMaxChunks / kCombineThreads;
  float2 mlv[kMlPerThread];
  float M = -INFINITY;
#pragma unroll
  for (int i = 0; i < kMlPerThread; ++i) {
    const int c = tid() + kCombineThreads * i;
    mlv[i] = c < a.n_chunks ? ml[c] : make_float2(-INFINITY, 0.f);
    M = fmaxf(M, mlv[i].x);
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) M = fmaxf(M, __shfl_xor(M, o));
  if (lane == 0) red[wave] = M;
  __syncthreads();
  M = red[0];
  for (int i = 1; i < kCombineThreads / 64; ++i) M = fmaxf(M, red[i]);
  __syncthreads();
  float ws = 0.f;
#pragma unroll
  for (int i = 0; i < kMlPerThread; ++i) {
    const int c = tid() + kCombineThreads * i;
    const float2 v = mlv[i];
    const float wc = (v.x == -INFINITY || M == -INFINITY) ? 0.f : fast_exp2(v.x - M);
    if (c < a.n_chunks) wts[c] = wc;
    ws += wc * v.y;
  }
  ws = warp_sum(ws);
  if (lane == 0) red[wave] = ws;
  __syncthreads();
  float wsum = 0.f;
  for (int i = 0; i < kCombineThreads / 64; ++i) wsum += red[i];
  const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
  if (d >= a.dv) return;
  // four accumulators over chunks c = 0, 4, 8, ... / 1, 5, ... (groups of
  // four while they are whole), the remaining chunks into the first
  float o0 = 0.f, o1 = 0.f, o2 = 0.f, o3 = 0.f;
  const int nfull = a.n_chunks & ~3;
#pragma unroll
  for (int cc = 0; cc < kCombineRegChunks; cc += 4) {
    if (cc + 4 <= nfull) {
      o0 = fmaf(wts[cc], pr[cc], o0);
      o1 = fmaf(wts[cc + 1], pr[cc + 1], o1);
      o2 = fmaf(wts[cc + 2], pr[cc + 2], o2);
      o3 = fmaf(wts[cc + 3], pr[cc + 3], o3);
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (cc + e < nreg) o0 = fmaf(wts[cc + e], pr[cc + e], o0);
    }
  }
  int c = kCombineRegChunks;
  for (; c + 4 <= a.n_chunks; c += 4) {
    o0 = fmaf(wts[c], part[(size_t)c * a.dv], o0);
    o1 = fmaf(wts[c + 1], part[(size_t)(c + 1) * a.dv], o1);
    o2 = fmaf(wts[c + 2], part[(size_t)(c + 2) * a.dv], o2);
    o3 = fmaf(wts[c + 3], part[(size_t)(c + 3) * a.dv], o3);
  }
  for (; c < a.n_chunks; ++c) o0 = fmaf(wts[c], part[(size_t)c * a.dv], o0);
  const float o = ((o0 + o1) + (o2 + o3)) * inv;
  const size_t oi = (size_t)bh * a.dv + d;
  if (a.out_bf16)
    ((uint16_t*)a.out)[oi] = (uint16_t)f32_to_bf16_bits(o);
  else
    ((float*)a.out)[oi] = o;
}

// ---------------------------------------------------------------- merge of the chunks
// The same merge as combine, with every load in flight at once, for calls of
// up to 16 chunks (the 128k batches' 8 and 16) and for calls split into more
// chunks than combine keeps in registers (a small batch spread over every CU
// in short chunks).  One 256-thread workgroup per (sequence, query head) and
// slice of DV value dims (d_v / DV slices: one, or four for 512-wide latent
// rows).  Thread t takes the slice's dims 4*(t % DG) .. 4*(t % DG) + 3 of
// chunks t / DG, t / DG + CL, ...: every partial and (m, l) load it needs is
// issued before the first is used, it merges its chunks against their
// largest reference, and the CL merges of each dim group are merged once
// more through LDS.  The slot id is tested after the barrier, so its load and
// the partial loads are in flight together (a skipped slot's workgroup merges
// what its workspace rows hold and stores nothing).
constexpr int kMergeThreads = 256;
constexpr int kMergeMaxChunks = 128;

template <int DV>
__global__ __launch_bounds__(kMergeThreads) void merge_chunks(CombineArgs a) {
  constexpr int DG = DV / 4;                 // float4 groups of a partial row
  constexpr int CL = kMergeThreads / DG;     // chunk lanes
  constexpr int PER = kMergeMaxChunks / CL;  // chunks per thread, at most
  __shared__ float4 sacc[kMergeThreads];
  __shared__ float2 sml[kMergeThreads];
  const int bh = bid_x(), b = bh / a.Hq;
  const int slot = a.slot_ids[b];
  if (!debug_check(a.n_chunks <= kMergeMaxChunks && a.dv % DV == 0, kDbgCombine)) return;
  const int t = tid(), dg = t % DG, cl = t / DG;
  const int d0 = bid_y() * DV;  // first value dim of the slice
  const int RG = a.dv / 4;      // float4 groups of a whole partial row
  const float4* part = (const float4*)(a.part + (size_t)bh * a.n_chunks * a.dv + d0) + dg;
  const float2* ml = a.ml + (size_t)bh * a.n_chunks;
  float4 pv[PER];
  float2 mv[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int c = cl + CL * i;
    pv[i] = c < a.n_chunks ? part[(size_t)c * RG] : make_float4(0.f, 0.f, 0.f, 0.f);
    mv[i] = c < a.n_chunks ? ml[c] : make_float2(-INFINITY, 0.f);
  }
  float m = -INFINITY;
#pragma unroll
  for (int i = 0; i < PER; ++i) m = fmaxf(m, mv[i].x);
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  float l = 0.f;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const float w = mv[i].x == -INFINITY ? 0.f : fast_exp2(mv[i].x - m);
    acc.x = fmaf(w, pv[i].x, acc.x);
    acc.y = fmaf(w, pv[i].y, acc.y);
    acc.z = fmaf(w, pv[i].z, acc.z);
    acc.w = fmaf(w, pv[i].w, acc.w);
    l = fmaf(w, mv[i].y, l);
  }
  sacc[t] = acc;
  sml[t] = make_float2(m, l);
  __syncthreads();
  if (cl != 0 || slot < 0 || slot >= a.n_slots) return;
  float M = -INFINITY;
#pragma unroll
  for (int j = 0; j < CL; ++j) M = fmaxf(M, sml[dg + DG * j].x);
  float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
  float L = 0.f;
#pragma unroll
  for (int j = 0; j < CL; ++j) {
    const float2 mj = sml[dg + DG * j];
    const float w = mj.x == -INFINITY ? 0.f : fast_exp2(mj.x - M);
    const float4 aj = sacc[dg + DG * j];
    o.x = fmaf(w, aj.x, o.x);
    o.y = fmaf(w, aj.y, o.y);
    o.z = fmaf(w, aj.z, o.z);
    o.w = fmaf(w, aj.w, o.w);
    L = fmaf(w, mj.y, L);
  }
  const float inv = L > 0.f ? 1.f / L : 0.f;
  const size_t oi = (size_t)bh * a.dv + d0 + 4 * dg;
  if (a.out_bf16) {
    const u32x2 w2 = {f32_to_bf16_bits(o.x * inv) | (f32_to_bf16_bits(o.y * inv) << 16),
                      f32_to_bf16_bits(o.z * inv) | (f32_to_bf16_bits(o.w * inv) << 16)};
    *(u32x2*)((uint16_t*)a.out + oi) = w2;
  } else {
    *(float4*)((float*)a.out + oi) = make_float4(o.x * inv, o.y * inv, o.z * inv, o.w * inv);
  }
}

// ---------------------------------------------------------------- append / advance
struct AppendArgs {
  const void* k_new;  // [n][Hkv][dk]
  const void* v_new;  // [n][Hkv][dv] or NULL
  void* ck;
  void* cv;
  const float* k_scale;
  const float* v_scale;
  const int32_t* pos;
  const int32_t* slot_ids;
  int Hkv, dk, dv, sink, recent, topk, n_slots;
};

template <typename In, typename Out>
__device__ __forceinline__ void put8(const In* src, Out* dst, float scale) {
  if constexpr (sizeof(Out) == 1 && sizeof(In) == 2) {
    *(u32x2*)dst = bf16x8_to_e4m3x8(*(const u32x4*)src, scale);
  } else if constexpr (sizeof(Out) == 1) {
    float f[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) f[i] = ((const float*)src)[i];
    u32x2 o;
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2) {
      uint32_t w = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) w |= f32_to_e4m3(f[h2 * 4 + i] / scale) << (8 * i);
      o[h2] = w;
    }
    *(u32x2*)dst = o;
  } else if constexpr (sizeof(In) == 2) {
    *(u32x4*)dst = *(const u32x4*)src;
  } else {
    *(u32x4*)dst = *(const u32x4*)src;
    *(u32x4*)((float*)dst + 4) = *(const u32x4*)((const float*)src + 4);
  }
}

template <typename In, typename Out>
__global__ __launch_bounds__(256) void append(AppendArgs a) {
  const int b = bid_x();
  const int slot = a.slot_ids[b];
  if (slot < 0 || slot >= a.n_slots) return;
  const int p = a.pos[slot];
  if (p < 0) return;
  const int s = a.sink, r = a.recent, B = s + r + a.topk;
  const int row = p < s ? p : s + (p - s) % r;
  if (!debug_check(row < s + r, kDbgAppend)) return;
  const int kc = a.dk / 8, vc = a.v_new ? a.dv / 8 : 0;
  for (int i = tid(); i < a.Hkv * (kc + vc); i += nthreads()) {
    const int g = i / (kc + vc), c = i % (kc + vc);
    const size_t crow = ((size_t)slot * a.Hkv + g) * (size_t)B + row;
    if (c < kc) {
      const float sc = sizeof(Out) == 1 ? a.k_scale[(size_t)slot * a.Hkv + g] : 1.f;
      put8<In, Out>((const In*)a.k_new + ((size_t)b * a.Hkv + g) * a.dk + 8 * c,
                    (Out*)a.ck + crow * a.dk + 8 * c, sc);
    } else {
      const int cc = c - kc;
      const float sc = sizeof(Out) == 1 ? a.v_scale[(size_t)slot * a.Hkv + g] : 1.f;
      put8<In, Out>((const In*)a.v_new + ((size_t)b * a.Hkv + g) * a.dv + 8 * cc,
                    (Out*)a.cv + crow * a.dv + 8 * cc, sc);
    }
  }
}

__global__ __launch_bounds__(256) void advance(int32_t* pos, int n_slots, int n, const int32_t* slot_ids) {
  for (int b = tid(); b < n; b += nthreads()) {  // one workgroup
    int s = slot_ids[b];
    if (s >= 0 && s < n_slots) atomicAdd(&pos[s], 1);
  }
}

// ---------------------------------------------------------------- host side
static inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

SNAP_DEBUG_READER(debug_flags_decode)

// workgroups per call for the LDS-staged latent decode: one per CU, all
// resident at once (more, smaller chunks measured slower: each workgroup pays
// its prologue and the combine grows)
constexpr int kLatentLdsWGs = 256;
// with the SNAP_KV_AUTO hint, decode calls reading at least this many cache
// bytes (at the full budget) use streaming loads: half the 256 MB last-level
// cache
constexpr size_t kStreamingCallBytes = (size_t)128 << 20;

Geometry decode_geometry(const snap_params& p, int n) {
  Geometry g{};
  const int B = p.sink + p.recent + p.topk;
  const int units = (n > 0 ? n : 1) * p.n_kv_heads;
  // latent caches run 4-wave workgroups (two per CU), the others one wave each
  const bool latent = p.v_in_k && p.d_qk == 576;
  const bool latent_lds = latent && p.kv_dtype == SNAP_BF16;  // one 4-wave workgroup per CU (LDS-bound)
  const int target = latent_lds ? kLatentLdsWGs : (latent ? 512 : 2048);
  // rounded down: a grid just above the resident capacity would leave a
  // partial second round of workgroups (measured 25% slower on the fp8 GQA
  // kernel at 248 units: 9 chunks against 8)
  const int want = target / units;
  // a small GQA batch (more chunks wanted than combine keeps in registers)
  // splits into chunks as short as one 32-row block, up to what merge_chunks
  // holds, so that a launch-bound call spreads over more waves
  const bool many = !latent && want > kCombineRegChunks;
  const int min_rows = latent ? 256 : (many ? 32 : 128);
  int maxc = (B + min_rows - 1) / min_rows;
  if (maxc < 1) maxc = 1;
  if (maxc > (many ? kMergeMaxChunks : kMaxChunks)) maxc = many ? kMergeMaxChunks : kMaxChunks;
  g.n_chunks = want < 1 ? 1 : (want > maxc ? maxc : want);
  // merge_chunks takes every call of at most 16 chunks and of 33 to 128
  // (small batches; also a few latent sequences, whose chunks are never
  // shorter than 256 rows); combine takes 17 to 32 chunks, where it measured
  // faster (the 8-sequence GQA batch's 32 chunks: 3%), and more than 128
  g.merge_many = (g.n_chunks <= 16 || g.n_chunks > kCombineRegChunks) && g.n_chunks <= kMergeMaxChunks;
  size_t off = 0;
  g.off_part = off;
  off = align256(off + (size_t)(n > 0 ? n : 1) * p.n_q_heads * g.n_chunks * p.d_v * sizeof(float));
  g.off_ml = off;
  off = align256(off + (size_t)(n > 0 ? n : 1) * p.n_q_heads * g.n_chunks * sizeof(float2));
  g.decode_bytes = off;
  return g;
}

snap_status launch_decode(const snap_params& p, const snap_cache& c, const int32_t* pos, const int32_t* n_topk,
                          int n, const int32_t* slot_ids, const void* q, const void* k_new, const void* v_new,
                          void* out, int out_dtype, void* ws, hipStream_t stream) {
  Geometry geo = decode_geometry(p, n);
  DecodeArgs a;
  a.q = q;
  a.ck = c.k;
  a.cv = p.v_in_k ? nullptr : c.v;
  a.k_scale = c.k_scale;
  a.v_scale = c.v_scale;
  a.pos = pos;
  a.n_topk = n_topk;
  a.slot_ids = slot_ids;
  a.part = (float*)((unsigned char*)ws + geo.off_part);
  a.ml = (float2*)((unsigned char*)ws + geo.off_ml);
  a.Hq = p.n_q_heads;
  a.Hkv = p.n_kv_heads;
  a.G = p.n_q_heads / p.n_kv_heads;
  a.dk = p.d_qk;
  a.dv = p.d_v;
  a.sink = p.sink;
  a.recent = p.recent;
  a.topk = p.topk;
  a.n_slots = c.n_slots;
  a.n_chunks = geo.n_chunks;
  a.q_f32 = p.in_dtype == SNAP_F32;
  a.scale = p.sm_scale > 0.f ? p.sm_scale : 1.0f / sqrtf((float)p.d_qk);
  a.k_new = nullptr;
  a.v_new = nullptr;

  const bool mfma_ok = p.in_dtype == SNAP_BF16 && !p.v_in_k && p.d_qk == 128 && p.d_v == 128 &&
                       (p.kv_dtype == SNAP_BF16 || p.kv_dtype == SNAP_FP8_E4M3);
  const bool mla_ok = p.in_dtype == SNAP_BF16 && p.v_in_k && p.n_kv_heads == 1 && p.d_qk == 576 && p.d_v == 512 &&
                      (p.kv_dtype == SNAP_BF16 || p.kv_dtype == SNAP_FP8_E4M3);
  if (k_new) {
    // the MFMA kernels (GQA: bf16 and fp8 caches; latent: bf16) take the new
    // token in the same launch; the others run the append kernel first (same
    // result)
    if (mfma_ok || (mla_ok && p.kv_dtype == SNAP_BF16)) {
      a.k_new = k_new;
      a.v_new = p.v_in_k ? nullptr : v_new;
    } else {
      const snap_status st = launch_append(p, c, pos, n, slot_ids, k_new, v_new, stream);
      if (st != SNAP_OK) return st;
    }
  }
  // streaming loads as the caller's hint says, or by default when the call's
  // cache rows (at the full budget) exceed what the last-level cache could
  // keep for the next call
  const size_t elt = p.kv_dtype == SNAP_F32 ? 4 : (p.kv_dtype == SNAP_BF16 ? 2 : 1);
  const size_t call_bytes = (size_t)n * p.n_kv_heads * (size_t)(p.sink + p.recent + p.topk) *
                            (size_t)(p.d_qk + (p.v_in_k ? 0 : p.d_v)) * elt;
  const bool nt = p.kv_reuse == SNAP_KV_STREAM || (p.kv_reuse == SNAP_KV_AUTO && call_bytes >= kStreamingCallBytes);
  if (mla_ok) {
    dim3 grid(geo.n_chunks, n);
    void (*k)(DecodeArgs);
    if (p.kv_dtype == SNAP_FP8_E4M3)
      k = nt ? decode_mla<true, true> : decode_mla<true, false>;
    else
      k = nt ? decode_mla_lds<true> : decode_mla_lds<false>;
    hipLaunchKernelGGL(k, grid, dim3(256), 0, stream, a);
  } else if (mfma_ok) {
    dim3 grid(geo.n_chunks, n * p.n_kv_heads);
    void (*k)(DecodeArgs);
    if (p.kv_dtype == SNAP_FP8_E4M3 && p.fp8_qk)
      k = nt ? decode_mfma<4, 1, true, true, true> : decode_mfma<4, 1, true, true, false>;
    else if (p.kv_dtype == SNAP_FP8_E4M3)
      k = nt ? decode_mfma<4, 1, true, false, true> : decode_mfma<4, 1, true, false, false>;
    else
      k = nt ? decode_mfma<4, 1, false, false, true> : decode_mfma<4, 1, false, false, false>;
    hipLaunchKernelGGL(k, grid, dim3(64), 0, stream, a);
  } else {
    dim3 grid(geo.n_chunks, n * p.n_q_heads);
    if (p.kv_dtype == SNAP_F32)
      hipLaunchKernelGGL((decode_generic<float>), grid, dim3(64), 0, stream, a);
    else if (p.kv_dtype == SNAP_BF16)
      hipLaunchKernelGGL((decode_generic<uint16_t>), grid, dim3(64), 0, stream, a);
    else
      hipLaunchKernelGGL((decode_generic<uint8_t>), grid, dim3(64), 0, stream, a);
  }
  if (hipGetLastError() != hipSuccess) return SNAP_ERR_HIP;
  CombineArgs ca;
  ca.part = a.part;
  ca.ml = a.ml;
  ca.slot_ids = slot_ids;
  ca.out = out;
  ca.Hq = p.n_q_heads;
  ca.dv = p.d_v;
  ca.n_chunks = geo.n_chunks;
  ca.n_slots = c.n_slots;
  ca.out_bf16 = out_dtype == SNAP_BF16;
  if (geo.merge_many && p.d_v == 64)
    hipLaunchKernelGGL(merge_chunks<64>, dim3(n * p.n_q_heads), dim3(kMergeThreads), 0, stream, ca);
  else if (geo.merge_many)  // d_v = 128 or 512: 128-dim slices
    hipLaunchKernelGGL(merge_chunks<128>, dim3(n * p.n_q_heads, p.d_v / 128), dim3(kMergeThreads), 0, stream, ca);
  else
    hipLaunchKernelGGL(combine, dim3(n * p.n_q_heads, (p.d_v + kCombineThreads - 1) / kCombineThreads),
                       dim3(kCombineThreads), 0, stream, ca);
  if (hipGetLastError() != hipSuccess) return SNAP_ERR_HIP;
  return SNAP_OK;
}

snap_status launch_append(const snap_params& p, const snap_cache& c, const int32_t* pos, int n,
                          const int32_t* slot_ids, const void* k_new, const void* v_new, hipStream_t stream) {
  AppendArgs a;
  a.k_new = k_new;
  a.v_new = p.v_in_k ? nullptr : v_new;
  a.ck = c.k;
  a.cv = p.v_in_k ? nullptr : c.v;
  a.k_scale = c.k_scale;
  a.v_scale = c.v_scale;
  a.pos = pos;
  a.slot_ids = slot_ids;
  a.Hkv = p.n_kv_heads;
  a.dk = p.d_qk;
  a.dv = p.d_v;
  a.sink = p.sink;
  a.recent = p.recent;
  a.topk = p.topk;
  a.n_slots = c.n_slots;
  if (p.kv_dtype == SNAP_FP8_E4M3)
    hipLaunchKernelGGL((append<uint16_t, uint8_t>), dim3(n), dim3(256), 0, stream, a);
  else if (p.kv_dtype == SNAP_BF16)
    hipLaunchKernelGGL((append<uint16_t, uint16_t>), dim3(n), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL((append<float, float>), dim3(n), dim3(256), 0, stream, a);
  return hipGetLastError() == hipSuccess ? SNAP_OK : SNAP_ERR_HIP;
}

snap_status launch_advance(int32_t* pos, int n_slots, int n, const int32_t* slot_ids, hipStream_t stream) {
  hipLaunchKernelGGL(advance, dim3(1), dim3(256), 0, stream, pos, n_slots, n, slot_ids);
  return hipGetLastError() == hipSuccess ? SNAP_OK : SNAP_ERR_HIP;
}

}  // namespace snap
