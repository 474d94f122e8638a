// compress.hip -- SnapStream compression at the end of prefill (arXiv
// 2511.03092, Sec. III-B): SnapKV window scores (Eq. 3), window + group sum
// (Eq. 1), 1-D pooling and top-K (Eq. 2), then the gather into the fixed-size
// sink / ring / top-K cache (Sec. III-A).
//
// Kernel sequence per call (one stream, no host synchronisation):
//   score_pass<STATS>   per (seq, KV head, key chunk): bf16 MFMA Q_obs x K^T,
//                       per-row running max / sum-exp of the softmax domain
//                       (skipped after the prefill attention, which writes
//                       those statistics itself)
//   stats_reduce        per (seq, KV head): row max + normaliser (fp64), and
//                       the reset of the selection scratch
//   score_pass<COLSUM>  recompute the scores, W = exp(z - c) * inv, column
//                       sums over the G*w window rows -> A[j]
//   pool_hist0          P = pool(A) over the candidates, histogram of the
//                       first radix digit
//   radix_scan x3       per (seq, KV head): pick the bin holding the K-th
//                       largest P for the digit just counted
//   radix_pass x2       histograms of the remaining digits (LDS per wave)
//   select_count/write  ordered compaction: P > t, plus the lowest-index ties
//   assemble            sinks, ring rows, kept rows, zero padding (+ fp8)
#include <float.h>
#include <math.h>

#include "lds_dma.h"
#include "snap_internal.h"

namespace snap {

// ============================================================ score passes
struct ScoreArgs {
  const void* q;        // [n_seq][Hq][w][D]
  const void* k;        // [n_seq][Hkv][max_len][D]
  const int32_t* lengths;
  float2* stats;        // [n_seq*Hkv][n_kchunks][rows_pad]  (max, sum exp)
  const float2* rowref; // [n_seq*Hkv][rows_pad]             (c, inv)
  float* A;             // [n_seq*Hkv][max_len]
  int Hq, Hkv, G, w, max_len, sink, recent, norm;
  int rows, rows_pad, key_chunk, n_kchunks;
  float scale;   // softmax scale
  float scale2;     // scale * log2(e) rounded to fp32 toward zero: logits in log2 units
  float scale2_lo;  // scale * log2(e) - scale2, > 0 (see split_scale2)
};

struct ScoreLane {
  int rpos[2][4];
  bool rval[2][4];
  float rm[2][4], rz[2][4], rc[2][4], rinv[2][4], rinvl[2][4];  // rinvl = rinv * ln2
};

// Normalised weight of one logit: 2^(y - c) * inv with y = acc * (s2 + s2lo).
// y is formed as the rounded product yh plus its exact error and the part of
// scale*log2(e) that fp32 s2 dropped; that small remainder enters to first
// order, 2^(yh + yl - c) = 2^(yh - c) * (1 + yl*ln2), folded into the row factor.
// No contraction here: fused into fma(acc, s2, -c), yh - c would no longer
// carry the rounding of yh that yl corrects, and for c != 0 that error would
// be counted twice.
__device__ __forceinline__ float weight(float acc, float s2, float s2lo, float c, float inv, float invl) {
#pragma clang fp contract(off)
  const float yh = acc * s2;
  float yl = fmaf(acc, s2, -yh);
  yl = fmaf(acc, s2lo, yl);
  return fast_exp2(yh - c) * fmaf(yl, invl, inv);
}

// Scores of one TK-key tile already resident in LDS against this wave's 32
// rows, then either the running row max / sum of powers of two (STATS) or the
// column sums of the normalised weights written to A (COLSUM).  Logits are
// kept in log2 units, y = <q,k> * scale * log2(e), formed by one rounded
// multiply, so exp(z) = exp2(y).  `interior` (uniform) means every key of the
// tile is a candidate that precedes every window row: no per-element masks.
// The work is split per 16-key sub-block into the products (score_mma_sb) and
// the softmax arithmetic (score_epi_sb), so a caller can run the two halves of
// a tile at different times.
//
// LDS fragment reads issued ahead of their MFMAs (measured: 4 is 4% faster
// than the scheduler's own 2 on the latent shape; 6 is no better).
constexpr int kReadAhead = 4;

// Products of sub-block sb (keys sb*16 .. sb*16+15 of the tile): acc[rb] holds
// rows rb*16 + 4*(lane/16) + e (e = 0..3) against key sb*16 + lane%16.
template <typename In, int KSTEPS, int TK>
__device__ __forceinline__ void score_mma_sb(const unsigned char* __restrict__ ktile, const bf16x8 (&qf)[2][KSTEPS],
                                             const float* qlds, int sb, int wave, int lane, bool wave_has_rows,
                                             f32x4 (&acc)[2]) {
  constexpr bool kBF16 = sizeof(In) == 2;
  constexpr int D = KSTEPS * 32;
  const int l16 = lane & 15, lg = lane >> 4;
  const int key = sb * 16 + l16;
  acc[0] = f32x4{0.f, 0.f, 0.f, 0.f};
  acc[1] = f32x4{0.f, 0.f, 0.f, 0.f};
  if constexpr (kBF16) {
    // waves without score rows multiply zero fragments (only tiny cases have them).
    // Even and odd k-steps accumulate in separate chains (shorter fp32
    // accumulation, two independent MFMA chains), summed at the end.
    f32x4 odd[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
#pragma unroll
    for (int t = 0; t < KSTEPS; ++t) {
      bf16x8 kf = __builtin_bit_cast(bf16x8, *(const u32x4*)(ktile + (size_t)tile_slot<TK>(key, KSTEPS * lg + t) * 16));
      if (t & 1) {
        odd[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qf[0][t], kf, odd[0], 0, 0, 0);
        odd[1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qf[1][t], kf, odd[1], 0, 0, 0);
      } else {
        acc[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qf[0][t], kf, acc[0], 0, 0, 0);
        acc[1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qf[1][t], kf, acc[1], 0, 0, 0);
      }
    }
    // the fragment reads run kReadAhead k-steps ahead of the MFMAs that use
    // them, so their LDS latency hides behind earlier products
    __builtin_amdgcn_sched_group_barrier(0x100, kReadAhead, 0);  // DS reads
#pragma unroll
    for (int t = 0; t < KSTEPS - kReadAhead; ++t) {
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);  // MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 2 * kReadAhead, 0);
    acc[0] += odd[0];
    acc[1] += odd[1];
  } else if (wave_has_rows) {
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float* qrow = qlds + (size_t)(wave * 32 + rb * 16 + lg * 4 + e) * D;
        // fp32 products are exact in fp64; only the final rounding remains
        double sacc = 0.0;
#pragma unroll 4
        for (int d = 0; d < D; ++d) {
          const float kd = *(const float*)(ktile + (size_t)tile_slot<TK>(key, d >> 2) * 16 + (d & 3) * 4);
          sacc = fma((double)qrow[d], (double)kd, sacc);
        }
        acc[rb][e] = (float)sacc;
      }
  }
}

// Softmax arithmetic of sub-block sb from its products: STATS keeps the
// products (masked ones at -inf) in xv for score_stats_tile; COLSUM writes this
// wave's column sums of the normalised weights to colbuf.
template <int NW, bool COLSUM, int TK>
__device__ __forceinline__ void score_epi_sb(const ScoreArgs& a, const f32x4 (&acc)[2], float* colbuf,
                                             const ScoreLane& sl, int t0, int c1, bool interior, int sb, int wave,
                                             int lane, float (&xv)[2][4][TK / 16]) {
  const int l16 = lane & 15, lg = lane >> 4;
  const float s2 = a.scale2, s2lo = a.scale2_lo;
  const int key = sb * 16 + l16;
  const int j = t0 + key;
  if (!COLSUM) {
    // the raw products: score_stats_tile forms each exponent from them with
    // the full scale (s2 + s2lo), as the column-sum weights do
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int e = 0; e < 4; ++e) xv[rb][e][sb] = acc[rb][e];
    if (!interior) {
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (!(sl.rval[rb][e] && j < c1 && j <= sl.rpos[rb][e])) xv[rb][e][sb] = -INFINITY;
    }
  } else {
    float colv[2][4];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        colv[rb][e] = weight(acc[rb][e], s2, s2lo, sl.rc[rb][e], sl.rinv[rb][e], sl.rinvl[rb][e]);
    if (!interior) {
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (!(sl.rval[rb][e] && j < c1 && j <= sl.rpos[rb][e])) colv[rb][e] = 0.f;
    }
    float cs = ((colv[0][0] + colv[0][1]) + (colv[0][2] + colv[0][3])) +
               ((colv[1][0] + colv[1][1]) + (colv[1][2] + colv[1][3]));
    cs += __shfl_xor(cs, 16);
    cs += __shfl_xor(cs, 32);
    if (lg == 0) colbuf[wave * TK + sb * 16 + l16] = cs;
  }
}

// STATS: fold one tile's products into the running row max / sum (log2
// units).  The reference mn is the rounded max of acc * s2; each term's
// exponent acc * (s2 + s2lo) - mn is formed with two fused steps, so the row
// sum carries neither the rounding of acc * s2 nor the part of the scale that
// fp32 s2 drops -- the same logits the column-sum weights use, whose sum it
// normalises.  s2lo > 0 keeps a masked -inf product at -inf.
__device__ __forceinline__ float stats_term(float x, float s2, float s2lo, float mn) {
  return fast_exp2(fmaf(x, s2lo, fmaf(x, s2, -mn)));
}
template <int TK>
__device__ __forceinline__ void score_stats_tile(ScoreLane& sl, const float (&xv)[2][4][TK / 16], float s2,
                                                 float s2lo) {
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float* x = xv[rb][e];
      float mt, mn;
      if constexpr (TK == 64) {
        mt = fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]));
      } else {
        mt = fmaxf(x[0], x[1]);
      }
      mn = fmaxf(sl.rm[rb][e], mt * s2);
      if (mn == -INFINITY) continue;
      float z = sl.rz[rb][e] * fast_exp2(sl.rm[rb][e] - mn);
      if constexpr (TK == 64) {
        z += (stats_term(x[0], s2, s2lo, mn) + stats_term(x[1], s2, s2lo, mn)) +
             (stats_term(x[2], s2, s2lo, mn) + stats_term(x[3], s2, s2lo, mn));
      } else {
        z += stats_term(x[0], s2, s2lo, mn) + stats_term(x[1], s2, s2lo, mn);
      }
      sl.rz[rb][e] = z;
      sl.rm[rb][e] = mn;
    }
}

// The whole tile in one go: products and softmax arithmetic sub-block by
// sub-block.
template <typename In, int KSTEPS, int NW, bool COLSUM, int TK>
__device__ __forceinline__ void score_tile(const ScoreArgs& a, const unsigned char* __restrict__ ktile,
                                           const bf16x8 (&qf)[2][KSTEPS], const float* qlds, float* colbuf,
                                           ScoreLane& sl, int t0, int c1, bool interior, int bg, int wave,
                                           int lane, bool wave_has_rows) {
  static_assert(TK == 64 || TK == 32, "tile of 64 or 32 keys");
  float xv[2][4][TK / 16];
#pragma unroll
  for (int sb = 0; sb < TK / 16; ++sb) {
    f32x4 acc[2];
    score_mma_sb<In, KSTEPS, TK>(ktile, qf, qlds, sb, wave, lane, wave_has_rows, acc);
    score_epi_sb<NW, COLSUM, TK>(a, acc, colbuf, sl, t0, c1, interior, sb, wave, lane, xv);
  }
  if (!COLSUM) score_stats_tile<TK>(sl, xv, a.scale2, a.scale2_lo);
}

// Column sums of one tile across the NW waves (fixed order), written to A.
// The caller places a barrier between the waves' colbuf writes and this.
template <int NW, int TK>
__device__ __forceinline__ void colsum_finish(const ScoreArgs& a, const float* colbuf, int t0, int c1, int bg) {
  if (tid() < TK) {
    const int j = t0 + tid();
    const float* c = colbuf + tid();
    float sum;
    if constexpr (NW == 4) {
      sum = (c[0] + c[TK]) + (c[2 * TK] + c[3 * TK]);
    } else {
      sum = ((c[0] + c[TK]) + (c[2 * TK] + c[3 * TK])) + ((c[4 * TK] + c[5 * TK]) + (c[6 * TK] + c[7 * TK]));
    }
    if (j < c1) a.A[(size_t)bg * a.max_len + j] = sum;
  }
}

// Row state of one lane: the MFMA 16x16 output gives lane l the rows
// 4*(l/16)+e (e = 0..3) of each 16-row block and the key column l%16.
// NW waves per workgroup; wave w owns score rows [32w, 32w+32).  Key tiles of
// TK keys stream through a ring of STAGES LDS stages with direct loads: while
// a tile is scored, the next STAGES-1 are in flight (the bytes in flight per
// CU, not the compute, bound a pass with fewer stages).
template <typename In, int KSTEPS, int NW, bool COLSUM, int TK, int STAGES>
__global__ __launch_bounds__(NW * 64) void score_pass(ScoreArgs a) {
  constexpr bool kBF16 = sizeof(In) == 2;
  constexpr int D = KSTEPS * 32;
  constexpr int kRowBytes = D * (int)sizeof(In);
  constexpr int CPR = kRowBytes / 16;                 // 16-byte chunks per key row
  constexpr int kTileBytes = TK * kRowBytes;
  __shared__ __align__(16) unsigned char tiles[STAGES][kTileBytes];
  __shared__ float colbuf[2][NW * TK];  // column partials, double-buffered for the ring
  __shared__ float qlds[kBF16 ? 1 : 128 * D];           // fp32 inputs: [rows_pad <= 128][D]

  const int lane = tid() & 63, wave = tid() >> 6;
  const int l16 = lane & 15, lg = lane >> 4;
  const int bg = bid_y(), b = bg / a.Hkv, g = bg % a.Hkv;
  int L = uniform(a.lengths[b]);
  L = L < 0 ? 0 : (L > a.max_len ? a.max_len : L);
  const int s = a.sink, r = a.recent;
  const int clo = s, chi = L - r;  // candidates [clo, chi)
  int lo, hi;
  if (COLSUM || a.norm == SNAP_NORM_CAND) {
    lo = clo;
    hi = chi;
  } else {
    lo = 0;
    hi = L;
  }
  const int c0 = lo + bid_x() * a.key_chunk;
  int c1 = min(c0 + a.key_chunk, hi);
  if (!debug_check(c0 >= 0 && c1 <= a.max_len, kDbgScoreRange)) c1 = c0;  // skip the chunk
  const int we = min(a.w, L);
  const bool wave_has_rows = wave * 32 < a.rows;

  ScoreLane sl;
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      int rho = wave * 32 + rb * 16 + lg * 4 + e;
      int ii = rho % a.w;
      sl.rval[rb][e] = rho < a.rows && ii >= a.w - we;
      sl.rpos[rb][e] = L - a.w + ii;
    }

  float2* st_out = a.stats + ((size_t)bg * a.n_kchunks + bid_x()) * a.rows_pad;
  if (c0 >= c1) {
    if (!COLSUM) {
      for (int t = tid(); t < a.rows_pad; t += nthreads()) st_out[t] = make_float2(-INFINITY, 0.f);
    }
    return;
  }

  const unsigned char* kbase =
      (const unsigned char*)a.k + ((size_t)b * a.Hkv + g) * (size_t)a.max_len * kRowBytes;

  // ---- query rows of this wave
  const In* qbase = (const In*)a.q + ((size_t)b * a.Hq + (size_t)g * a.G) * a.w * D;
  bf16x8 qf[2][KSTEPS];
  if constexpr (kBF16) {
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      int rho = wave * 32 + rb * 16 + l16;
      int ii = rho % a.w;
      bool ok = rho < a.rows && ii >= a.w - we;
#pragma unroll
      for (int t = 0; t < KSTEPS; ++t) {
        u32x4 v = {0u, 0u, 0u, 0u};
        if (ok) v = *(const u32x4*)(qbase + (size_t)rho * D + 8 * (KSTEPS * lg + t));
        qf[rb][t] = __builtin_bit_cast(bf16x8, v);
      }
    }
  } else {
    for (int i = tid(); i < a.rows_pad * D; i += nthreads()) {
      int rho = i / D;
      qlds[i] = rho < a.rows ? ((const float*)qbase)[i] : 0.f;
    }
  }

#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      sl.rm[rb][e] = -INFINITY;
      sl.rz[rb][e] = 0.f;
      if (COLSUM) {
        int rho = wave * 32 + rb * 16 + lg * 4 + e;
        float2 rf = rho < a.rows_pad ? a.rowref[(size_t)bg * a.rows_pad + rho] : make_float2(0.f, 0.f);
        sl.rc[rb][e] = sl.rval[rb][e] ? rf.x : 0.f;  // already in log2 units
        sl.rinv[rb][e] = sl.rval[rb][e] ? rf.y : 0.f;
        sl.rinvl[rb][e] = sl.rinv[rb][e] * 0.69314718055994531f;
      }
    }
  // The query fragments and row normalisers must have landed before the first
  // tile load is issued: the loop's waits only count tile loads (stores issued
  // later only add to the count, which makes those waits stricter).
  wait_vm<0>();
  const int nt = (c1 - c0 + TK - 1) / TK;  // tiles of this chunk
  const int nload = tile_loads<CPR, NW, TK>(__builtin_amdgcn_readfirstlane(wave));
  // prologue: tile 0 (the double buffer issues each next tile inside its
  // loop), or the first STAGES-1 tiles of the ring
  for (int st = 0; st < (STAGES == 2 ? 1 : STAGES - 1) && st < nt; ++st)
    issue_tile<CPR, NW, TK>(kbase, kRowBytes, c0 + st * TK, c1, &tiles[st][0], wave, lane);

  // a tile is interior when all its keys are in range and precede the first
  // window position (rows of negative position exist only when L < w)
  const int first_row_pos = L - a.w;
  auto interior_of = [&](int t) { return t + TK <= c1 && t + TK - 1 <= first_row_pos; };

  if constexpr (STAGES == 2) {
    // double buffer, unrolled by two (tile0 <- even tiles, tile1 <- odd
    // tiles): the next tile is issued just before the current one is waited
    // for.  Measured faster than the general ring for the small-row shapes.
    constexpr int IPW = CPR * TK / 64 / NW;
    static_assert(CPR * TK / 64 % NW == 0, "equal loads per wave");
    unsigned char* tile0 = &tiles[0][0];
    unsigned char* tile1 = &tiles[1][0];
    for (int t0 = c0; t0 < c1; t0 += 2 * TK) {
      {
        lds_barrier();  // every wave is done reading tile1
        if (t0 + TK < c1) {
          issue_tile<CPR, NW, TK>(kbase, kRowBytes, t0 + TK, c1, tile1, wave, lane);
          wait_vm<IPW>();
        } else {
          wait_vm<0>();
        }
        lds_barrier();  // tile0 holds keys [t0, t0+TK)
        score_tile<In, KSTEPS, NW, COLSUM, TK>(a, tile0, qf, qlds, colbuf[0], sl, t0, c1, interior_of(t0), bg,
                                               wave, lane, wave_has_rows);
        if constexpr (COLSUM) {
          lds_barrier();
          colsum_finish<NW, TK>(a, colbuf[0], t0, c1, bg);
        }
      }
      const int t1 = t0 + TK;
      if (t1 < c1) {
        lds_barrier();  // every wave is done reading tile0
        if (t1 + TK < c1) {
          issue_tile<CPR, NW, TK>(kbase, kRowBytes, t1 + TK, c1, tile0, wave, lane);
          wait_vm<IPW>();
        } else {
          wait_vm<0>();
        }
        lds_barrier();  // tile1 holds keys [t1, t1+TK)
        score_tile<In, KSTEPS, NW, COLSUM, TK>(a, tile1, qf, qlds, colbuf[0], sl, t1, c1, interior_of(t1), bg,
                                               wave, lane, wave_has_rows);
        if constexpr (COLSUM) {
          lds_barrier();
          colsum_finish<NW, TK>(a, colbuf[0], t1, c1, bg);
        }
      }
    }
  } else {
    // Ring, one barrier per tile: past the barrier of tile i every wave has
    // finished tile i-1, so its stage takes tile i+STAGES-1 right away and
    // its column partials (the other colbuf half) can be summed.
    for (int i = 0; i < nt; ++i) {
      wait_vm_dyn(min(nt - 1 - i, STAGES - 2) * nload);  // tile i has landed
      lds_barrier();                                      // ... for every wave
      const int t = c0 + i * TK;
      if (i + STAGES - 1 < nt)
        issue_tile<CPR, NW, TK>(kbase, kRowBytes, t + (STAGES - 1) * TK, c1, &tiles[(i + STAGES - 1) % STAGES][0],
                                wave, lane);
      if constexpr (COLSUM) {
        if (i > 0) colsum_finish<NW, TK>(a, colbuf[(i - 1) & 1], t - TK, c1, bg);
      }
      score_tile<In, KSTEPS, NW, COLSUM, TK>(a, &tiles[i % STAGES][0], qf, qlds, colbuf[i & 1], sl, t, c1,
                                             interior_of(t), bg, wave, lane, wave_has_rows);
    }
    if constexpr (COLSUM) {
      lds_barrier();
      colsum_finish<NW, TK>(a, colbuf[(nt - 1) & 1], c0 + (nt - 1) * TK, c1, bg);
    }
  }

  if (!COLSUM) {
    // combine the 16 key columns of each row (lanes with equal l/16)
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float m = sl.rm[rb][e], z = sl.rz[rb][e];
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) {
          float m2 = __shfl_xor(m, o), z2 = __shfl_xor(z, o);
          float mn = fmaxf(m, m2);
          if (mn != -INFINITY) {
            z = z * fast_exp2(m - mn) + z2 * fast_exp2(m2 - mn);
            m = mn;
          }
        }
        const int rho = wave * 32 + rb * 16 + lg * 4 + e;
        if (l16 == 0 && rho < a.rows_pad) st_out[rho] = make_float2(m, z);
      }
  }
}

// ============================================================ row normalisers
struct ReduceArgs {
  const float2* stats;
  float2* rowref;
  double2* rowz;       // [groups][rows_pad] (max in log2 units, sum of 2^(y - max)) in fp64
  int32_t* band_n;     // [groups] members of the re-score band (reset here)
  const int32_t* lengths;
  uint32_t* hist;      // [3][groups][kRadixBins]
  RadixState* state;   // [groups]
  int groups, Hkv, max_len, sink, recent, topk;
  int rows_pad, n_kchunks;
};

// Row max m over every chunk and the normaliser, in log2 units (the stats
// pass keeps m2 = max y and sum 2^(y - m2) with y = z*log2(e)).  The reference
// c2 is 0 when the natural-log max lies in [-20, 64] (then 2^y is taken
// directly, keeping the full fp32 accuracy of small logits), otherwise
// c2 = m2; inv = 1 / sum_j 2^(y_j - c2), accumulated in fp64.  A wave owns a
// row (chunks strided by 64, a few hundred at most) and combines with in-wave
// shuffles; block 0 of each group also resets the group's selection scratch.
constexpr int kReduceLanes = 64;
constexpr int kReduceRows = 256 / kReduceLanes;  // rows per workgroup
__global__ __launch_bounds__(256) void stats_reduce(ReduceArgs a) {
  const int bg = bid_y(), b = bg / a.Hkv;
  const int sub = tid() % kReduceLanes;
  const int rho = bid_x() * kReduceRows + tid() / kReduceLanes;
  const float2* st = a.stats + (size_t)bg * a.n_kchunks * a.rows_pad;
  if (rho < a.rows_pad) {
    float m = -INFINITY;
    for (int c = sub; c < a.n_kchunks; c += kReduceLanes) m = fmaxf(m, st[(size_t)c * a.rows_pad + rho].x);
#pragma unroll
    for (int o = 1; o < kReduceLanes; o <<= 1) m = fmaxf(m, __shfl_xor(m, o));
    double z = 0.0;
    if (m != -INFINITY) {
      for (int c = sub; c < a.n_kchunks; c += kReduceLanes) {
        float2 v = st[(size_t)c * a.rows_pad + rho];
        if (v.x != -INFINITY) z += (double)v.y * exp2((double)v.x - (double)m);
      }
    }
#pragma unroll
    for (int o = 1; o < kReduceLanes; o <<= 1) z += __shfl_xor(z, o);
    if (sub == 0) {
      float2 ref = make_float2(0.f, 0.f);
      if (m != -INFINITY) {
        const double m_nat = (double)m * 0.69314718055994530942;
        if (m_nat >= -20.0 && m_nat <= 64.0) {
          ref.x = 0.f;
          ref.y = (float)(1.0 / (z * exp2((double)m)));
        } else {
          ref.x = m;
          ref.y = (float)(1.0 / z);
        }
      }
      a.rowref[(size_t)bg * a.rows_pad + rho] = ref;
      a.rowz[(size_t)bg * a.rows_pad + rho] = make_double2((double)m, z);
    }
  }
  if (bid_x() != 0) return;
  if (tid() == 0) a.band_n[bg] = 0;
  for (int pass = 0; pass < 3; ++pass) {
    uint32_t* h = a.hist + ((size_t)pass * a.groups + bg) * kRadixBins;
    for (int i = tid(); i < kRadixBins; i += nthreads()) h[i] = 0u;
  }
  if (tid() == 0) {
    int L = uniform(a.lengths[b]);
    L = L < 0 ? 0 : (L > a.max_len ? a.max_len : L);
    int n = L - a.sink - a.recent;
    n = n < 0 ? 0 : n;
    int keff = n < a.topk ? n : a.topk;
    RadixState s;
    s.prefix = 0u;
    s.mask = 0u;
    s.krem = keff;
    s.keff = keff;
    s.mode = keff == 0 ? 0 : (keff == n ? 1 : 2);
    s.pad[0] = s.pad[1] = s.pad[2] = 0;
    a.state[bg] = s;
  }
}

// ============================================================ pooling + selection
struct SelectArgs {
  const float* A;        // [groups][max_len]
  float* P;              // [groups][max_len]
  float* pooled_out;     // optional [groups][max_len]
  const int32_t* lengths;
  uint32_t* hist;        // [3][groups][kRadixBins]
  RadixState* state;     // [groups]
  uint2* counts;         // [groups][n_splits] (greater, equal)
  int32_t* sel;          // [groups][topk]
  int32_t* band_n;       // [groups] candidates in the re-score band
  int32_t* band_idx;     // [groups][kBandCap] their token indices (in arrival order)
  uint32_t* band_above;  // [groups][n_splits] candidates above the band per split
  int groups, Hkv, max_len, sink, recent, topk, pool_kernel, pool, n_splits;
};

// The re-score band around the K-th largest pooled score tau (fp32 bits of a
// non-negative value): [tau (1 - 2^-17), tau (1 + 2^-17)] as bit patterns.
// The fp32 score path is accurate to under 2e-6 relative (measured up to
// 1.6e-6 anywhere, 1.2e-6 near the threshold with one window row), so a
// candidate outside the band cannot be on the other side of the threshold.
constexpr float kBandRel = 1.0f / 131072.0f;
__device__ __forceinline__ void band_limits(uint32_t tau_bits, uint32_t& lo, uint32_t& hi) {
  const float t = __uint_as_float(tau_bits);
  lo = __float_as_uint(t * (1.0f - kBandRel));
  hi = __float_as_uint(t * (1.0f + kBandRel));
}

// the group's selection state, with every field in scalar registers
__device__ __forceinline__ RadixState load_state(const RadixState* p) {
  RadixState s = *p;
  s.prefix = (uint32_t)uniform((int)s.prefix);
  s.mask = (uint32_t)uniform((int)s.mask);
  s.krem = uniform(s.krem);
  s.keff = uniform(s.keff);
  s.mode = uniform(s.mode);
  return s;
}

__device__ __forceinline__ void seq_range(const SelectArgs& a, int bg, int& c0, int& c1) {
  int b = bg / a.Hkv;
  int L = uniform(a.lengths[b]);
  L = L < 0 ? 0 : (L > a.max_len ? a.max_len : L);
  c0 = a.sink;
  c1 = L - a.recent;
  if (c1 < c0) c1 = c0;
}

// digit of pass d: bits [31:21], [20:10], [9:0]
__device__ __forceinline__ uint32_t radix_digit(uint32_t bits, int pass) {
  return pass == 0 ? (bits >> 21) : (pass == 1 ? ((bits >> 10) & 0x7ffu) : (bits & 0x3ffu));
}
__device__ __forceinline__ uint32_t radix_shift(int pass) { return pass == 0 ? 21u : (pass == 1 ? 10u : 0u); }
__device__ __forceinline__ uint32_t radix_dmask(int pass) { return pass == 2 ? 0x3ffu : 0x7ffu; }

// Each wave of a workgroup counts into its own LDS histogram (pooled scores of
// neighbouring candidates share high bits, so one shared histogram would
// serialise on a few bins); the four are summed and published with one
// global atomic per non-empty bin.
constexpr int kSubHists = kSelThreads / 64;
__device__ __forceinline__ void radix_flush(const SelectArgs& a, int bg, int pass, uint32_t (*lhist)[kRadixBins]) {
  const int nb = pass == 2 ? 1024 : 2048;
  uint32_t* gh = a.hist + ((size_t)pass * a.groups + bg) * kRadixBins;
  __syncthreads();
  for (int i = tid(); i < nb; i += nthreads()) {
    uint32_t v = 0;
#pragma unroll
    for (int w = 0; w < kSubHists; ++w) v += lhist[w][i];
    if (v) atomicAdd(&gh[i], v);
  }
}

__device__ __forceinline__ void clear_hists(uint32_t (*lhist)[kRadixBins]) {
  for (int i = tid(); i < kSubHists * kRadixBins; i += nthreads()) (&lhist[0][0])[i] = 0u;
}

// P = pool(A) on this workgroup's candidates (+ the debug copy) and the first
// radix digit.
__global__ __launch_bounds__(kSelThreads) void pool_hist0(SelectArgs a) {
  __shared__ float la[kCandChunk + 64];
  __shared__ uint32_t lhist[kSubHists][kRadixBins];
  const int bg = bid_y(), split = bid_x();
  const int wave = tid() >> 6;
  int c0, c1;
  seq_range(a, bg, c0, c1);
  const int half = a.pool_kernel / 2;
  const int j0 = c0 + split * kCandChunk, j1 = min(j0 + kCandChunk, c1);
  const RadixState st = load_state(&a.state[bg]);
  float* Pg = a.P + (size_t)bg * a.max_len;

  if (a.pooled_out && split == 0) {
    float* po = a.pooled_out + (size_t)bg * a.max_len;
    for (int j = tid(); j < a.max_len; j += nthreads())
      if (j < c0 || j >= c1) po[j] = __uint_as_float(kQuietNaN);
  }
  if (st.mode == 2) clear_hists(lhist);
  if (j0 < j1) {
    const float* Ag = a.A + (size_t)bg * a.max_len;
    const float padv = a.pool == SNAP_POOL_MAX ? -INFINITY : 0.f;
    for (int i = tid(); i < (j1 - j0) + 2 * half; i += nthreads()) {
      int t = j0 - half + i;
      la[i] = (t >= c0 && t < c1) ? Ag[t] : padv;
    }
    __syncthreads();
    for (int j = j0 + tid(); j < j1; j += nthreads()) {
      const float* w = la + (j - j0);
      float v;
      if (a.pool == SNAP_POOL_MAX) {
        v = w[0];
        for (int t = 1; t < a.pool_kernel; ++t) v = fmaxf(v, w[t]);
      } else {
        v = 0.f;
        for (int t = 0; t < a.pool_kernel; ++t) v += w[t];
        v = v / (float)a.pool_kernel;
      }
      Pg[j] = v;
      if (a.pooled_out) a.pooled_out[(size_t)bg * a.max_len + j] = v;
      if (st.mode == 2) atomicAdd(&lhist[wave][radix_digit(__float_as_uint(v), 0)], 1u);
    }
  }
  if (st.mode == 2) radix_flush(a, bg, 0, lhist);
}

__global__ __launch_bounds__(kSelThreads) void radix_pass(SelectArgs a, int pass) {
  __shared__ uint32_t lhist[kSubHists][kRadixBins];
  const int bg = bid_y(), split = bid_x();
  const int wave = tid() >> 6;
  const RadixState st = load_state(&a.state[bg]);
  if (st.mode != 2) return;
  int c0, c1;
  seq_range(a, bg, c0, c1);
  const int j0 = c0 + split * kCandChunk, j1 = min(j0 + kCandChunk, c1);
  clear_hists(lhist);
  __syncthreads();
  const float* Pg = a.P + (size_t)bg * a.max_len;
  for (int j = j0 + tid(); j < j1; j += nthreads()) {
    uint32_t bits = __float_as_uint(Pg[j]);
    if ((bits & st.mask) == st.prefix) atomicAdd(&lhist[wave][radix_digit(bits, pass)], 1u);
  }
  radix_flush(a, bg, pass, lhist);
}

// One workgroup per group: find the bin that holds the krem-th largest of the
// elements still matching the prefix, counting from the top bin down, and
// narrow the threshold.  Thread t owns the 8 (or 4) bins just below the bins
// of thread t-1, so its exclusive prefix is the count above its bins.
__device__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* lds, uint32_t& total);
__global__ __launch_bounds__(kSelThreads) void radix_scan(SelectArgs a, int pass) {
  __shared__ uint32_t lds[8];
  const int bg = bid_x();
  RadixState st = load_state(&a.state[bg]);
  if (st.mode != 2) return;
  const int nb = pass == 2 ? 1024 : 2048;
  const int per = nb / kSelThreads;  // 8 or 4
  const uint32_t* gh = a.hist + ((size_t)pass * a.groups + bg) * kRadixBins;
  const int top = nb - per * tid();  // this thread's bins: [top - per, top)
  uint32_t hv[8];
  uint32_t tot = 0;
  for (int i = 0; i < per; ++i) {
    hv[i] = gh[top - 1 - i];
    tot += hv[i];
  }
  uint32_t total;
  const uint32_t above = block_exclusive_scan(tot, lds, total);
  const uint32_t krem = (uint32_t)st.krem;
  if (above < krem && above + tot >= krem) {
    uint32_t cum = above;
    for (int i = 0; i < per; ++i) {
      if (cum + hv[i] >= krem) {
        uint32_t bin = (uint32_t)(top - 1 - i);
        st.krem -= (int32_t)cum;
        st.prefix |= bin << radix_shift(pass);
        st.mask |= radix_dmask(pass) << radix_shift(pass);
        a.state[bg] = st;
        break;
      }
      cum += hv[i];
    }
  }
}

// block-wide exclusive scan of one value per thread (lds holds one value per wave)
__device__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* lds, uint32_t& total) {
  const int lane = tid() & 63, wave = tid() >> 6;
  uint32_t x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    uint32_t y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) lds[wave] = x;
  __syncthreads();
  uint32_t base = 0;
  total = 0;
  for (int w2 = 0; w2 < (int)(nthreads() >> 6); ++w2) {
    uint32_t t = lds[w2];
    if (w2 < wave) base += t;
    total += t;
  }
  __syncthreads();
  return base + x - v;
}

constexpr int kPerThread = kCandChunk / kSelThreads;  // 8 consecutive candidates per thread

__global__ __launch_bounds__(kSelThreads) void select_count(SelectArgs a) {
  __shared__ uint32_t lds[8];
  const int bg = bid_y(), split = bid_x();
  const RadixState st = load_state(&a.state[bg]);
  if (st.mode != 2) return;
  int c0, c1;
  seq_range(a, bg, c0, c1);
  const int j0 = c0 + split * kCandChunk, j1 = min(j0 + kCandChunk, c1);
  const float* Pg = a.P + (size_t)bg * a.max_len;
  uint32_t lo, hi;
  band_limits(st.prefix, lo, hi);
  uint32_t gt = 0, eq = 0, above = 0;
  for (int j = j0 + tid(); j < j1; j += nthreads()) {
    uint32_t bits = __float_as_uint(Pg[j]);
    gt += bits > st.prefix;
    eq += bits == st.prefix;
    above += bits > hi;
    if (bits >= lo && bits <= hi) {
      const int m = atomicAdd(&a.band_n[bg], 1);
      if (m < kBandCap) a.band_idx[(size_t)bg * kBandCap + m] = j;
    }
  }
  uint32_t tg, te, ta;
  block_exclusive_scan(gt, lds, tg);
  block_exclusive_scan(eq, lds, te);
  block_exclusive_scan(above, lds, ta);
  if (tid() == 0) {
    a.counts[(size_t)bg * a.n_splits + split] = make_uint2(tg, te);
    a.band_above[(size_t)bg * a.n_splits + split] = ta;
  }
}

// ============================================================ fp64 re-score of the band
// Every candidate in the band gets its pooled score again in fp64 (Eq. 1-3
// with exact products of the bf16 / fp32 inputs, fp64 exponentials and the
// rows' fp64 normalisers), so the selection near the threshold does not rest
// on the fp32 logits of the score passes.  band_rescore forms the summed
// attention A of every key in the members' pooling windows, once per key:
// with the members sorted by token, member m owns the keys of its window
// past the previous member's window.  band_decide then pools, ranks and
// decides.
struct BandArgs {
  const void* q;          // [n_seq][Hq][w][D]
  const void* k;          // [n_seq][Hkv][max_len][D]
  const int32_t* lengths;
  const double2* rowz;    // [groups][rows_pad]
  const RadixState* state;
  const int32_t* band_n;
  const int32_t* band_idx;
  double* A64;            // [groups][max_len] fp64 A of the window keys
  double* band_p;         // [groups][kBandCap] fp64 pooled scores of the members
  float* pooled_out;      // optional debug copy: the members' re-scored values
  float* P;               // [groups][max_len]
  uint2* counts;          // [groups][n_splits]
  const uint32_t* band_above;
  RadixState* state_w;
  int Hq, Hkv, G, w, D, max_len, sink, recent, pool_kernel, pool, rows, rows_pad, n_splits, in_f32;
  int band_wgs;           // workgroups per group of band_rescore (work items strided over them)
  int rows_per_pass;      // score rows per band_rescore pass (kBandThreads / query-dim slices)
  double scale2;          // sm_scale * log2(e) in fp64
};

// Members ranked by token index (the members are distinct): rank[i] = how
// many members precede member i.  One pass over the list per member, no
// barriers; nb <= kBandCap.
__device__ __forceinline__ int token_rank(const int32_t* s, int nb, int i) {
  const int32_t x = s[i];
  int r = 0;
  for (int u = 0; u < nb; ++u) r += s[u] < x;
  return r;
}

// The keys whose fp64 A the band needs, in token order: with the members
// sorted by token, member m owns the keys of its pooling window (within the
// candidates) that lie past the previous member's window.  Fills first[m] =
// index of member m's first key in that order (first[nb] = the key count) and
// tok[m] = the sorted members; returns the key count.  Every thread calls it.
__device__ int band_keys(const int32_t* members, int nb, int half, int c0, int c1, int32_t* tok, int32_t* first,
                         uint32_t* scan_lds) {
  for (int i = tid(); i < nb; i += nthreads()) tok[token_rank(members, nb, i)] = members[i];
  __syncthreads();
  // owned key counts, then an exclusive scan over the (<= kBandCap) members
  uint32_t total = 0;
  for (int base = 0; base < nb; base += nthreads()) {
    const int m = base + tid();
    uint32_t cnt = 0;
    if (m < nb) {
      const int j = tok[m];
      int t0 = max(j - half, c0);
      if (m > 0) t0 = max(t0, tok[m - 1] + half + 1);
      const int t1 = min(j + half, c1 - 1);
      cnt = t1 >= t0 ? (uint32_t)(t1 - t0 + 1) : 0u;
    }
    uint32_t part;
    const uint32_t ex = block_exclusive_scan(cnt, scan_lds, part);
    if (m < nb) first[m] = (int)(total + ex);
    total += part;
  }
  if (tid() == 0) first[nb] = (int)total;
  __syncthreads();
  return (int)total;
}

// Token of key x in the band's key order (first[] from band_keys).
__device__ __forceinline__ int band_key_token(const int32_t* tok, const int32_t* first, int nb, int half, int c0,
                                              int x) {
  int lo = 0, hi = nb - 1;  // the member m with first[m] <= x < first[m+1]
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (first[mid] <= x) lo = mid; else hi = mid - 1;
  }
  const int j = tok[lo];
  int t0 = max(j - half, c0);
  if (lo > 0) t0 = max(t0, tok[lo - 1] + half + 1);
  return t0 + (x - first[lo]);
}

constexpr int kBandWGs = 16;       // band_rescore workgroups per group (work items strided over them)
constexpr int kBandKeys = 4;       // keys per block (staged in LDS together)
constexpr int kBandThreads = 512;  // rows x slices of the query dims
constexpr int kBandKeyCap = 1024;  // band keys per group; more keeps the fp32 selection
constexpr int kBandMaxPass = 4;    // row passes of a key block (rows_pad / rows per pass)
// Workgroup of kBandThreads threads: thread = (score row, slice of SLICES of the
// query dims), rows taken kBandThreads / SLICES at a time.  Each block of
// kBandKeys keys is staged in LDS with one load round trip; the thread's
// query slice is loaded once per block and row pass.
template <typename In, int D, int SLICES>
__device__ void band_rescore_body(const BandArgs& a, int bg, int b, int g, int nkeys, const int32_t* tok,
                                  const int32_t* first, int nb, int half, int c0, int L, unsigned char* kl,
                                  double (*red)[kBandKeys]) {
  constexpr int kEl = 16 / (int)sizeof(In);         // elements per 16-byte chunk
  constexpr int kRowChunks = D / kEl;
  constexpr int CH = kRowChunks / SLICES;           // chunks per slice
  constexpr int RPP = kBandThreads / SLICES;        // rows per pass
  const int sl = tid() % SLICES;
  const int we = min(a.w, L);
  const In* qg = (const In*)a.q + ((size_t)b * a.Hq + (size_t)g * a.G) * a.w * D;
  const size_t krow0 = ((size_t)b * a.Hkv + g) * (size_t)a.max_len;
  const int lane = tid() & 63, wave = tid() >> 6;
  const int npass = (a.rows_pad + RPP - 1) / RPP;
  const int nblk = (nkeys + kBandKeys - 1) / kBandKeys;
  // work items (key block, row pass), strided over the group's workgroups
  for (int item = bid_x(); item < nblk * npass; item += a.band_wgs) {
    const int x0 = (item / npass) * kBandKeys, r0 = (item % npass) * RPP;
    const int nk = min(kBandKeys, nkeys - x0);
    // stage the block's key rows (chunk c of key e at kl + (e * kRowChunks + c) * 16)
    for (int i = tid(); i < nk * kRowChunks; i += nthreads()) {
      const int e = i / kRowChunks, c = i % kRowChunks;
      const int t = band_key_token(tok, first, nb, half, c0, x0 + e);
      if (debug_check(t >= c0 && t < L - a.recent, kDbgBand))
        *((u32x4*)kl + i) = *((const u32x4*)((const In*)a.k + (krow0 + t) * D) + c);
    }
    int kt[kBandKeys];
#pragma unroll
    for (int e = 0; e < kBandKeys; ++e) kt[e] = e < nk ? band_key_token(tok, first, nb, half, c0, x0 + e) : 0;
    // this thread's row and its query slice
    const int rho = r0 + tid() / SLICES;
    const int ii = rho % a.w;
    const bool rval = rho < a.rows && ii >= a.w - we;
    const int rpos = L - a.w + ii;
    const double2 nz = rval ? a.rowz[(size_t)bg * a.rows_pad + rho] : make_double2(0.0, 0.0);
    const bool live = rval && nz.y > 0.0;
    u32x4 qv[CH];
#pragma unroll
    for (int c = 0; c < CH; ++c)
      qv[c] = live ? *((const u32x4*)(qg + (size_t)rho * D) + sl * CH + c) : u32x4{0u, 0u, 0u, 0u};
    __syncthreads();
#pragma unroll
    for (int e = 0; e < kBandKeys; ++e) {
      double s = 0.0;
      if (e < nk) {
#pragma unroll
        for (int c = 0; c < CH; ++c) {
          const u32x4 kv = *((const u32x4*)kl + e * kRowChunks + sl * CH + c);
          if constexpr (sizeof(In) == 2) {
            // a bf16 x bf16 product is exact in fp32; the sums run in fp64
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              s += (double)(bf16_bits_to_f32(qv[c][i] & 0xffffu) * bf16_bits_to_f32(kv[i] & 0xffffu));
              s += (double)(bf16_bits_to_f32(qv[c][i] >> 16) * bf16_bits_to_f32(kv[i] >> 16));
            }
          } else {
#pragma unroll
            for (int i = 0; i < 4; ++i) s = fma((double)__uint_as_float(qv[c][i]), (double)__uint_as_float(kv[i]), s);
          }
        }
      }
      // the row's dot product: sum of its slices (adjacent lanes)
#pragma unroll
      for (int o = 1; o < SLICES; o <<= 1) s += __shfl_xor(s, o);
      double wv = 0.0;
      if (sl == 0 && live && e < nk && kt[e] <= rpos) wv = exp2(s * a.scale2 - nz.x) / nz.y;
      // summed over this pass's rows (fixed order)
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) wv += __shfl_xor(wv, o);
      if (lane == 0) red[wave][e] = wv;
    }
    __syncthreads();
    if (tid() < nk) {
      double s = 0.0;
      for (int w2 = 0; w2 < kBandThreads / 64; ++w2) s += red[w2][tid()];
      a.A64[((size_t)bg * kBandKeyCap + x0 + tid()) * kBandMaxPass + item % npass] = s;
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(kBandThreads) void band_rescore(BandArgs a) {
  __shared__ int32_t mem[kBandCap];
  __shared__ int32_t tok[kBandCap];
  __shared__ int32_t first[kBandCap + 1];
  __shared__ uint32_t scan_lds[kBandThreads / 64];
  __shared__ double red[kBandThreads / 64][kBandKeys];
  __shared__ __align__(16) unsigned char kl[kBandKeys * 576 * 2];
  const int bg = bid_y(), b = bg / a.Hkv, g = bg % a.Hkv;
  const RadixState st = load_state(&a.state[bg]);
  if (st.mode != 2) return;
  const int nb = uniform(a.band_n[bg]);
  if (nb > kBandCap) return;  // too many: the fp32 selection stands
  // at most pool_kernel keys per member, so at most this many work items:
  // workgroups past them have nothing to do
  if (bid_x() >= (nb * a.pool_kernel + kBandKeys - 1) / kBandKeys * kBandMaxPass) return;
  int L = uniform(a.lengths[b]);
  L = L < 0 ? 0 : (L > a.max_len ? a.max_len : L);
  const int c0 = a.sink, c1 = L - a.recent, half = a.pool_kernel / 2;
  for (int i = tid(); i < nb; i += nthreads()) mem[i] = a.band_idx[(size_t)bg * kBandCap + i];
  __syncthreads();
  const int nkeys = band_keys(mem, nb, half, c0, c1, tok, first, scan_lds);
  if (nkeys > kBandKeyCap) return;
  // threads per score row (rows_pad <= 256, or 128 for fp32 inputs)
  if (a.in_f32) {
    if (a.D == 64) band_rescore_body<float, 64, 8>(a, bg, b, g, nkeys, tok, first, nb, half, c0, L, kl, red);
    else band_rescore_body<float, 128, 8>(a, bg, b, g, nkeys, tok, first, nb, half, c0, L, kl, red);
  } else {
    if (a.D == 64) band_rescore_body<uint16_t, 64, 4>(a, bg, b, g, nkeys, tok, first, nb, half, c0, L, kl, red);
    else if (a.D == 128) band_rescore_body<uint16_t, 128, 4>(a, bg, b, g, nkeys, tok, first, nb, half, c0, L, kl, red);
    else band_rescore_body<uint16_t, 576, 8>(a, bg, b, g, nkeys, tok, first, nb, half, c0, L, kl, red);
  }
}

// One workgroup per group: pool each member from the fp64 A of its window
// (Eq. 2), rank the members by (fp64 pooled score descending, token index
// ascending), keep the first K_eff - (candidates above the band), and
// rewrite the members' P so that the ordered compaction keeps exactly the
// candidates above the band and the kept members: P > hi for kept ones, 0
// for the others, threshold hi, no ties.
__global__ __launch_bounds__(kSelThreads) void band_decide(BandArgs a) {
  __shared__ double sp[kBandCap];
  __shared__ int32_t sj[kBandCap];
  __shared__ int32_t tok[kBandCap];
  __shared__ int32_t first[kBandCap + 1];
  __shared__ uint32_t lds[8];
  const int bg = bid_x();
  RadixState st = load_state(&a.state[bg]);
  if (st.mode != 2) return;
  const int nb = uniform(a.band_n[bg]);
  if (nb > kBandCap) return;
  const int b = bg / a.Hkv;
  int L = uniform(a.lengths[b]);
  L = L < 0 ? 0 : (L > a.max_len ? a.max_len : L);
  const int c0 = a.sink, c1 = L - a.recent, half = a.pool_kernel / 2;
  for (int i = tid(); i < nb; i += nthreads()) sj[i] = a.band_idx[(size_t)bg * kBandCap + i];
  __syncthreads();
  if (band_keys(sj, nb, half, c0, c1, tok, first, lds) > kBandKeyCap) return;  // as band_rescore
  uint32_t lo, hi;
  band_limits(st.prefix, lo, hi);
  // candidates above the band (all kept)
  uint32_t above = 0;
  for (int s = tid(); s < a.n_splits; s += nthreads()) above += a.band_above[(size_t)bg * a.n_splits + s];
  uint32_t n_above;
  block_exclusive_scan(above, lds, n_above);
  const int need = st.keff - (int)n_above;  // in [1, nb] (tau itself is a member)
  if (need < 0 || need > nb) return;         // not for finite scores; the fp32 selection stands
  const double* Ag = a.A64 + (size_t)bg * kBandKeyCap * kBandMaxPass;
  const int npass = (a.rows_pad + a.rows_per_pass - 1) / a.rows_per_pass;
  for (int i = tid(); i < nb; i += nthreads()) {
    const int j = sj[i];
    const int t0 = max(j - half, c0), t1 = min(j + half, c1 - 1);
    double pooled = a.pool == SNAP_POOL_MAX ? -1.0 : 0.0;
    for (int t = t0; t <= t1; ++t) {
      // key index of t: the first member (by token) whose window holds t
      // owns it (see band_keys)
      int lo = 0, hi2 = nb - 1;
      while (lo < hi2) {
        const int mid = (lo + hi2) >> 1;
        if (tok[mid] >= t - half) hi2 = mid; else lo = mid + 1;
      }
      int k0 = max(tok[lo] - half, c0);
      if (lo > 0) k0 = max(k0, tok[lo - 1] + half + 1);
      const int x = first[lo] + (t - k0);
      double At = 0.0;
      for (int pp = 0; pp < npass; ++pp) At += Ag[(size_t)x * kBandMaxPass + pp];
      if (a.pool == SNAP_POOL_MAX)
        pooled = At > pooled ? At : pooled;
      else
        pooled += At;
    }
    if (a.pool != SNAP_POOL_MAX) pooled /= (double)a.pool_kernel;
    sp[i] = pooled;
    a.band_p[(size_t)bg * kBandCap + i] = pooled;
    if (a.pooled_out) a.pooled_out[(size_t)bg * a.max_len + j] = (float)pooled;
  }
  __syncthreads();
  // rank by (score desc, token asc): kept when fewer than `need` come first
  float* Pg = a.P + (size_t)bg * a.max_len;
  for (int i = tid(); i < nb; i += nthreads()) {
    const double pi = sp[i];
    const int ji = sj[i];
    int r = 0;
    for (int u = 0; u < nb; ++u) r += sp[u] > pi || (sp[u] == pi && sj[u] < ji);
    tok[i] = r < need;
  }
  __syncthreads();
  // per-split counts of what the compaction keeps: the candidates above the
  // band and the kept members
  for (int s = tid(); s < a.n_splits; s += nthreads()) {
    uint32_t n = a.band_above[(size_t)bg * a.n_splits + s];
    for (int i = 0; i < nb; ++i) n += tok[i] && (sj[i] - c0) / kCandChunk == s;
    a.counts[(size_t)bg * a.n_splits + s] = make_uint2(n, 0u);
  }
  for (int i = tid(); i < nb; i += nthreads()) Pg[sj[i]] = __uint_as_float(tok[i] ? hi + 1u : 0u);
  if (tid() == 0) {
    st.prefix = hi;
    st.krem = 0;
    a.state_w[bg] = st;
  }
}

// Ordered compaction: a candidate is kept when P > t, or P == t and it is among
// the krem lowest-index candidates equal to t.  Output is in token order.
__global__ __launch_bounds__(kSelThreads) void select_write(SelectArgs a) {
  __shared__ uint32_t lds[8];
  const int bg = bid_y(), split = bid_x();
  const RadixState st = load_state(&a.state[bg]);
  if (st.mode == 0) return;
  int c0, c1;
  seq_range(a, bg, c0, c1);
  const int j0 = c0 + split * kCandChunk, j1 = min(j0 + kCandChunk, c1);
  int32_t* sg = a.sel + (size_t)bg * a.topk;
  if (st.mode == 1) {
    for (int j = j0 + tid(); j < j1; j += nthreads()) sg[j - c0] = j;
    return;
  }
  uint32_t gt_before = 0, eq_before = 0;
  for (int t = 0; t < split; ++t) {
    uint2 c = a.counts[(size_t)bg * a.n_splits + t];
    gt_before += c.x;
    eq_before += c.y;
  }
  const uint32_t krem = (uint32_t)st.krem;
  const uint32_t ties_here = krem > eq_before ? krem - eq_before : 0u;
  const uint32_t out_base = gt_before + (eq_before < krem ? eq_before : krem);
  const float* Pg = a.P + (size_t)bg * a.max_len;
  const int jt = j0 + tid() * kPerThread;
  uint32_t bits[kPerThread];
  uint32_t neq = 0;
#pragma unroll
  for (int i = 0; i < kPerThread; ++i) {
    int j = jt + i;
    bits[i] = j < j1 ? __float_as_uint(Pg[j]) : 0u;
    neq += (j < j1 && bits[i] == st.prefix);
  }
  uint32_t tot;
  uint32_t eq_rank = block_exclusive_scan(neq, lds, tot);
  bool keep[kPerThread];
  uint32_t nkeep = 0;
#pragma unroll
  for (int i = 0; i < kPerThread; ++i) {
    int j = jt + i;
    bool in = j < j1;
    bool k = false;
    if (in && bits[i] > st.prefix) k = true;
    if (in && bits[i] == st.prefix) {
      k = eq_rank < ties_here;
      ++eq_rank;
    }
    keep[i] = k;
    nkeep += k;
  }
  uint32_t pos = out_base + block_exclusive_scan(nkeep, lds, tot);
  const uint32_t keff = (uint32_t)st.keff;
#pragma unroll
  for (int i = 0; i < kPerThread; ++i)
    if (keep[i]) {
      if (debug_check(pos < keff, kDbgSelWrite) && pos < keff) sg[pos] = jt + i;  // never past the group's K slots
      ++pos;
    }
}

// ============================================================ assemble
struct AssembleArgs {
  const void* k;       // [n_seq][Hkv][max_len][dk]
  const void* v;       // or NULL
  void* ck;            // [n_slots][Hkv][B][dk]
  void* cv;
  float* k_scale;      // [n_slots][Hkv], fp8 only (written in SNAP_FP8_SCALES_AMAX mode)
  float* v_scale;
  const int32_t* slot_ids;
  const int32_t* lengths;
  const int32_t* sel;  // [groups][topk]
  const RadixState* state;
  int32_t* sel_out;    // optional [groups][topk]
  int32_t* pos;
  int32_t* n_topk;
  float2* amax;        // [groups][n_rowblocks] (K, V) amax of the kept rows, or NULL
  int Hkv, max_len, sink, recent, topk, dk, dv, n_slots, rows_per_block, n_rowblocks;
};

constexpr int kAsmRows = 64;  // cache rows per assemble workgroup

// First ring token l0 = max(L - r, s) and ring_base = (l0 - s) mod r, the
// ring row of token l0 counted from s (one division per thread, not per row).
struct RingMap {
  int l0, base;
};
__device__ __forceinline__ RingMap ring_map(int L, int s, int r) {
  const int l0 = L - r > s ? L - r : s;
  return RingMap{l0, (l0 - s) % r};
}

// Source token of cache row `row` (or -1 for a zero padding row).
__device__ __forceinline__ int row_source(int row, int L, int s, int r, int keff, const int32_t* sel,
                                          RingMap rm) {
  if (row < s) return row < L ? row : -1;
  if (row < s + r) {
    // token l0 + ((row - s) - base) mod r, with both terms in [0, r)
    int off = (row - s) - rm.base;
    if (off < 0) off += r;
    int t = rm.l0 + off;
    return t < L ? t : -1;
  }
  int m = row - s - r;
  if (m >= keff) return -1;
  const int t = sel[m];
  return debug_check(t >= s && t < L - r, kDbgAsmSource) ? t : -1;
}

// x / scale rounded once to fp32, as an IEEE division gives it, from a
// correctly rounded reciprocal inv = 1 / scale and one fused correction:
// q0 = x * inv, r = x - q0 * scale (exact by fma), q = q0 + r * inv (Markstein's
// theorem: correctly rounded when neither r nor the quotient leaves the
// normal range).  Where q0 is 0 or not finite it is kept: the E4M3 code of a
// zero, of a quotient too small for a non-zero code, or of a saturated one
// does not depend on the correction.  Checked on the host against the
// division for every finite bf16 x over 353 scales (amax / 448 of 256 bf16
// maxima, 64 random magnitudes, powers of two and their neighbours):
// identical E4M3 codes.
__device__ __forceinline__ float div_by_scale(float x, float scale, float inv) {
  const float q0 = x * inv;
  const float r = __builtin_fmaf(-q0, scale, x);
  const float q = __builtin_fmaf(r, inv, q0);
  return (q0 == 0.f || !__builtin_isfinite(q0)) ? q0 : q;
}

// 8 elements of an input row in raw form: 16 bytes of bf16 or 32 of fp32
// (zeros for a NULL source, a padding row).  The gather reads each prompt row
// and writes each cache row once: both carry the non-temporal (streaming)
// hint (measured 1-2% off the compress call).
template <typename In>
struct Raw8In {
  u32x4 w[sizeof(In) / 2];
};
template <typename In>
__device__ __forceinline__ Raw8In<In> load8(const In* src) {
  Raw8In<In> x;
#pragma unroll
  for (int i = 0; i < (int)(sizeof(In) / 2); ++i)
    x.w[i] = src ? __builtin_nontemporal_load((const u32x4*)src + i) : u32x4{0u, 0u, 0u, 0u};
  return x;
}
// ... stored into the cache, quantised to E4M3 codes of x / scale when the
// cache is fp8 (the correctly rounded quotient, then the conversion
// instruction: e4m3x4_hw).
template <typename In, typename Out>
__device__ __forceinline__ void store8(const Raw8In<In>& x, Out* dst, float scale, float inv) {
  if constexpr (sizeof(Out) == 1) {
    float f[8];
    if constexpr (sizeof(In) == 2) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        f[2 * i] = bf16_bits_to_f32(x.w[0][i] & 0xffffu);
        f[2 * i + 1] = bf16_bits_to_f32(x.w[0][i] >> 16);
      }
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) f[i] = __uint_as_float(x.w[i >> 2][i & 3]);
    }
    float qv[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) qv[i] = div_by_scale(f[i], scale, inv);
    u32x2 o;
    o[0] = e4m3x4_hw(qv[0], qv[1], qv[2], qv[3]);
    o[1] = e4m3x4_hw(qv[4], qv[5], qv[6], qv[7]);
    __builtin_nontemporal_store(o, (u32x2*)dst);
  } else {
#pragma unroll
    for (int i = 0; i < (int)(sizeof(In) / 2); ++i) __builtin_nontemporal_store(x.w[i], (u32x4*)dst + i);
  }
}

// Largest magnitude of one workgroup's values (LDS across the waves); every
// thread gets it.
__device__ __forceinline__ uint32_t block_max_u32(uint32_t v, uint32_t* lds) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = max(v, (uint32_t)__shfl_xor((int)v, o));
  __syncthreads();
  if ((tid() & 63) == 0) lds[tid() >> 6] = v;
  __syncthreads();
  v = 0;
  for (int w = 0; w < (int)(nthreads() >> 6); ++w) v = max(v, lds[w]);
  return v;
}

// fp8 scales from the data (SNAP_FP8_SCALES_AMAX): per (group, block of
// rows_per_block cache rows) the largest |K| and |V| among the rows the block
// keeps; padding rows add nothing.  bf16 magnitudes order like their bit
// patterns, so the maxima are taken on the 15 low bits.
__global__ __launch_bounds__(256) void fp8_amax(AssembleArgs a) {
  __shared__ uint32_t lds[4];
  const int bg = bid_y(), b = bg / a.Hkv, g = bg % a.Hkv;
  const int slot = uniform(a.slot_ids[b]);
  if (slot < 0 || slot >= a.n_slots) return;
  const int s = a.sink, r = a.recent, B = s + r + a.topk;
  int L = uniform(a.lengths[b]);
  L = L < 0 ? 0 : (L > a.max_len ? a.max_len : L);
  const int keff = a.topk == 0 ? 0 : uniform(a.state[bg].keff);
  const int32_t* sg = a.sel + (size_t)bg * a.topk;
  const int row0 = bid_x() * a.rows_per_block;
  const int row1 = min(row0 + a.rows_per_block, B);
  const size_t in_row0 = ((size_t)b * a.Hkv + g) * (size_t)a.max_len;
  const int kp = a.dk / 8, vp = a.v ? a.dv / 8 : 0, per_row = kp + vp;
  const int items = (row1 - row0) * per_row;
  const RingMap rm = ring_map(L, s, r);
  uint32_t mk = 0, mv = 0;
  for (int it = tid(); it < items; it += nthreads()) {
    const int row = row0 + it / per_row, piece = it % per_row;
    const int t = row_source(row, L, s, r, keff, sg, rm);
    if (t < 0) continue;
    const u32x4 x = piece < kp ? *((const u32x4*)((const uint16_t*)a.k + (in_row0 + t) * a.dk) + piece)
                               : *((const u32x4*)((const uint16_t*)a.v + (in_row0 + t) * a.dv) + (piece - kp));
    uint32_t m = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) m = max(m, max(x[i] & 0x7fffu, (x[i] >> 16) & 0x7fffu));
    if (piece < kp)
      mk = max(mk, m);
    else
      mv = max(mv, m);
  }
  mk = block_max_u32(mk, lds);
  mv = block_max_u32(mv, lds);
  if (tid() == 0)
    a.amax[(size_t)bg * a.n_rowblocks + bid_x()] = make_float2(bf16_bits_to_f32(mk), bf16_bits_to_f32(mv));
}

// Each workgroup rewrites rows_per_block cache rows of one (sequence, KV
// head); threads walk (row, 8-element piece) pairs so every lane copies, kAsmU
// pairs at a time: their selected-index reads, then their row reads, are all
// issued before the first store (two memory round trips per kAsmU pieces).
constexpr int kAsmU = 8;
template <typename In, typename Out>
__global__ __launch_bounds__(256) void assemble(AssembleArgs a) {
  const int bg = bid_y(), b = bg / a.Hkv, g = bg % a.Hkv;
  const int slot = uniform(a.slot_ids[b]);
  const int s = a.sink, r = a.recent, B = s + r + a.topk;
  int L = uniform(a.lengths[b]);
  L = L < 0 ? 0 : (L > a.max_len ? a.max_len : L);
  const int keff = a.topk == 0 ? 0 : uniform(a.state[bg].keff);  // no selection ran when topk = 0
  const int32_t* sg = a.sel + (size_t)bg * a.topk;
  const int row0 = bid_x() * a.rows_per_block;
  const int row1 = min(row0 + a.rows_per_block, B);

  if (a.sel_out) {
    for (int m = row0 + tid(); m < row1; m += nthreads()) {
      int mm = m - s - r;
      if (mm >= 0) a.sel_out[(size_t)bg * a.topk + mm] = mm < keff ? sg[mm] : -1;
    }
  }
  if (slot < 0 || slot >= a.n_slots) return;
  if (bid_x() == 0 && g == 0 && tid() == 0) {
    a.pos[slot] = L;
    a.n_topk[slot] = keff;
  }
  const size_t in_row0 = ((size_t)b * a.Hkv + g) * (size_t)a.max_len;
  const size_t out_row0 = ((size_t)slot * a.Hkv + g) * (size_t)B;
  float ks = 1.f, vs = 1.f;
  if constexpr (sizeof(Out) == 1) {
    if (a.amax) {
      // scales from the group's amax over every row block: amax / 448, or 1
      // when every kept value is zero; block 0 records them for decoding
      __shared__ uint32_t lds[4];
      uint32_t mk = 0, mv = 0;
      for (int i = tid(); i < a.n_rowblocks; i += nthreads()) {
        const float2 m = a.amax[(size_t)bg * a.n_rowblocks + i];
        mk = max(mk, __float_as_uint(m.x));
        mv = max(mv, __float_as_uint(m.y));
      }
      const float ak = __uint_as_float(block_max_u32(mk, lds));
      const float av = __uint_as_float(block_max_u32(mv, lds));
      ks = ak > 0.f ? ak / 448.f : 1.f;
      vs = av > 0.f ? av / 448.f : 1.f;
      if (bid_x() == 0 && tid() == 0) {
        a.k_scale[(size_t)slot * a.Hkv + g] = ks;
        if (a.v) a.v_scale[(size_t)slot * a.Hkv + g] = vs;
      }
    } else {
      ks = a.k_scale[(size_t)slot * a.Hkv + g];
      if (a.v) vs = a.v_scale[(size_t)slot * a.Hkv + g];
    }
  }
  const float kinv = 1.0f / ks, vinv = 1.0f / vs;
  const RingMap rm = ring_map(L, s, r);
  const int kp = a.dk / 8, vp = a.v ? a.dv / 8 : 0, per_row = kp + vp;
  const int items = (row1 - row0) * per_row;
  // item it = row * per_row + piece; this thread's items advance by
  // nthreads(), i.e. by (step_r rows, step_p pieces) with a carry, so the
  // division runs once per thread
  const int step_r = nthreads() / per_row, step_p = nthreads() % per_row;
  int cur_r = tid() / per_row, cur_p = tid() % per_row;
  for (int it0 = tid(); it0 < items; it0 += kAsmU * nthreads()) {
    int row_u[kAsmU], piece_u[kAsmU], src_t[kAsmU];
#pragma unroll
    for (int u = 0; u < kAsmU; ++u) {
      const int it = it0 + u * nthreads();
      row_u[u] = row0 + cur_r;
      piece_u[u] = cur_p;
      cur_r += step_r;
      cur_p += step_p;
      if (cur_p >= per_row) {
        cur_p -= per_row;
        ++cur_r;
      }
      src_t[u] = it < items ? row_source(row_u[u], L, s, r, keff, sg, rm) : -1;
    }
    Raw8In<In> x[kAsmU];
#pragma unroll
    for (int u = 0; u < kAsmU; ++u) {
      const int it = it0 + u * nthreads();
      const int piece = piece_u[u], t = src_t[u];
      const In* src = nullptr;
      if (it < items && t >= 0)
        src = piece < kp ? (const In*)a.k + (in_row0 + t) * a.dk + 8 * piece
                         : (const In*)a.v + (in_row0 + t) * a.dv + 8 * (piece - kp);
      x[u] = load8<In>(src);
    }
#pragma unroll
    for (int u = 0; u < kAsmU; ++u) {
      const int it = it0 + u * nthreads();
      if (it >= items) break;
      const int row = row_u[u], piece = piece_u[u];
      if (piece < kp)
        store8<In, Out>(x[u], (Out*)a.ck + (out_row0 + row) * a.dk + 8 * piece, ks, kinv);
      else
        store8<In, Out>(x[u], (Out*)a.cv + (out_row0 + row) * a.dv + 8 * (piece - kp), vs, vinv);
    }
  }
}

// ============================================================ host side
static inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// scale * log2(e) as hi + lo: hi the fp32 value rounded toward zero, lo the
// rest, strictly positive (a tiny positive value when hi is exact, where it
// changes no finite product): a masked -inf product times lo stays -inf.
void split_scale2(float scale, float& hi, float& lo) {
  const double x = (double)scale * 1.4426950408889634074;
  float h = (float)x;
  if ((double)h > x) h = nextafterf(h, 0.f);
  const float l = (float)(x - (double)h);
  hi = h;
  lo = l > 0.f ? l : 1e-30f;
}

SNAP_DEBUG_READER(debug_flags_compress)

Geometry compress_geometry(const snap_params& p, int n_seq, int max_len) {
  Geometry g{};
  int G = p.n_q_heads / p.n_kv_heads;
  g.rows = G * p.obs_window;
  g.rows_pad = (g.rows + 31) / 32 * 32;
  int groups = n_seq * p.n_kv_heads;
  // Key chunks: enough workgroups to cover the 256 CUs several times (about
  // 4096), but each chunk at least 4 * rows_pad keys (16 * rows_pad for the
  // wide latent groups, whose query block is 295 KB), so that its keys
  // outweigh the query fragments every workgroup loads first (measured: the
  // 256-row latent shape is fastest at 4096-key chunks; a single 128-row GQA
  // prompt at 512-key chunks, 28% faster score passes than at 2048, and its
  // compress call 4-8% faster than at 256).
  long target = 4096;
  long per_group = (target + groups - 1) / (groups > 0 ? groups : 1);
  long kc = (max_len + per_group - 1) / (per_group > 0 ? per_group : 1);
  const long kc_min = (g.rows_pad > 128 ? 16L : 4L) * g.rows_pad;
  if (kc < kc_min) kc = kc_min;
  kc = (kc + kKeyTile - 1) / kKeyTile * kKeyTile;
  if (kc > 16384) kc = 16384;
  g.key_chunk = (int)kc;
  g.n_kchunks = (int)((max_len + kc - 1) / kc);
  if (g.n_kchunks < 1) g.n_kchunks = 1;
  int ncand = max_len - p.sink - p.recent;
  if (ncand < 1) ncand = 1;
  g.n_splits = (ncand + kCandChunk - 1) / kCandChunk;
  size_t off = 0;
  g.off_stats = off;
  off = align256(off + (size_t)groups * g.n_kchunks * g.rows_pad * sizeof(float2));
  g.off_rowref = off;
  off = align256(off + (size_t)groups * g.rows_pad * sizeof(float2));
  g.off_A = off;
  off = align256(off + (size_t)groups * max_len * sizeof(float));
  g.off_P = off;
  off = align256(off + (size_t)groups * max_len * sizeof(float));
  g.off_hist = off;
  off = align256(off + (size_t)3 * groups * kRadixBins * sizeof(uint32_t));
  g.off_state = off;
  off = align256(off + (size_t)groups * sizeof(RadixState));
  g.off_counts = off;
  off = align256(off + (size_t)groups * g.n_splits * sizeof(uint2));
  g.off_sel = off;
  off = align256(off + (size_t)groups * (p.topk > 0 ? p.topk : 1) * sizeof(int32_t));
  // per (group, assemble row block): amax of the kept K and V rows (fp8 scales)
  g.n_rowblocks = (p.sink + p.recent + p.topk + kAsmRows - 1) / kAsmRows;
  g.off_amax = off;
  off = align256(off + (size_t)groups * g.n_rowblocks * sizeof(float2));
  g.off_rowz = off;
  off = align256(off + (size_t)groups * g.rows_pad * sizeof(double2));
  g.off_band_n = off;
  off = align256(off + (size_t)groups * sizeof(int32_t));
  g.off_band_idx = off;
  off = align256(off + (size_t)groups * kBandCap * sizeof(int32_t));
  g.off_band_p = off;
  off = align256(off + (size_t)groups * kBandCap * sizeof(double));
  g.off_band_above = off;
  off = align256(off + (size_t)groups * g.n_splits * sizeof(uint32_t));
  g.off_A64 = off;
  off = align256(off + (size_t)groups * kBandKeyCap * kBandMaxPass * sizeof(double));
  g.compress_bytes = off;
  return g;
}

template <typename In, int KS, int NW, int TK, int STAGES>
static hipError_t launch_score_nw(const ScoreArgs& sa, bool colsum, int groups, int n_kchunks, hipStream_t st) {
  dim3 grid(n_kchunks, groups), block(64 * NW);
  if (colsum)
    hipLaunchKernelGGL((score_pass<In, KS, NW, true, TK, STAGES>), grid, block, 0, st, sa);
  else
    hipLaunchKernelGGL((score_pass<In, KS, NW, false, TK, STAGES>), grid, block, 0, st, sa);
  return hipGetLastError();
}

// Waves per workgroup: 4 while the score rows fit in 128, else 8.  Tiles and
// stages per shape, as measured: the 576-wide latent rows take 32-key tiles in
// 4 stages (147 KB, one workgroup per CU: three tiles in flight while one is
// scored; 8% faster than two 64-key stages); 64/128-wide bf16 rows keep two
// 64-key stages (three workgroups per CU; three or four stages measured
// slower); fp32 rows 3 or 2 stages next to their fp32 query block.
template <typename In>
static hipError_t launch_score(const ScoreArgs& sa, int dk, bool colsum, int groups, int n_kchunks, hipStream_t st) {
  const bool wide = sa.rows_pad > 128;
  if constexpr (sizeof(In) == 2) {
    if (dk == 64) return wide ? launch_score_nw<In, 2, 8, 64, 2>(sa, colsum, groups, n_kchunks, st)
                              : launch_score_nw<In, 2, 4, 64, 2>(sa, colsum, groups, n_kchunks, st);
    if (dk == 128) return wide ? launch_score_nw<In, 4, 8, 64, 2>(sa, colsum, groups, n_kchunks, st)
                               : launch_score_nw<In, 4, 4, 64, 2>(sa, colsum, groups, n_kchunks, st);
    if (dk == 576) return wide ? launch_score_nw<In, 18, 8, 32, 4>(sa, colsum, groups, n_kchunks, st)
                               : launch_score_nw<In, 18, 4, 32, 4>(sa, colsum, groups, n_kchunks, st);
  } else {
    if (wide) return hipErrorInvalidValue;  // fp32 inputs: at most 128 score rows
    if (dk == 64) return launch_score_nw<In, 2, 4, 64, 3>(sa, colsum, groups, n_kchunks, st);
    if (dk == 128) return launch_score_nw<In, 4, 4, 64, 2>(sa, colsum, groups, n_kchunks, st);
  }
  return hipErrorInvalidValue;
}

snap_status launch_compress(const snap_params& p, const snap_cache& c, int32_t* pos, int32_t* n_topk, int n_seq,
                            const int32_t* slot_ids, const int32_t* lengths, int max_len, const void* q_obs,
                            const void* k, const void* v, int32_t* sel_out, float* pooled_out, void* ws,
                            hipStream_t stream, bool stats_given) {
  Geometry geo = compress_geometry(p, n_seq, max_len);
  const int groups = n_seq * p.n_kv_heads;
  const int G = p.n_q_heads / p.n_kv_heads;
  const float scale = p.sm_scale > 0.f ? p.sm_scale : 1.0f / sqrtf((float)p.d_qk);
  unsigned char* w = (unsigned char*)ws;
  float2* stats = (float2*)(w + geo.off_stats);
  float2* rowref = (float2*)(w + geo.off_rowref);
  float* A = (float*)(w + geo.off_A);
  float* P = (float*)(w + geo.off_P);
  uint32_t* hist = (uint32_t*)(w + geo.off_hist);
  RadixState* state = (RadixState*)(w + geo.off_state);
  uint2* counts = (uint2*)(w + geo.off_counts);
  int32_t* sel = (int32_t*)(w + geo.off_sel);
  double2* rowz = (double2*)(w + geo.off_rowz);
  int32_t* band_n = (int32_t*)(w + geo.off_band_n);
  int32_t* band_idx = (int32_t*)(w + geo.off_band_idx);
  double* band_p = (double*)(w + geo.off_band_p);
  uint32_t* band_above = (uint32_t*)(w + geo.off_band_above);
  double* A64 = (double*)(w + geo.off_A64);

  ScoreArgs sa;
  sa.q = q_obs;
  sa.k = k;
  sa.lengths = lengths;
  sa.stats = stats;
  sa.rowref = rowref;
  sa.A = A;
  sa.Hq = p.n_q_heads;
  sa.Hkv = p.n_kv_heads;
  sa.G = G;
  sa.w = p.obs_window;
  sa.max_len = max_len;
  sa.sink = p.sink;
  sa.recent = p.recent;
  sa.norm = p.norm;
  sa.rows = geo.rows;
  sa.rows_pad = geo.rows_pad;
  sa.key_chunk = geo.key_chunk;
  sa.n_kchunks = geo.n_kchunks;
  sa.scale = scale;
  split_scale2(scale, sa.scale2, sa.scale2_lo);
  const bool bf = p.in_dtype == SNAP_BF16;
  hipError_t e;
  // With no selected rows (StreamingLLM alone) the cache is sinks and ring
  // only: nothing is scored or selected (unless the pooled scores are asked
  // for), the assembly is the whole call.
  const bool select = p.topk > 0 || pooled_out;

  if (select) {
    // stats_given: the prefill attention pass already wrote each window row's
    // (max, sum) over its whole domain, as a single chunk
    if (!stats_given) {
      e = bf ? launch_score<uint16_t>(sa, p.d_qk, false, groups, geo.n_kchunks, stream)
             : launch_score<float>(sa, p.d_qk, false, groups, geo.n_kchunks, stream);
      if (e != hipSuccess) return SNAP_ERR_HIP;
    }

    ReduceArgs ra;
    ra.stats = stats;
    ra.rowref = rowref;
    ra.rowz = rowz;
    ra.band_n = band_n;
    ra.lengths = lengths;
    ra.hist = hist;
    ra.state = state;
    ra.groups = groups;
    ra.Hkv = p.n_kv_heads;
    ra.max_len = max_len;
    ra.sink = p.sink;
    ra.recent = p.recent;
    ra.topk = p.topk;
    ra.rows_pad = geo.rows_pad;
    ra.n_kchunks = stats_given ? 1 : geo.n_kchunks;
    hipLaunchKernelGGL(stats_reduce, dim3((geo.rows_pad + kReduceRows - 1) / kReduceRows, groups), dim3(256), 0,
                       stream, ra);
    if (hipGetLastError() != hipSuccess) return SNAP_ERR_HIP;

    e = bf ? launch_score<uint16_t>(sa, p.d_qk, true, groups, geo.n_kchunks, stream)
           : launch_score<float>(sa, p.d_qk, true, groups, geo.n_kchunks, stream);
    if (e != hipSuccess) return SNAP_ERR_HIP;

    SelectArgs se;
    se.A = A;
    se.P = P;
    se.pooled_out = pooled_out;
    se.lengths = lengths;
    se.hist = hist;
    se.state = state;
    se.counts = counts;
    se.sel = sel;
    se.band_n = band_n;
    se.band_idx = band_idx;
    se.band_above = band_above;
    se.groups = groups;
    se.Hkv = p.n_kv_heads;
    se.max_len = max_len;
    se.sink = p.sink;
    se.recent = p.recent;
    se.topk = p.topk;
    se.pool_kernel = p.pool_kernel;
    se.pool = p.pool;
    se.n_splits = geo.n_splits;
    dim3 sgrid(geo.n_splits, groups);
    hipLaunchKernelGGL(pool_hist0, sgrid, dim3(kSelThreads), 0, stream, se);
    hipLaunchKernelGGL(radix_scan, dim3(groups), dim3(kSelThreads), 0, stream, se, 0);
    hipLaunchKernelGGL(radix_pass, sgrid, dim3(kSelThreads), 0, stream, se, 1);
    hipLaunchKernelGGL(radix_scan, dim3(groups), dim3(kSelThreads), 0, stream, se, 1);
    hipLaunchKernelGGL(radix_pass, sgrid, dim3(kSelThreads), 0, stream, se, 2);
    hipLaunchKernelGGL(radix_scan, dim3(groups), dim3(kSelThreads), 0, stream, se, 2);
    hipLaunchKernelGGL(select_count, sgrid, dim3(kSelThreads), 0, stream, se);
    // fp64 re-score of the candidates next to the threshold, then the final
    // decision among them
    BandArgs ba;
    ba.q = q_obs;
    ba.k = k;
    ba.lengths = lengths;
    ba.rowz = rowz;
    ba.state = state;
    ba.band_n = band_n;
    ba.band_idx = band_idx;
    ba.A64 = A64;
    ba.band_p = band_p;
    ba.pooled_out = pooled_out;
    ba.P = P;
    ba.counts = counts;
    ba.band_above = band_above;
    ba.state_w = state;
    ba.Hq = p.n_q_heads;
    ba.Hkv = p.n_kv_heads;
    ba.G = G;
    ba.w = p.obs_window;
    ba.D = p.d_qk;
    ba.max_len = max_len;
    ba.sink = p.sink;
    ba.recent = p.recent;
    ba.pool_kernel = p.pool_kernel;
    ba.pool = p.pool;
    ba.rows = geo.rows;
    ba.rows_pad = geo.rows_pad;
    ba.n_splits = geo.n_splits;
    ba.in_f32 = !bf;
    ba.band_wgs = kBandWGs;
    // query-dim slices per score row: 8 for 576-wide bf16 rows and for fp32
    // rows, else 4 (as band_rescore dispatches)
    ba.rows_per_pass = kBandThreads / ((!bf || p.d_qk == 576) ? 8 : 4);
    ba.scale2 = (double)scale * 1.4426950408889634074;
    hipLaunchKernelGGL(band_rescore, dim3(kBandWGs, groups), dim3(kBandThreads), 0, stream, ba);
    hipLaunchKernelGGL(band_decide, dim3(groups), dim3(kSelThreads), 0, stream, ba);
    hipLaunchKernelGGL(select_write, sgrid, dim3(kSelThreads), 0, stream, se);
    if (hipGetLastError() != hipSuccess) return SNAP_ERR_HIP;
  }

  AssembleArgs aa;
  aa.k = k;
  aa.v = p.v_in_k ? nullptr : v;
  aa.ck = c.k;
  aa.cv = p.v_in_k ? nullptr : c.v;
  aa.k_scale = c.k_scale;
  aa.v_scale = c.v_scale;
  aa.slot_ids = slot_ids;
  aa.lengths = lengths;
  aa.sel = sel;
  aa.state = state;
  aa.sel_out = sel_out;
  aa.pos = pos;
  aa.n_topk = n_topk;
  aa.Hkv = p.n_kv_heads;
  aa.max_len = max_len;
  aa.sink = p.sink;
  aa.recent = p.recent;
  aa.topk = p.topk;
  aa.dk = p.d_qk;
  aa.dv = p.d_v;
  aa.n_slots = c.n_slots;
  aa.rows_per_block = kAsmRows;
  aa.n_rowblocks = geo.n_rowblocks;
  aa.amax = nullptr;
  dim3 agrid(geo.n_rowblocks, groups);
  if (p.kv_dtype == SNAP_FP8_E4M3 && p.fp8_scales == SNAP_FP8_SCALES_AMAX) {
    aa.amax = (float2*)(w + geo.off_amax);
    hipLaunchKernelGGL(fp8_amax, agrid, dim3(256), 0, stream, aa);
  }
  if (p.kv_dtype == SNAP_FP8_E4M3) {
    if (bf)
      hipLaunchKernelGGL((assemble<uint16_t, uint8_t>), agrid, dim3(256), 0, stream, aa);
    else
      hipLaunchKernelGGL((assemble<float, uint8_t>), agrid, dim3(256), 0, stream, aa);
  } else if (bf) {
    hipLaunchKernelGGL((assemble<uint16_t, uint16_t>), agrid, dim3(256), 0, stream, aa);
  } else {
    hipLaunchKernelGGL((assemble<float, float>), agrid, dim3(256), 0, stream, aa);
  }
  if (hipGetLastError() != hipSuccess) return SNAP_ERR_HIP;
  return SNAP_OK;
}

}  // namespace snap
