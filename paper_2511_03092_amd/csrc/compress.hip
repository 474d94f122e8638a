// compress.hip -- SnapStream compression at the end of prefill (arXiv
// 2511.03092, Sec. III-B): SnapKV window scores (Eq. 3), window + group sum
// (Eq. 1), 1-D pooling and top-K (Eq. 2), then the gather into the fixed-size
// sink / ring / top-K cache (Sec. III-A).
//
// Kernel sequence per call (one stream, no host synchronisation):
//   score_pass<STATS>   per (seq, KV head, key chunk): bf16 MFMA Q_obs x K^T,
//                       per-row running max / sum-exp of the softmax domain
//   stats_reduce        per (seq, KV head): row max + normaliser (fp64), and
//                       the reset of the selection scratch
//   score_pass<COLSUM>  recompute the scores, W = exp(z - c) * inv, column
//                       sums over the G*w window rows -> A[j]
//   pool_hist0          P = pool(A) over the candidates, first radix digit
//   radix_pass x2       remaining digits of the K-th largest P (LDS histograms,
//                       the last workgroup of a group picks the bin)
//   select_count/write  ordered compaction: P > t, plus the lowest-index ties
//   assemble            sinks, ring rows, kept rows, zero padding (+ fp8)
#include <float.h>
#include <math.h>

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
  float scale;
};

// Row state of one lane: the MFMA 16x16 output gives lane l the rows
// 4*(l/16)+e (e = 0..3) of each 16-row block and the key column l%16.
template <typename In, int KSTEPS, bool COLSUM>
__global__ __launch_bounds__(512) void score_pass(ScoreArgs a) {
  constexpr bool kBF16 = sizeof(In) == 2;
  constexpr int D = KSTEPS * 32;
  constexpr int kPitch = D * (int)sizeof(In) + 16;  // padded LDS row (bytes)
  extern __shared__ __align__(16) unsigned char smem[];
  unsigned char* ktile = smem;                                   // [kKeyTile][kPitch]
  float* colbuf = (float*)(smem + kKeyTile * kPitch);            // [waves][kKeyTile]
  float* qlds = colbuf + 8 * kKeyTile;                           // fp32 inputs: [rows_pad][D]

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nwaves = blockDim.x >> 6;
  const int l16 = lane & 15, lg = lane >> 4;
  const int bg = blockIdx.y, b = bg / a.Hkv, g = bg % a.Hkv;
  int L = a.lengths[b];
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
  const int c0 = lo + blockIdx.x * a.key_chunk;
  const int c1 = min(c0 + a.key_chunk, hi);
  const int we = min(a.w, L);

  // positions and validity of this lane's 8 rows
  int rpos[2][4];
  bool rval[2][4];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      int rho = wave * 32 + rb * 16 + lg * 4 + e;
      int ii = rho % a.w;
      rval[rb][e] = rho < a.rows && ii >= a.w - we;
      rpos[rb][e] = L - a.w + ii;
    }

  float2* st_out = a.stats + ((size_t)bg * a.n_kchunks + blockIdx.x) * a.rows_pad;
  if (c0 >= c1) {
    if (!COLSUM) {
      for (int t = threadIdx.x; t < a.rows_pad; t += blockDim.x) st_out[t] = make_float2(-INFINITY, 0.f);
    }
    return;
  }

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
    for (int i = threadIdx.x; i < a.rows_pad * D; i += blockDim.x) {
      int rho = i / D;
      qlds[i] = rho < a.rows ? ((const float*)qbase)[i] : 0.f;
    }
  }

  float rm[2][4], rz[2][4], rc[2][4], rinv[2][4];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      rm[rb][e] = -INFINITY;
      rz[rb][e] = 0.f;
      if (COLSUM) {
        int rho = wave * 32 + rb * 16 + lg * 4 + e;
        float2 rf = a.rowref[(size_t)bg * a.rows_pad + rho];
        rc[rb][e] = rf.x;
        rinv[rb][e] = rval[rb][e] ? rf.y : 0.f;
      }
    }

  const unsigned char* kbase = (const unsigned char*)a.k + ((size_t)b * a.Hkv + g) * (size_t)a.max_len * D * sizeof(In);
  constexpr int kChunks16 = D * (int)sizeof(In) / 16;  // 16-byte pieces per key row

  for (int t0 = c0; t0 < c1; t0 += kKeyTile) {
    __syncthreads();
    for (int i = threadIdx.x; i < kKeyTile * kChunks16; i += blockDim.x) {
      int kk = i / kChunks16, pc = i % kChunks16;
      int j = t0 + kk;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (j < c1) v = *(const u32x4*)(kbase + (size_t)j * D * sizeof(In) + pc * 16);
      *(u32x4*)(ktile + kk * kPitch + pc * 16) = v;
    }
    __syncthreads();

    float xv[2][4][kKeyTile / 16];
#pragma unroll
    for (int sb = 0; sb < kKeyTile / 16; ++sb) {
      f32x4 acc[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
      if constexpr (kBF16) {
        const unsigned char* krow = ktile + (sb * 16 + l16) * kPitch;
#pragma unroll
        for (int t = 0; t < KSTEPS; ++t) {
          bf16x8 kf = __builtin_bit_cast(bf16x8, *(const u32x4*)(krow + 16 * (KSTEPS * lg + t)));
          acc[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qf[0][t], kf, acc[0], 0, 0, 0);
          acc[1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qf[1][t], kf, acc[1], 0, 0, 0);
        }
      } else {
        const float* krow = (const float*)(ktile + (sb * 16 + l16) * kPitch);
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float* qrow = qlds + (size_t)(wave * 32 + rb * 16 + lg * 4 + e) * D;
            // fp32 products are exact in fp64; only the final rounding remains
            double sacc = 0.0;
#pragma unroll 4
            for (int d = 0; d < D; ++d) sacc = fma((double)qrow[d], (double)krow[d], sacc);
            acc[rb][e] = (float)sacc;
          }
      }
      const int j = t0 + sb * 16 + l16;
      float colv[2][4];
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          bool in = rval[rb][e] && j < c1 && j <= rpos[rb][e];
          float x = acc[rb][e] * a.scale;
          if (!COLSUM) {
            xv[rb][e][sb] = in ? x : -INFINITY;
          } else {
            colv[rb][e] = in ? expf(x - rc[rb][e]) * rinv[rb][e] : 0.f;
          }
        }
      if (COLSUM) {
        float cs = ((colv[0][0] + colv[0][1]) + (colv[0][2] + colv[0][3])) +
                   ((colv[1][0] + colv[1][1]) + (colv[1][2] + colv[1][3]));
        cs += __shfl_xor(cs, 16);
        cs += __shfl_xor(cs, 32);
        if (lg == 0) colbuf[wave * kKeyTile + sb * 16 + l16] = cs;
      }
    }

    if (!COLSUM) {
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float mt = xv[rb][e][0];
#pragma unroll
          for (int sb = 1; sb < kKeyTile / 16; ++sb) mt = fmaxf(mt, xv[rb][e][sb]);
          float mn = fmaxf(rm[rb][e], mt);
          if (mn == -INFINITY) continue;
          float z = rz[rb][e] * __expf(rm[rb][e] - mn);
#pragma unroll
          for (int sb = 0; sb < kKeyTile / 16; ++sb) z += __expf(xv[rb][e][sb] - mn);
          rz[rb][e] = z;
          rm[rb][e] = mn;
        }
    } else {
      __syncthreads();
      if (threadIdx.x < kKeyTile) {
        int j = t0 + threadIdx.x;
        float sum = 0.f;
        if (nwaves == 4) {
          sum = (colbuf[threadIdx.x] + colbuf[kKeyTile + threadIdx.x]) +
                (colbuf[2 * kKeyTile + threadIdx.x] + colbuf[3 * kKeyTile + threadIdx.x]);
        } else if (nwaves == 8) {
          const float* c = colbuf + threadIdx.x;
          sum = ((c[0] + c[kKeyTile]) + (c[2 * kKeyTile] + c[3 * kKeyTile])) +
                ((c[4 * kKeyTile] + c[5 * kKeyTile]) + (c[6 * kKeyTile] + c[7 * kKeyTile]));
        } else {
          for (int wv = 0; wv < nwaves; ++wv) sum += colbuf[wv * kKeyTile + threadIdx.x];
        }
        if (j < c1) a.A[(size_t)bg * a.max_len + j] = sum;
      }
    }
  }

  if (!COLSUM) {
    // combine the 16 key columns of each row (lanes with equal l/16)
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float m = rm[rb][e], z = rz[rb][e];
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) {
          float m2 = __shfl_xor(m, o), z2 = __shfl_xor(z, o);
          float mn = fmaxf(m, m2);
          if (mn != -INFINITY) {
            z = z * __expf(m - mn) + z2 * __expf(m2 - mn);
            m = mn;
          }
        }
        if (l16 == 0) st_out[wave * 32 + rb * 16 + lg * 4 + e] = make_float2(m, z);
      }
  }
}

// ============================================================ row normalisers
struct ReduceArgs {
  const float2* stats;
  float2* rowref;
  const int32_t* lengths;
  uint32_t* hist;      // [3][groups][kRadixBins]
  RadixState* state;   // [groups]
  int groups, Hkv, max_len, sink, recent, topk;
  int rows_pad, n_kchunks;
};

// Row max m over every chunk and the normaliser.  The reference c is 0 when the
// max lies in [-20, 64] (then exp(z) is taken directly, keeping the full fp32
// accuracy of small logits), otherwise c = m; inv = 1 / sum_j exp(z_j - c),
// accumulated in fp64.  Eight lanes share a row (chunks strided by 8) and
// combine with in-wave shuffles; block 0 of each group also resets the
// group's selection scratch.
constexpr int kReduceLanes = 8;
__global__ __launch_bounds__(256) void stats_reduce(ReduceArgs a) {
  const int bg = blockIdx.y, b = bg / a.Hkv;
  const int sub = threadIdx.x % kReduceLanes;
  const int rho = blockIdx.x * (256 / kReduceLanes) + threadIdx.x / kReduceLanes;
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
        if (v.x != -INFINITY) z += (double)v.y * exp((double)v.x - (double)m);
      }
    }
#pragma unroll
    for (int o = 1; o < kReduceLanes; o <<= 1) z += __shfl_xor(z, o);
    if (sub == 0) {
      float2 ref = make_float2(0.f, 0.f);
      if (m != -INFINITY) {
        if (m >= -20.f && m <= 64.f) {
          ref.x = 0.f;
          ref.y = (float)(1.0 / (z * exp((double)m)));
        } else {
          ref.x = m;
          ref.y = (float)(1.0 / z);
        }
      }
      a.rowref[(size_t)bg * a.rows_pad + rho] = ref;
    }
  }
  if (blockIdx.x != 0) return;
  for (int pass = 0; pass < 3; ++pass) {
    uint32_t* h = a.hist + ((size_t)pass * a.groups + bg) * kRadixBins;
    for (int i = threadIdx.x; i < kRadixBins; i += blockDim.x) h[i] = 0u;
  }
  if (threadIdx.x == 0) {
    int L = a.lengths[b];
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
  int groups, Hkv, max_len, sink, recent, topk, pool_kernel, pool, n_splits;
};

__device__ __forceinline__ void seq_range(const SelectArgs& a, int bg, int& c0, int& c1) {
  int b = bg / a.Hkv;
  int L = a.lengths[b];
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
  for (int i = threadIdx.x; i < nb; i += blockDim.x) {
    uint32_t v = 0;
#pragma unroll
    for (int w = 0; w < kSubHists; ++w) v += lhist[w][i];
    if (v) atomicAdd(&gh[i], v);
  }
}

__device__ __forceinline__ void clear_hists(uint32_t (*lhist)[kRadixBins]) {
  for (int i = threadIdx.x; i < kSubHists * kRadixBins; i += blockDim.x) (&lhist[0][0])[i] = 0u;
}

// P = pool(A) on this workgroup's candidates (+ the debug copy) and the first
// radix digit.
__global__ __launch_bounds__(kSelThreads) void pool_hist0(SelectArgs a) {
  __shared__ float la[kCandChunk + 64];
  __shared__ uint32_t lhist[kSubHists][kRadixBins];
  const int bg = blockIdx.y, split = blockIdx.x;
  const int wave = threadIdx.x >> 6;
  int c0, c1;
  seq_range(a, bg, c0, c1);
  const int half = a.pool_kernel / 2;
  const int j0 = c0 + split * kCandChunk, j1 = min(j0 + kCandChunk, c1);
  const RadixState st = a.state[bg];
  float* Pg = a.P + (size_t)bg * a.max_len;

  if (a.pooled_out && split == 0) {
    float* po = a.pooled_out + (size_t)bg * a.max_len;
    for (int j = threadIdx.x; j < a.max_len; j += blockDim.x)
      if (j < c0 || j >= c1) po[j] = __builtin_nanf("");
  }
  if (st.mode == 2) clear_hists(lhist);
  if (j0 < j1) {
    const float* Ag = a.A + (size_t)bg * a.max_len;
    const float padv = a.pool == SNAP_POOL_MAX ? -INFINITY : 0.f;
    for (int i = threadIdx.x; i < (j1 - j0) + 2 * half; i += blockDim.x) {
      int t = j0 - half + i;
      la[i] = (t >= c0 && t < c1) ? Ag[t] : padv;
    }
    __syncthreads();
    for (int j = j0 + threadIdx.x; j < j1; j += blockDim.x) {
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
  const int bg = blockIdx.y, split = blockIdx.x;
  const int wave = threadIdx.x >> 6;
  const RadixState st = a.state[bg];
  if (st.mode != 2) return;
  int c0, c1;
  seq_range(a, bg, c0, c1);
  const int j0 = c0 + split * kCandChunk, j1 = min(j0 + kCandChunk, c1);
  clear_hists(lhist);
  __syncthreads();
  const float* Pg = a.P + (size_t)bg * a.max_len;
  for (int j = j0 + threadIdx.x; j < j1; j += blockDim.x) {
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
  const int bg = blockIdx.x;
  RadixState st = a.state[bg];
  if (st.mode != 2) return;
  const int nb = pass == 2 ? 1024 : 2048;
  const int per = nb / kSelThreads;  // 8 or 4
  const uint32_t* gh = a.hist + ((size_t)pass * a.groups + bg) * kRadixBins;
  const int top = nb - per * threadIdx.x;  // this thread's bins: [top - per, top)
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

// block-wide exclusive scan of one value per thread (kSelThreads threads)
__device__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* lds, uint32_t& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
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
  for (int w2 = 0; w2 < kSelThreads / 64; ++w2) {
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
  const int bg = blockIdx.y, split = blockIdx.x;
  const RadixState st = a.state[bg];
  if (st.mode != 2) return;
  int c0, c1;
  seq_range(a, bg, c0, c1);
  const int j0 = c0 + split * kCandChunk, j1 = min(j0 + kCandChunk, c1);
  const float* Pg = a.P + (size_t)bg * a.max_len;
  uint32_t gt = 0, eq = 0;
  for (int j = j0 + threadIdx.x; j < j1; j += blockDim.x) {
    uint32_t bits = __float_as_uint(Pg[j]);
    gt += bits > st.prefix;
    eq += bits == st.prefix;
  }
  uint32_t tg, te;
  block_exclusive_scan(gt, lds, tg);
  block_exclusive_scan(eq, lds, te);
  if (threadIdx.x == 0) a.counts[(size_t)bg * a.n_splits + split] = make_uint2(tg, te);
}

// Ordered compaction: a candidate is kept when P > t, or P == t and it is among
// the krem lowest-index candidates equal to t.  Output is in token order.
__global__ __launch_bounds__(kSelThreads) void select_write(SelectArgs a) {
  __shared__ uint32_t lds[8];
  const int bg = blockIdx.y, split = blockIdx.x;
  const RadixState st = a.state[bg];
  if (st.mode == 0) return;
  int c0, c1;
  seq_range(a, bg, c0, c1);
  const int j0 = c0 + split * kCandChunk, j1 = min(j0 + kCandChunk, c1);
  int32_t* sg = a.sel + (size_t)bg * a.topk;
  if (st.mode == 1) {
    for (int j = j0 + threadIdx.x; j < j1; j += blockDim.x) sg[j - c0] = j;
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
  const int jt = j0 + threadIdx.x * kPerThread;
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
      if (pos < keff) sg[pos] = jt + i;  // never past the group's K slots
      ++pos;
    }
}

// ============================================================ assemble
struct AssembleArgs {
  const void* k;       // [n_seq][Hkv][max_len][dk]
  const void* v;       // or NULL
  void* ck;            // [n_slots][Hkv][B][dk]
  void* cv;
  const float* k_scale;
  const float* v_scale;
  const int32_t* slot_ids;
  const int32_t* lengths;
  const int32_t* sel;  // [groups][topk]
  const RadixState* state;
  int32_t* sel_out;    // optional [groups][topk]
  int32_t* pos;
  int32_t* n_topk;
  int Hkv, max_len, sink, recent, topk, dk, dv, n_slots, rows_per_block;
};

// Source token of cache row `row` (or -1 for a zero padding row).
__device__ __forceinline__ int row_source(int row, int L, int s, int r, int keff, const int32_t* sel) {
  if (row < s) return row < L ? row : -1;
  if (row < s + r) {
    int l0 = L - r > s ? L - r : s;  // first ring token
    int off = ((row - s) - (l0 - s)) % r;
    if (off < 0) off += r;
    int t = l0 + off;
    return t < L ? t : -1;
  }
  int m = row - s - r;
  return m < keff ? sel[m] : -1;
}

template <typename In, typename Out>
__device__ __forceinline__ void copy_row(const In* src, Out* dst, int width, float inv_scale_unused, float scale,
                                         int tid, int nthr) {
  (void)inv_scale_unused;
  if constexpr (sizeof(Out) == 1) {
    // quantise 8 elements per step (In = bf16 or fp32)
    for (int c = tid; c < width / 8; c += nthr) {
      float f[8];
      if constexpr (sizeof(In) == 2) {
        u32x4 raw = src ? *(const u32x4*)(src + c * 8) : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          f[2 * i] = bf16_bits_to_f32(raw[i] & 0xffffu);
          f[2 * i + 1] = bf16_bits_to_f32(raw[i] >> 16);
        }
      } else {
        for (int i = 0; i < 8; ++i) f[i] = src ? ((const float*)src)[c * 8 + i] : 0.f;
      }
      u32x2 o;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        uint32_t w = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) w |= f32_to_e4m3(f[h * 4 + i] / scale) << (8 * i);
        o[h] = w;
      }
      *(u32x2*)((uint8_t*)dst + c * 8) = o;
    }
  } else {
    constexpr int per = 16 / sizeof(In);
    for (int c = tid; c < width / per; c += nthr) {
      u32x4 raw = src ? *(const u32x4*)(src + c * per) : u32x4{0u, 0u, 0u, 0u};
      *(u32x4*)(dst + c * per) = raw;
    }
  }
}

template <typename In, typename Out>
__global__ __launch_bounds__(256) void assemble(AssembleArgs a) {
  const int bg = blockIdx.y, b = bg / a.Hkv, g = bg % a.Hkv;
  const int slot = a.slot_ids[b];
  const int s = a.sink, r = a.recent, B = s + r + a.topk;
  int L = a.lengths[b];
  L = L < 0 ? 0 : (L > a.max_len ? a.max_len : L);
  const int keff = a.state[bg].keff;
  const int32_t* sg = a.sel + (size_t)bg * a.topk;
  const int row0 = blockIdx.x * a.rows_per_block;
  const int row1 = min(row0 + a.rows_per_block, B);

  if (a.sel_out) {
    for (int m = row0 + threadIdx.x; m < row1; m += blockDim.x) {
      int mm = m - s - r;
      if (mm >= 0) a.sel_out[(size_t)bg * a.topk + mm] = mm < keff ? sg[mm] : -1;
    }
  }
  if (slot < 0 || slot >= a.n_slots) return;
  if (blockIdx.x == 0 && g == 0 && threadIdx.x == 0) {
    a.pos[slot] = L;
    a.n_topk[slot] = keff;
  }
  const size_t in_row0 = ((size_t)b * a.Hkv + g) * (size_t)a.max_len;
  const size_t out_row0 = ((size_t)slot * a.Hkv + g) * (size_t)B;
  const float ks = (sizeof(Out) == 1) ? a.k_scale[(size_t)slot * a.Hkv + g] : 1.f;
  const float vs = (sizeof(Out) == 1 && a.v) ? a.v_scale[(size_t)slot * a.Hkv + g] : 1.f;
  // one wave per row at a time
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  for (int row = row0 + wave; row < row1; row += nw) {
    int t = row_source(row, L, s, r, keff, sg);
    const In* ksrc = t >= 0 ? (const In*)a.k + (in_row0 + t) * a.dk : nullptr;
    copy_row<In, Out>(ksrc, (Out*)a.ck + (out_row0 + row) * a.dk, a.dk, 0.f, ks, lane, 64);
    if (a.v) {
      const In* vsrc = t >= 0 ? (const In*)a.v + (in_row0 + t) * a.dv : nullptr;
      copy_row<In, Out>(vsrc, (Out*)a.cv + (out_row0 + row) * a.dv, a.dv, 0.f, vs, lane, 64);
    }
  }
}

// ============================================================ host side
static inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

Geometry compress_geometry(const snap_params& p, int n_seq, int max_len) {
  Geometry g{};
  int G = p.n_q_heads / p.n_kv_heads;
  g.rows = G * p.obs_window;
  g.rows_pad = (g.rows + 31) / 32 * 32;
  int groups = n_seq * p.n_kv_heads;
  // enough workgroups to cover 256 CUs several times, at most 4096 keys each
  long target = 4096;
  long per_group = (target + groups - 1) / (groups > 0 ? groups : 1);
  long kc = (max_len + per_group - 1) / (per_group > 0 ? per_group : 1);
  kc = (kc + kKeyTile - 1) / kKeyTile * kKeyTile;
  if (kc < kKeyTile) kc = kKeyTile;
  if (kc > 4096) kc = 4096;
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
  g.compress_bytes = off;
  return g;
}

template <typename In>
static hipError_t launch_score(const ScoreArgs& sa, int dk, int nwaves, bool colsum, int groups, int n_kchunks,
                               hipStream_t st) {
  dim3 grid(n_kchunks, groups);
  dim3 block(64 * nwaves);
  size_t pitch = (size_t)dk * sizeof(In) + 16;
  size_t lds = kKeyTile * pitch + 8 * kKeyTile * sizeof(float);
  if (sizeof(In) == 4) lds += (size_t)sa.rows_pad * dk * sizeof(float);
#define SNAP_SCORE(KS)                                                                        \
  if (dk == KS * 32) {                                                                        \
    const void* fn = colsum ? (const void*)score_pass<In, KS, true> : (const void*)score_pass<In, KS, false>; \
    if (lds > 65536) {                                                                        \
      hipError_t ae = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds); \
      if (ae != hipSuccess) return ae;                                                        \
    }                                                                                         \
    if (colsum)                                                                               \
      hipLaunchKernelGGL((score_pass<In, KS, true>), grid, block, lds, st, sa);               \
    else                                                                                      \
      hipLaunchKernelGGL((score_pass<In, KS, false>), grid, block, lds, st, sa);              \
    return hipGetLastError();                                                                 \
  }
  if constexpr (sizeof(In) == 2) {
    SNAP_SCORE(2)
    SNAP_SCORE(4)
    SNAP_SCORE(18)
  } else {
    SNAP_SCORE(2)
    SNAP_SCORE(4)
  }
#undef SNAP_SCORE
  return hipErrorInvalidValue;
}

snap_status launch_compress(const snap_params& p, const snap_cache& c, int32_t* pos, int32_t* n_topk, int n_seq,
                            const int32_t* slot_ids, const int32_t* lengths, int max_len, const void* q_obs,
                            const void* k, const void* v, int32_t* sel_out, float* pooled_out, void* ws,
                            hipStream_t stream) {
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
  const int nwaves = geo.rows_pad / 32;
  const bool bf = p.in_dtype == SNAP_BF16;
  hipError_t e;

  e = bf ? launch_score<uint16_t>(sa, p.d_qk, nwaves, false, groups, geo.n_kchunks, stream)
         : launch_score<float>(sa, p.d_qk, nwaves, false, groups, geo.n_kchunks, stream);
  if (e != hipSuccess) return SNAP_ERR_HIP;

  ReduceArgs ra;
  ra.stats = stats;
  ra.rowref = rowref;
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
  ra.n_kchunks = geo.n_kchunks;
  hipLaunchKernelGGL(stats_reduce, dim3((geo.rows_pad + 31) / 32, groups), dim3(256), 0, stream, ra);
  if (hipGetLastError() != hipSuccess) return SNAP_ERR_HIP;

  e = bf ? launch_score<uint16_t>(sa, p.d_qk, nwaves, true, groups, geo.n_kchunks, stream)
         : launch_score<float>(sa, p.d_qk, nwaves, true, groups, geo.n_kchunks, stream);
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
  hipLaunchKernelGGL(select_write, sgrid, dim3(kSelThreads), 0, stream, se);
  if (hipGetLastError() != hipSuccess) return SNAP_ERR_HIP;

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
  aa.rows_per_block = 64;
  const int B = p.sink + p.recent + p.topk;
  dim3 agrid((B + aa.rows_per_block - 1) / aa.rows_per_block, groups);
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
