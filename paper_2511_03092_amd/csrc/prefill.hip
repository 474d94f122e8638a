// prefill.hip -- causal attention over the whole prompt with the SnapKV
// observation-window statistics fused in (arXiv 2511.03092).
//
// The paper's prefill graph runs a FlashAttention-style attention kernel
// (Sec. IV-A: Q K^T, softmax and P V in one kernel, the attention matrix never
// stored) and recomputes the window rows' scores outside it (Sec. III-B.2),
// a cost it leaves to future work.  Here the attention kernel itself produces,
// for the last w query rows of every (sequence, KV head), the softmax
// statistics the SnapKV scores need (row max and sum of exponentials over the
// normaliser domain of Eq. 3, or over the whole causal row) and writes the
// window queries out, so the scoring stage reads the keys once (the column
// sums) instead of twice.
//
// Kernel sequence per call (one stream, no host synchronisation):
//   vt_transpose   V -> V^T per (sequence, KV head): keys contiguous, zero past
//                  the prompt (the A operand of the P V product)
//   prefill_attn   per (KV head, block of query positions): online softmax over
//                  64-key tiles streamed into LDS, bf16 MFMA for both products;
//                  blocks holding window rows also write their statistics and
//                  queries
//   stats_reduce, score_pass<COLSUM>, pool / select, assemble (compress.hip)
#include <math.h>

#include "lds_dma.h"
#include "snap_internal.h"

namespace snap {

constexpr int kPfTK = 64;  // keys per tile
constexpr int kPfNW = 8;   // waves per workgroup, 32 query rows each

struct PrefillArgs {
  const uint16_t* q;   // [n_seq][Hq][max_len][D]
  const uint16_t* k;   // [n_seq][Hkv][max_len][D]
  const uint16_t* vt;  // [n_seq*Hkv][D][ld_vt]
  uint16_t* out;       // [n_seq][Hq][max_len][D]
  const int32_t* lengths;
  float2* stats;       // [n_seq*Hkv][rows_pad]: (max, sum of 2^(y - max)), y in log2 units
  uint16_t* qobs;      // [n_seq][Hq][w][D]
  int Hq, Hkv, G, max_len, ld_vt, w, sink, recent, norm, rows, rows_pad, want_stats;
  int P;               // query positions per workgroup
  int n_qblocks, groups;  // workgroups per group (max_len / P rounded up), n_seq * Hkv
  float scale2;        // softmax scale * log2(e) as scale2 + scale2_lo (split_scale2)
  float scale2_lo;
};

// Query positions per workgroup for G heads per KV head: the 256 rows of a
// workgroup are (head, position) pairs of one KV head, so every key tile in
// LDS serves all G heads.
static inline int prefill_positions(int G) { return 256 / G; }

// Head within the group and position offset within the workgroup of row block
// rb (16 rows) of wave w: the workgroup's 16 row blocks run over the G heads
// fastest, then over blocks of 16 positions.
__device__ __forceinline__ void pf_rowblock(int G, int w, int rb, int& hl, int& po) {
  const int rbi = 2 * w + rb;
  hl = rbi % G;
  po = 16 * (rbi / G);
}

// Key order of V^T within each 32-key group: stored position u = 8q + 4h + e
// holds key 16h + 4q + e (q < 4, h < 2, e < 4), so that the eight keys one
// lane group needs for an MFMA operand (keys 4q..4q+3 and 16+4q..16+4q+3,
// the layout the S^T product leaves the probabilities in) are one 16-byte
// chunk.
__device__ __forceinline__ int vt_key(int u) {
  return (u & ~31) + 16 * ((u >> 2) & 1) + 4 * ((u >> 3) & 3) + (u & 3);
}

// V [bg][max_len][D] -> V^T [bg][D][ld_vt] for 64 keys per workgroup; keys at
// or past the prompt length are written as zeros (they meet a zero weight in
// the P V product, and must be finite for that).
template <int D>
__global__ __launch_bounds__(256) void vt_transpose(const uint16_t* __restrict__ v, uint16_t* __restrict__ vt,
                                                    const int32_t* lengths, int Hkv, int max_len, int ld_vt) {
  __shared__ uint16_t tile[64][D + 2];
  const int bg = bid_y(), b = bg / Hkv;
  int L = uniform(lengths[b]);
  L = L < 0 ? 0 : (L > max_len ? max_len : L);
  const int k0 = bid_x() * 64;
  constexpr int C8 = D / 8;  // 16-byte chunks per row
  for (int c = tid(); c < 64 * C8; c += nthreads()) {
    const int key = c / C8, d8 = c % C8;
    const int j = k0 + key;
    u32x4 x = {0u, 0u, 0u, 0u};
    if (j < L) x = *(const u32x4*)(v + ((size_t)bg * max_len + j) * D + d8 * 8);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      tile[key][d8 * 8 + 2 * i] = (uint16_t)(x[i] & 0xffffu);
      tile[key][d8 * 8 + 2 * i + 1] = (uint16_t)(x[i] >> 16);
    }
  }
  __syncthreads();
  for (int c = tid(); c < D * 8; c += nthreads()) {
    const int dv = c / 8, kc = c % 8;
    u32x4 x;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      x[i] = (uint32_t)tile[vt_key(kc * 8 + 2 * i)][dv] | ((uint32_t)tile[vt_key(kc * 8 + 2 * i + 1)][dv] << 16);
    *(u32x4*)(vt + ((size_t)bg * D + dv) * ld_vt + k0 + kc * 8) = x;
  }
}

// Max over the four lanes l, l^16, l^32, l^48 (the lane groups that share a
// query row in the S^T layout), by the two lane-swap instructions of gfx950
// (no LDS round trip).
__device__ __forceinline__ float lanes4_max(float x) {
  const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
  const auto q = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(q[0]), __uint_as_float(q[1]));
}

// One workgroup per (KV head group bg, block kb of P query positions counted
// from the end of the prompt: block 0 holds positions [L-P, L), the window).
// Rows: 8 waves x 32 (head, position) pairs.  Products, per 64-key tile:
//   S^T = K Q^T   (A = K fragment from LDS, B = Q fragment held in registers):
//                 lane l gets query row l%16 against keys 4*(l/16)+e of each
//                 16-key block, so a row's softmax is lane-local up to a
//                 reduction over the four lane groups;
//   O^T += V^T P^T (A = V^T fragment from LDS, B = the probabilities exactly
//                 as the first product left them in registers, cast to bf16).
// Two LDS stages, each a K tile then a V^T tile, filled by direct loads.
template <int KS>
__global__ __launch_bounds__(512) void prefill_attn(PrefillArgs a) {
  constexpr int D = KS * 32;
  constexpr int CPR = D / 8;   // 16-byte chunks per key row
  constexpr int DVB = D / 16;  // value blocks of 16 dims
  constexpr int kKBytes = kPfTK * D * 2;
  constexpr int kLoadsPerWave = CPR / kPfNW;  // per tile and per operand
  static_assert(CPR % kPfNW == 0, "equal loads per wave");
  __shared__ __align__(16) unsigned char lds[4 * kKBytes];  // two stages of (K tile, V^T tile)

  const int lane = tid() & 63, wave = tid() >> 6;
  const int l16 = lane & 15, lg = lane >> 4;
  // Workgroup order: consecutive workgroups go to the 8 XCDs in turn; XCD x
  // takes KV heads (groups) x, x+8, x+16, ... one after the other, each from
  // its last positions (the most keys) to its first, so that the workgroups
  // resident on one XCD share the same K and V tiles in its L2.
  const int xcd = bid_x() % 8, r = bid_x() / 8;
  const int bg = (r / a.n_qblocks) * 8 + xcd;
  const int kblk = r % a.n_qblocks;
  if (bg >= a.groups) return;
  const int b = bg / a.Hkv, g = bg % a.Hkv;
  int L = uniform(a.lengths[b]);
  L = L < 0 ? 0 : (L > a.max_len ? a.max_len : L);
  const int P = a.P;
  const int top = L - P * kblk;  // one past this workgroup's last position
  if (top <= 0) return;
  if (!debug_check(top <= L && L <= a.max_len, kDbgPrefill)) return;
  const int pos0 = top - P;  // first position (negative in a partial block)
  const int nt = (top + kPfTK - 1) / kPfTK;
  const float s2 = a.scale2;

  int hl[2], prow[2];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    int po;
    pf_rowblock(a.G, wave, rb, hl[rb], po);
    prow[rb] = pos0 + po + l16;
  }

  // query fragments: row l16 of each row block, chunks KS*lg + t
  bf16x8 qf[2][KS];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    const uint16_t* qrow =
        a.q + (((size_t)b * a.Hq + (size_t)g * a.G + hl[rb]) * a.max_len + (prow[rb] < 0 ? 0 : prow[rb])) * D;
#pragma unroll
    for (int t = 0; t < KS; ++t) {
      u32x4 x = {0u, 0u, 0u, 0u};
      if (prow[rb] >= 0) x = *(const u32x4*)(qrow + 8 * (KS * lg + t));
      qf[rb][t] = __builtin_bit_cast(bf16x8, x);
    }
  }

  f32x4 o[2][DVB];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int d = 0; d < DVB; ++d) o[rb][d] = f32x4{0.f, 0.f, 0.f, 0.f};
  // Row sums: each tile's 16 terms per lane are summed in fp32, the running
  // sums are kept in fp64 (a window row's normaliser sums up to L terms and
  // feeds the selection directly).
  float m[2] = {-INFINITY, -INFINITY};
  double ls[2] = {0.0, 0.0};
  // window workgroups also keep the window rows' statistics over the
  // normaliser's domain -- C = [sink, L - recent) intersected with the
  // causal prefix (Eq. 3), or the causal row -- with the full scale
  // (s2 + s2lo) of the compression's weights in their exponents, which the
  // attention's own softmax does not carry
  const bool win = a.want_stats && top > L - a.w;
  const bool cand_norm = a.norm == SNAP_NORM_CAND;
  const int clo = cand_norm ? a.sink : 0, chi = cand_norm ? L - a.recent : L;
  const float s2lo = a.scale2_lo;
  float mc[2] = {-INFINITY, -INFINITY};
  double zc[2] = {0.0, 0.0};

  const unsigned char* kbase = (const unsigned char*)(a.k + ((size_t)b * a.Hkv + g) * (size_t)a.max_len * D);
  const unsigned char* vtbase = (const unsigned char*)(a.vt + (size_t)bg * D * a.ld_vt);
  const int wu = __builtin_amdgcn_readfirstlane(wave);
  // Both tiles of keys [t0, t0+64) into stage st: K chunk-major (slot
  // c*64 + key; keys past the last position re-read that position), V^T
  // chunk-major (slot kc*D + dv holds stored keys t0+8kc .. t0+8kc+7 of dim
  // dv, in vt_key order).
  auto issue = [&](int t0, unsigned char* st) {
    issue_tile<CPR, kPfNW, kPfTK>(kbase, (size_t)D * 2, t0, top, st, wave, lane);
#pragma unroll
    for (int kk = 0; kk < kLoadsPerWave; ++kk) {
      const int ii = wu + kk * kPfNW;
      const int sl = ii * 64 + lane;
      const int kc = sl / D, dv = sl % D;
      dma16(vtbase + ((size_t)dv * a.ld_vt + t0 + 8 * kc) * 2, st + kKBytes + (size_t)ii * 1024);
    }
  };
  constexpr int kStage = 2 * kKBytes;
  constexpr float kRescale = 8.f;  // log2 units the running max may lag the row max

  // one tile: keys [t0, t0+64) in stage st; the next tile loads into st_next
  auto step = [&](int i, const unsigned char* st, unsigned char* st_next) {
    const int t0 = i * kPfTK;
    wait_vm<0>();   // this wave's part of tile i
    lds_barrier();  // every wave's part; every wave is done with tile i-1 (stage st_next)
    if (i + 1 < nt) issue(t0 + kPfTK, st_next);
    f32x4 s[2][4];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) s[rb][kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int t = 0; t < KS; ++t)
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        const bf16x8 kf =
            __builtin_bit_cast(bf16x8, *(const u32x4*)(st + (size_t)((KS * lg + t) * kPfTK + kb * 16 + l16) * 16));
#pragma unroll
        for (int rb = 0; rb < 2; ++rb) s[rb][kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[rb][t], s[rb][kb], 0, 0, 0);
      }
    if (t0 + kPfTK - 1 > pos0) {
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (t0 + kb * 16 + 4 * lg + e > prow[rb]) s[rb][kb][e] = -INFINITY;
    }
    if (win) {
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
        float cm = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int j = t0 + kb * 16 + 4 * lg + e;
            cm = fmaxf(cm, (j >= clo && j < chi) ? s[rb][kb][e] : -INFINITY);
          }
        cm = lanes4_max(cm);
        const float cn = fmaxf(mc[rb], cm * s2);
        if (cn != -INFINITY) {
          float z = 0.f;
#pragma unroll
          for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              // a select, not a branch: as a conditional sum the larger
              // exponent made the compiler branch per element
              const int j = t0 + kb * 16 + 4 * lg + e;
              const float xs = s[rb][kb][e];
              const float t = fast_exp2(fmaf(xs, s2lo, fmaf(xs, s2, -cn)));
              z += (j >= clo && j < chi) ? t : 0.f;
            }
          zc[rb] = fma(zc[rb], (double)fast_exp2(mc[rb] - cn), (double)z);
          mc[rb] = cn;
        }
      }
    }
    // Online softmax with a lazily moved reference: exponentials are taken
    // against m (<= the row max), and m moves up only when the row max
    // exceeds it by more than kRescale, so the weights stay below 2^kRescale
    // and O is rescaled on few tiles.  (m, sum 2^(y - m)) is a valid pair for
    // the row's statistics whatever m is.
    bool need[2];
    float mt[2];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      const f32x4* x = s[rb];
      const float a0 = fmaxf(fmaxf(x[0][0], x[0][1]), x[0][2]);
      const float a1 = fmaxf(fmaxf(x[0][3], x[1][0]), x[1][1]);
      const float a2 = fmaxf(fmaxf(x[1][2], x[1][3]), x[2][0]);
      const float a3 = fmaxf(fmaxf(x[2][1], x[2][2]), x[2][3]);
      const float a4 = fmaxf(fmaxf(x[3][0], x[3][1]), x[3][2]);
      float mx = fmaxf(fmaxf(fmaxf(a0, a1), a2), fmaxf(fmaxf(a3, a4), x[3][3]));
      mt[rb] = lanes4_max(mx) * s2;
      need[rb] = mt[rb] > m[rb] + kRescale;
    }
    if (wave_any(need[0] || need[1])) {
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
        const float mn = need[rb] ? mt[rb] : m[rb];
        const float alpha = need[rb] ? fast_exp2(m[rb] - mn) : 1.f;
        m[rb] = mn;
        ls[rb] *= (double)alpha;
#pragma unroll
        for (int d = 0; d < DVB; ++d) o[rb][d] *= alpha;
      }
    }
    bf16x8 pf[2][2];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      const float mu = m[rb] == -INFINITY ? 0.f : m[rb];  // rows with nothing visible yet
      float pe[4][4];
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int e = 0; e < 4; ++e) pe[kb][e] = fast_exp2(fmaf(s[rb][kb][e], s2, -mu));
      const float sum = (((pe[0][0] + pe[0][1]) + (pe[0][2] + pe[0][3])) + ((pe[1][0] + pe[1][1]) + (pe[1][2] + pe[1][3]))) +
                        (((pe[2][0] + pe[2][1]) + (pe[2][2] + pe[2][3])) + ((pe[3][0] + pe[3][1]) + (pe[3][2] + pe[3][3])));
      ls[rb] += (double)sum;
#pragma unroll
      for (int mm = 0; mm < 2; ++mm) {
        const u32x4 w4 = {pack_bf16x2(pe[2 * mm][0], pe[2 * mm][1]), pack_bf16x2(pe[2 * mm][2], pe[2 * mm][3]),
                          pack_bf16x2(pe[2 * mm + 1][0], pe[2 * mm + 1][1]),
                          pack_bf16x2(pe[2 * mm + 1][2], pe[2 * mm + 1][3])};
        pf[rb][mm] = __builtin_bit_cast(bf16x8, w4);
      }
    }
    const unsigned char* vst = st + kKBytes;
#pragma unroll
    for (int d = 0; d < DVB; ++d)
#pragma unroll
      for (int mm = 0; mm < 2; ++mm) {
        const bf16x8 vf =
            __builtin_bit_cast(bf16x8, *(const u32x4*)(vst + (size_t)((4 * mm + lg) * D + d * 16 + l16) * 16));
#pragma unroll
        for (int rb = 0; rb < 2; ++rb) o[rb][d] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf[rb][mm], o[rb][d], 0, 0, 0);
      }
  };

  wait_vm<0>();  // the query loads, before the waits below count tile loads
  issue(0, lds);
  // unrolled by two so that both stages are at fixed LDS addresses
  for (int i = 0; i < nt; i += 2) {
    step(i, lds, lds + kStage);
    if (i + 1 < nt) step(i + 1, lds + kStage, lds);
  }

  // ---- normalise and store; window rows: statistics and queries
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    double ld = ls[rb];
    ld += __shfl_xor(ld, 16);
    ld += __shfl_xor(ld, 32);
    double zd = zc[rb];
    zd += __shfl_xor(zd, 16);
    zd += __shfl_xor(zd, 32);
    const float l = (float)ld, zt = (float)zd;
    if (prow[rb] < 0) continue;
    const float inv = 1.f / l;
    const size_t row = ((size_t)b * a.Hq + (size_t)g * a.G + hl[rb]) * a.max_len + prow[rb];
    uint16_t* orow = a.out + row * D;
#pragma unroll
    for (int d = 0; d < DVB; ++d) {
      const u32x2 w2 = {pack_bf16x2(o[rb][d][0] * inv, o[rb][d][1] * inv), pack_bf16x2(o[rb][d][2] * inv, o[rb][d][3] * inv)};
      *(u32x2*)(orow + d * 16 + 4 * lg) = w2;
    }
    const int ii = prow[rb] - (L - a.w);
    if (win && ii >= 0) {
      const int rho = hl[rb] * a.w + ii;
      if (lg == 0)
        a.stats[(size_t)bg * a.rows_pad + rho] = make_float2(mc[rb], zt);
      uint16_t* qo = a.qobs + (((size_t)b * a.Hq + (size_t)g * a.G + hl[rb]) * a.w + ii) * D;
#pragma unroll
      for (int t = 0; t < KS; ++t) *(u32x4*)(qo + 8 * (KS * lg + t)) = __builtin_bit_cast(u32x4, qf[rb][t]);
    }
  }
  // rows of the score layout that no position fills: padding, and window rows
  // before position 0 when L < w
  if (a.want_stats && kblk == 0) {
    const int we = a.w < L ? a.w : L;
    for (int rho = tid(); rho < a.rows_pad; rho += nthreads()) {
      if (rho >= a.rows || rho % a.w < a.w - we) a.stats[(size_t)bg * a.rows_pad + rho] = make_float2(-INFINITY, 0.f);
    }
  }
}

// ============================================================ host side
static inline size_t align256p(size_t x) { return (x + 255) & ~(size_t)255; }

SNAP_DEBUG_READER(debug_flags_prefill)

Geometry prefill_geometry(const snap_params& p, int n_seq, int max_len) {
  Geometry g = compress_geometry(p, n_seq, max_len);
  size_t off = g.compress_bytes;
  g.off_qobs = off;
  off = align256p(off + (size_t)n_seq * p.n_q_heads * p.obs_window * p.d_qk * sizeof(uint16_t));
  g.ld_vt = (max_len + kPfTK - 1) / kPfTK * kPfTK;
  g.off_vt = off;
  off = align256p(off + (size_t)n_seq * p.n_kv_heads * p.d_v * (size_t)g.ld_vt * sizeof(uint16_t));
  g.prefill_bytes = off;
  return g;
}

snap_status launch_prefill_attn(const snap_params& p, int n_seq, const int32_t* lengths, int max_len, const void* q,
                                const void* k, const void* v, void* out, bool want_stats, void* ws,
                                hipStream_t stream) {
  const Geometry geo = prefill_geometry(p, n_seq, max_len);
  const int groups = n_seq * p.n_kv_heads;
  const int G = p.n_q_heads / p.n_kv_heads;
  const float scale = p.sm_scale > 0.f ? p.sm_scale : 1.0f / sqrtf((float)p.d_qk);
  unsigned char* w = (unsigned char*)ws;
  uint16_t* vt = (uint16_t*)(w + geo.off_vt);

  dim3 tgrid(geo.ld_vt / 64, groups);
  if (p.d_qk == 128)
    hipLaunchKernelGGL(vt_transpose<128>, tgrid, dim3(256), 0, stream, (const uint16_t*)v, vt, lengths, p.n_kv_heads,
                       max_len, geo.ld_vt);
  else
    hipLaunchKernelGGL(vt_transpose<64>, tgrid, dim3(256), 0, stream, (const uint16_t*)v, vt, lengths, p.n_kv_heads,
                       max_len, geo.ld_vt);
  if (hipGetLastError() != hipSuccess) return SNAP_ERR_HIP;

  PrefillArgs pa;
  pa.q = (const uint16_t*)q;
  pa.k = (const uint16_t*)k;
  pa.vt = vt;
  pa.out = (uint16_t*)out;
  pa.lengths = lengths;
  pa.stats = (float2*)(w + geo.off_stats);
  pa.qobs = (uint16_t*)(w + geo.off_qobs);
  pa.Hq = p.n_q_heads;
  pa.Hkv = p.n_kv_heads;
  pa.G = G;
  pa.max_len = max_len;
  pa.ld_vt = geo.ld_vt;
  pa.w = p.obs_window;
  pa.sink = p.sink;
  pa.recent = p.recent;
  pa.norm = p.norm;
  pa.rows = geo.rows;
  pa.rows_pad = geo.rows_pad;
  pa.want_stats = want_stats ? 1 : 0;
  pa.P = prefill_positions(G);
  split_scale2(scale, pa.scale2, pa.scale2_lo);
  pa.n_qblocks = (max_len + pa.P - 1) / pa.P;
  pa.groups = groups;
  dim3 grid(8 * ((groups + 7) / 8) * pa.n_qblocks);
  if (p.d_qk == 128)
    hipLaunchKernelGGL(prefill_attn<4>, grid, dim3(512), 0, stream, pa);
  else
    hipLaunchKernelGGL(prefill_attn<2>, grid, dim3(512), 0, stream, pa);
  if (hipGetLastError() != hipSuccess) return SNAP_ERR_HIP;
  return SNAP_OK;
}

snap_status launch_prefill(const snap_params& p, const snap_cache& c, int32_t* pos, int32_t* n_topk, int n_seq,
                           const int32_t* slot_ids, const int32_t* lengths, int max_len, const void* q, const void* k,
                           const void* v, void* out, int32_t* sel_out, float* pooled_out, void* ws,
                           hipStream_t stream) {
  const bool select = p.topk > 0 || pooled_out;
  snap_status st = launch_prefill_attn(p, n_seq, lengths, max_len, q, k, v, out, select, ws, stream);
  if (st != SNAP_OK) return st;
  const Geometry geo = prefill_geometry(p, n_seq, max_len);
  return launch_compress(p, c, pos, n_topk, n_seq, slot_ids, lengths, max_len, (unsigned char*)ws + geo.off_qobs, k,
                         v, sel_out, pooled_out, ws, stream, /*stats_given=*/true);
}

}  // namespace snap
