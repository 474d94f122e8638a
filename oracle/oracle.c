/*
 * oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, fp64 CPU implementation of the SnapStream hot path
 * (arXiv 2511.03092): SnapKV selection at the end of prefill, the
 * StreamingLLM sink + ring-buffer cache, and decode attention over the
 * fixed-size compressed cache.  It exists so the HIP library can be checked
 * against something written straight from the paper.  Only tests/, the smoke
 * check and the benchmark's CPU-baseline leg may load it; the product path
 * never does.  It shares no code with the HIP library.
 *
 * Conventions (all 0-based token positions 0..L-1):
 *   s = sink length, r = recent (ring) length >= 1, K = top-K length,
 *   budget B = s + r + K, w = observation window, kp = pool kernel (odd),
 *   G = query heads per KV head.
 *   Candidates C = [s, L-r): every prompt token that is neither a sink nor in
 *   the recent window (Sec. III, "the remaining L-(L_sink+L_recent) tokens";
 *   Sec. III-B.2 defines K_evict as exactly these keys).
 *
 * Each function cites the passage it follows.  Where the paper is ambiguous
 * the reading taken is stated next to the code.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define POOL_MAX 0
#define POOL_AVG 1
#define NORM_CAND 0 /* softmax normaliser over the eviction candidates (Eq. 3) */
#define NORM_ROW 1  /* softmax normaliser over the whole causal row */

/* Cache row of token position p (Sec. III-C, Eq. for L_rb, plus the p < L_sink
 * branch of the decode update): sinks are stored in place, every later token
 * goes to the ring slot s + ((p - s) mod r).  For p >= s this equals
 * (p - s + r) mod r + s, the paper's closed form. */
int oracle_slot_of(int64_t p, int s, int r) {
  if (p < s) return (int)p;
  return s + (int)((p - s) % r);
}

/* Number of real (non-padding) rows in the top-K region: the candidates that
 * exist, capped at K (Sec. III-B.2 padding metadata; the prefill listing's
 * valid_topk). */
int oracle_n_topk(int64_t L, int s, int r, int K) {
  int64_t n = L - (int64_t)s - (int64_t)r;
  if (n < 0) n = 0;
  return (int)(n < K ? n : K);
}

/* Eq. 1 with W from Eq. 3: summed attention of the observation window onto
 * the candidates of ONE KV-head group.
 *
 *   q : [G][w][D]   query rows of the group's G heads; row ii is position
 *                   L - w + ii (row w-1 is the last prompt token).  Rows with a
 *                   negative position (L < w) do not exist and are skipped.
 *   k : [L][D]      keys of the group.
 *   A : [L]         output; A[j] for j in C, 0 elsewhere.
 *
 * For window row i the logits are z_j = sm_scale * <q_i, k_j>; the softmax
 * normaliser runs over N_i = C intersect [0, i] (NORM_CAND, Eq. 3) or over the
 * causal row [0, i] (NORM_ROW).  W_ij = exp(z_j - m_i) / Z_i for j in C, j <= i
 * (causal), and A[j] = sum over the G heads and the window rows of W_ij: one
 * index set per KV head, so the group's heads are summed (Eq. 1 sums over the
 * window; the GQA group sum is this implementation's reading).            */
void oracle_window_scores(int G, int w, int D, int64_t L, int s, int r, int norm,
                          double sm_scale, const double* q, const double* k,
                          double* A) {
  int64_t c0 = s, c1 = L - r; /* candidates [c0, c1) */
  for (int64_t j = 0; j < L; ++j) A[j] = 0.0;
  if (c1 <= c0) return;
  double* z = (double*)malloc(sizeof(double) * (size_t)L);
  int we = (int)(L < w ? L : w);
  for (int h = 0; h < G; ++h) {
    for (int ii = w - we; ii < w; ++ii) {
      int64_t i = L - w + ii; /* absolute position of this window row */
      const double* qi = q + ((size_t)h * w + ii) * D;
      int64_t lo = (norm == NORM_CAND) ? c0 : 0;
      int64_t hi = (norm == NORM_CAND) ? (c1 - 1 < i ? c1 - 1 : i) : i; /* inclusive */
      if (hi < lo) continue; /* empty normaliser domain: the row adds nothing */
      double m = -INFINITY;
      for (int64_t j = lo; j <= hi; ++j) {
        double acc = 0.0;
        const double* kj = k + (size_t)j * D;
        for (int d = 0; d < D; ++d) acc += qi[d] * kj[d];
        z[j] = sm_scale * acc;
        if (z[j] > m) m = z[j];
      }
      double Z = 0.0;
      for (int64_t j = lo; j <= hi; ++j) Z += exp(z[j] - m);
      int64_t jc_hi = (c1 - 1 < i ? c1 - 1 : i);
      for (int64_t j = c0; j <= jc_hi; ++j) A[j] += exp(z[j] - m) / Z;
    }
  }
  free(z);
}

/* Eq. 2's 1-D pooling, stride 1, padding kp/2, restricted to the candidates
 * (the prefill SnapKV routine pools then slices; here the pool window only
 * sees candidates, so sink and recent scores never leak in).
 * MAX: P[j] = max A[t] over t in C with |t-j| <= kp/2.
 * AVG: P[j] = (1/kp) * sum of the same A[t] (zero padding, fixed divisor). */
void oracle_pool(int64_t L, int s, int r, int kp, int pool, const double* A,
                 double* P) {
  int64_t c0 = s, c1 = L - r;
  int half = kp / 2;
  for (int64_t j = 0; j < L; ++j) P[j] = 0.0;
  for (int64_t j = c0; j < c1; ++j) {
    double acc = (pool == POOL_MAX) ? -INFINITY : 0.0;
    for (int64_t t = j - half; t <= j + half; ++t) {
      if (t < c0 || t >= c1) continue;
      if (pool == POOL_MAX) {
        if (A[t] > acc) acc = A[t];
      } else {
        acc += A[t];
      }
    }
    P[j] = (pool == POOL_MAX) ? acc : acc / (double)kp;
  }
}

/* A candidate and its pooled score, so the ranking comparator needs no state
 * outside its arguments (the oracle runs units on several threads at once). */
typedef struct {
  double p;
  int64_t t;
} ranked;
static int cmp_rank(const void* a, const void* b) {
  const ranked* x = (const ranked*)a;
  const ranked* y = (const ranked*)b;
  if (x->p > y->p) return -1; /* larger pooled score first */
  if (x->p < y->p) return 1;
  return (x->t < y->t) ? -1 : (x->t > y->t); /* equal scores: lower token index first */
}
static int cmp_i64(const void* a, const void* b) {
  int64_t x = *(const int64_t*)a, y = *(const int64_t*)b;
  return (x < y) ? -1 : (x > y);
}

/* Eq. 2's Top_K over the pooled candidate scores.  Candidates are ranked by
 * (P descending, token index ascending) and the first min(K, |C|) kept; the
 * kept set is returned in ascending token order (the paper's top-k returns
 * value order, which does not change attention; ascending order makes the
 * cache bytes canonical).  Returns the count kept. */
int oracle_topk(int64_t L, int s, int r, int K, const double* P, int32_t* sel) {
  int64_t c0 = s, c1 = L - r;
  int64_t n = c1 - c0;
  if (n <= 0 || K <= 0) return 0;
  ranked* rk = (ranked*)malloc(sizeof(ranked) * (size_t)n);
  for (int64_t t = 0; t < n; ++t) {
    rk[t].p = P[c0 + t];
    rk[t].t = c0 + t;
  }
  qsort(rk, (size_t)n, sizeof(ranked), cmp_rank);
  int keff = (int)(n < K ? n : K);
  int64_t* idx = (int64_t*)malloc(sizeof(int64_t) * (size_t)keff);
  for (int m = 0; m < keff; ++m) idx[m] = rk[m].t;
  qsort(idx, (size_t)keff, sizeof(int64_t), cmp_i64);
  for (int m = 0; m < keff; ++m) sel[m] = (int32_t)idx[m];
  free(idx);
  free(rk);
  return keff;
}

/* Compressed cache of one group (Sec. III-A, both cases; Sec. III-B.1).
 *   rows [0, min(s, L))        <- tokens 0.. (attention sinks)
 *   token t in [max(s, L-r), L) -> row oracle_slot_of(t) (the ring; the last
 *                                  r prompt tokens, placed where the decode
 *                                  update will later find them)
 *   row s + r + m              <- token sel[m] for m < keff (top-K region)
 *   every other row            <- 0 (padding)
 * x : [L][width] input rows; out : [B][width]. */
void oracle_assemble(int64_t L, int s, int r, int K, int width, const double* x,
                     const int32_t* sel, int keff, double* out) {
  int B = s + r + K;
  memset(out, 0, sizeof(double) * (size_t)B * (size_t)width);
  for (int64_t t = 0; t < L && t < s; ++t)
    memcpy(out + (size_t)t * width, x + (size_t)t * width, sizeof(double) * (size_t)width);
  int64_t lo = L - r > s ? L - r : s;
  for (int64_t t = lo; t < L; ++t) {
    int row = oracle_slot_of(t, s, r);
    memcpy(out + (size_t)row * width, x + (size_t)t * width, sizeof(double) * (size_t)width);
  }
  for (int m = 0; m < keff; ++m)
    memcpy(out + (size_t)(s + r + m) * width, x + (size_t)sel[m] * width,
           sizeof(double) * (size_t)width);
}

/* Whole compression of one (sequence, KV-head group): Eq. 3 -> Eq. 1 ->
 * Eq. 2 -> gather into the sink/ring/top-K cache.  kv_width is the stored
 * row width of K; v may be NULL when V is the first dv dims of each K row
 * (latent caches, Sec. VI: the low-rank latents are what is compressed).
 * Writes A, P (length L), sel (length K, -1 padded), cache_k [B][dk],
 * cache_v [B][dv] (skipped when v == NULL).  Returns the number of real
 * top-K rows. */
int oracle_compress_group(int G, int w, int dk, int dv, int64_t L, int s, int r,
                          int K, int kp, int pool, int norm, double sm_scale,
                          const double* q, const double* k, const double* v,
                          double* A, double* P, int32_t* sel, double* cache_k,
                          double* cache_v) {
  oracle_window_scores(G, w, dk, L, s, r, norm, sm_scale, q, k, A);
  oracle_pool(L, s, r, kp, pool, A, P);
  for (int m = 0; m < K; ++m) sel[m] = -1;
  int keff = oracle_topk(L, s, r, K, P, sel);
  oracle_assemble(L, s, r, K, dk, k, sel, keff, cache_k);
  if (v) oracle_assemble(L, s, r, K, dv, v, sel, keff, cache_v);
  return keff;
}

/* Decode attention of one KV-head group over its compressed cache, after the
 * token at position p has been written to row oracle_slot_of(p).
 * Valid rows: [0, min(p+1, s+r)) -- sinks and ring filled so far -- and the
 * n_topk real rows [s+r, s+r+n_topk) (the padding rows are masked, Sec.
 * III-B.2).  For each of the G heads: out = sum_j softmax_j(sm_scale q.k_j) v_j.
 *   q : [G][dk], ck : [B][ck_width] (keys = first dk dims), cv : [B][cv_width]
 *   (values = first dv dims; pass cv = ck for a latent cache), out : [G][dv]. */
void oracle_decode_attn(int G, int dk, int dv, int ck_width, int cv_width, int s,
                        int r, int64_t p, int n_topk, double sm_scale,
                        const double* q, const double* ck, const double* cv,
                        double* out) {
  int B = s + r + n_topk; /* rows beyond this are never read */
  int n1 = (int)((p + 1) < (int64_t)(s + r) ? (p + 1) : (int64_t)(s + r));
  double* z = (double*)malloc(sizeof(double) * (size_t)(B > 0 ? B : 1));
  for (int h = 0; h < G; ++h) {
    const double* qh = q + (size_t)h * dk;
    double m = -INFINITY;
    for (int j = 0; j < B; ++j) {
      int valid = (j < n1) || (j >= s + r && j < s + r + n_topk);
      if (!valid) continue;
      double acc = 0.0;
      for (int d = 0; d < dk; ++d) acc += qh[d] * ck[(size_t)j * ck_width + d];
      z[j] = sm_scale * acc;
      if (z[j] > m) m = z[j];
    }
    double Z = 0.0;
    double* oh = out + (size_t)h * dv;
    for (int d = 0; d < dv; ++d) oh[d] = 0.0;
    for (int j = 0; j < B; ++j) {
      int valid = (j < n1) || (j >= s + r && j < s + r + n_topk);
      if (!valid) continue;
      double e = exp(z[j] - m);
      Z += e;
      for (int d = 0; d < dv; ++d) oh[d] += e * cv[(size_t)j * cv_width + d];
    }
    for (int d = 0; d < dv; ++d) oh[d] /= Z;
  }
  free(z);
}

/* Causal self-attention over the whole prompt for one KV-head group: the
 * attention step of the prefill graph (Sec. IV-A, the MHA kernel that fuses
 * Q K^T, softmax and P V), whose last w query rows are the observation window
 * of Sec. III-B.2.  For each of the G query heads h and every position i in
 * [i0, i1) (0 <= i0 <= i1 <= L):
 *   out[h][i - i0] = sum_{j <= i} softmax_j(sm_scale q_{h,i}.k_j) v_j.
 * If lse is not NULL, lse[h][i - i0] = log sum_{j <= i} exp(sm_scale q_{h,i}.k_j)
 * (the row's natural-log normaliser).
 *   q : [G][L][dk], k : [L][dk], v : [L][dv], out : [G][i1-i0][dv],
 *   lse : [G][i1-i0]. */
void oracle_prefill_attn(int G, int dk, int dv, int64_t L, int64_t i0, int64_t i1,
                         double sm_scale, const double* q, const double* k,
                         const double* v, double* out, double* lse) {
  int64_t n = i1 - i0;
  double* z = (double*)malloc(sizeof(double) * (size_t)(L > 0 ? L : 1));
  for (int h = 0; h < G; ++h) {
    for (int64_t i = i0; i < i1; ++i) {
      const double* qi = q + ((size_t)h * L + i) * dk;
      double m = -INFINITY;
      for (int64_t j = 0; j <= i; ++j) {
        double acc = 0.0;
        for (int d = 0; d < dk; ++d) acc += qi[d] * k[(size_t)j * dk + d];
        z[j] = sm_scale * acc;
        if (z[j] > m) m = z[j];
      }
      double Z = 0.0;
      double* oi = out + ((size_t)h * n + (i - i0)) * dv;
      for (int d = 0; d < dv; ++d) oi[d] = 0.0;
      for (int64_t j = 0; j <= i; ++j) {
        double e = exp(z[j] - m);
        Z += e;
        for (int d = 0; d < dv; ++d) oi[d] += e * v[(size_t)j * dv + d];
      }
      for (int d = 0; d < dv; ++d) oi[d] /= Z;
      if (lse) lse[(size_t)h * n + (i - i0)] = m + log(Z);
    }
  }
  free(z);
}

/* ---- fp8 storage (OCP E4M3 "fn": 1 sign, 4 exponent bits with bias 7, 3
 * mantissa bits, no infinities, 0x7F/0xFF = NaN, largest finite 448). ----
 * Written from the format definition, not from any library. */

/* Exact value of an E4M3 code. */
double oracle_e4m3_value(uint8_t code) {
  int sign = code >> 7, e = (code >> 3) & 0xF, m = code & 7;
  if (e == 0xF && m == 7) return NAN;
  double mag = (e == 0) ? ldexp((double)m, -9) /* subnormal: m * 2^-6 / 8 */
                        : ldexp(1.0 + m / 8.0, e - 7);
  return sign ? -mag : mag;
}

/* Round-to-nearest-even, saturating encode of an fp32 value: the code whose
 * value is nearest to v (ties to the even mantissa), values beyond +-448 clamp
 * to +-448, NaN maps to 0x7F. */
uint8_t oracle_e4m3_encode(float v) {
  if (v != v) return 0x7F;
  uint8_t sign = (v < 0.0f || (v == 0.0f && signbit(v))) ? 0x80 : 0;
  double a = fabs((double)v);
  if (a >= 448.0) return sign | 0x7E;
  /* brute force over the 127 non-negative finite codes: nearest value,
   * ties broken toward the even code (even mantissa LSB). */
  int best = 0;
  double bestd = INFINITY;
  for (int c = 0; c < 0x7F; ++c) {
    double d = fabs(oracle_e4m3_value((uint8_t)c) - a);
    if (d < bestd || (d == bestd && (c & 1) == 0)) {
      bestd = d;
      best = c;
    }
  }
  return sign | (uint8_t)best;
}

/* A scale chosen from the data (not from the paper, which keeps bf16 caches):
 * the largest magnitude among n values divided by 448, the largest E4M3
 * magnitude, so that value maps to the top code and nothing saturates; 1 when
 * every value is zero.  The division is an fp32 one, as a device computes it. */
float oracle_fp8_scale(const double* x, int64_t n) {
  double amax = 0.0;
  for (int64_t i = 0; i < n; ++i) {
    double a = fabs(x[i]);
    if (a > amax) amax = a;
  }
  if (amax == 0.0) return 1.0f;
  float af = (float)amax;
  return af / 448.0f;
}

/* Quantise n values with one scale, deciding each code in fp32 the way a
 * device kernel does: the fp32 quotient x / scale, then the encode above. */
void oracle_quantize(const double* x, int64_t n, float scale, uint8_t* codes) {
  for (int64_t i = 0; i < n; ++i) {
    float xf = (float)x[i];
    float qv = xf / scale;
    codes[i] = oracle_e4m3_encode(qv);
  }
}
