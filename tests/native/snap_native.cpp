// A native caller of the C ABI: one GQA layer with a bf16 cache, driven from
// C++ with the HIP runtime alone (no Python, no torch).  snap_compress of a
// seeded prompt is checked against the fp64 oracle (liboracle, test
// infrastructure): the kept set against the oracle's pooled scores (every
// kept candidate at or above the K-th largest score, every dropped one at or
// below it, to a relative 1e-6 for fp32 rounding) and the cache bytes against
// the oracle's assembly of that set.  Decode steps (snap_decode_step +
// snap_advance) follow, each output checked against the oracle's attention
// over the cache bytes the library wrote, and each appended row against the
// input at the oracle's ring row.
// Built by tests/native/build.py, run by tests/test_gpu_native.py; prints
// "NATIVE OK" and exits 0 when every check holds.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <functional>
#include <vector>

#include "snapstream.h"

extern "C" {
int oracle_slot_of(int64_t p, int s, int r);
int oracle_topk(int64_t L, int s, int r, int K, const double* P, int32_t* sel);
void oracle_assemble(int64_t L, int s, int r, int K, int width, const double* x, const int32_t* sel, int keff,
                     double* out);
int oracle_compress_group(int G, int w, int dk, int dv, int64_t L, int s, int r, int K, int kp, int pool, int norm,
                          double sm_scale, const double* q, const double* k, const double* v, double* A, double* P,
                          int32_t* sel, double* cache_k, double* cache_v);
void oracle_decode_attn(int G, int dk, int dv, int ck_width, int cv_width, int s, int r, int64_t p, int n_topk,
                        double sm_scale, const double* q, const double* ck, const double* cv, double* out);
}

#define HIP_OK(x)                                                             \
  do {                                                                        \
    hipError_t e_ = (x);                                                      \
    if (e_ != hipSuccess) {                                                   \
      std::fprintf(stderr, "%s: %s\n", #x, hipGetErrorString(e_));            \
      return 2;                                                               \
    }                                                                         \
  } while (0)
#define SNAP_OK_(x)                                                                     \
  do {                                                                                  \
    snap_status s_ = (x);                                                               \
    if (s_ != SNAP_OK) {                                                                \
      std::fprintf(stderr, "%s: %s (%s)\n", #x, snap_status_str(s_), snap_last_error()); \
      return 2;                                                                         \
    }                                                                                   \
  } while (0)

// seeded inputs: splitmix64 -> uniform -> normal (Box-Muller) -> bf16 bits
static uint64_t g_state = 0x2511030920251202ull;
static uint64_t next_u64() {
  uint64_t z = (g_state += 0x9e3779b97f4a7c15ull);
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}
static double next_normal() {
  const double u1 = ((next_u64() >> 11) + 0.5) * (1.0 / 9007199254740992.0);
  const double u2 = ((next_u64() >> 11) + 0.5) * (1.0 / 9007199254740992.0);
  return std::sqrt(-2.0 * std::log(u1)) * std::cos(6.283185307179586 * u2);
}
static uint16_t to_bf16(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
static double from_bf16(uint16_t h) {
  const uint32_t u = (uint32_t)h << 16;
  float f;
  std::memcpy(&f, &u, 4);
  return f;
}
static std::vector<uint16_t> normals(size_t n) {
  std::vector<uint16_t> v(n);
  for (auto& x : v) x = to_bf16((float)next_normal());
  return v;
}

int main() {
  const int Hq = 8, Hkv = 2, G = Hq / Hkv, D = 128, sink = 4, recent = 64, topk = 200, w = 16;
  const int L = 1500, steps = 80;  // the ring of 64 rows wraps
  snap_params p;
  std::memset(&p, 0, sizeof(p));
  p.n_q_heads = Hq;
  p.n_kv_heads = Hkv;
  p.d_qk = D;
  p.d_v = D;
  p.sink = sink;
  p.recent = recent;
  p.topk = topk;
  p.obs_window = w;
  p.pool_kernel = 7;
  p.pool = SNAP_POOL_MAX;
  p.norm = SNAP_NORM_CAND;
  p.in_dtype = SNAP_BF16;
  p.kv_dtype = SNAP_BF16;
  p.kv_reuse = SNAP_KV_AUTO;
  const int B = sink + recent + topk;

  // prompt: window queries [1][Hq][w][D], keys / values [1][Hkv][L][D]
  auto hq = normals((size_t)Hq * w * D), hk = normals((size_t)Hkv * L * D), hv = normals((size_t)Hkv * L * D);
  void *dq, *dk, *dv, *ck, *cv, *ws, *wsd, *dqd, *dkn, *dvn, *dout;
  int32_t *dpos, *dntop, *dslot, *dlen, *dsel;
  HIP_OK(hipMalloc(&dq, hq.size() * 2));
  HIP_OK(hipMalloc(&dk, hk.size() * 2));
  HIP_OK(hipMalloc(&dv, hv.size() * 2));
  HIP_OK(hipMalloc(&ck, (size_t)Hkv * B * D * 2));
  HIP_OK(hipMalloc(&cv, (size_t)Hkv * B * D * 2));
  HIP_OK(hipMemset(ck, 0, (size_t)Hkv * B * D * 2));
  HIP_OK(hipMemset(cv, 0, (size_t)Hkv * B * D * 2));
  HIP_OK(hipMalloc(&dpos, 4));
  HIP_OK(hipMalloc(&dntop, 4));
  HIP_OK(hipMalloc(&dslot, 4));
  HIP_OK(hipMalloc(&dlen, 4));
  HIP_OK(hipMalloc(&dsel, (size_t)Hkv * topk * 4));
  const int32_t zero = 0, len = L;
  HIP_OK(hipMemcpy(dslot, &zero, 4, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(dlen, &len, 4, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(dq, hq.data(), hq.size() * 2, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(dk, hk.data(), hk.size() * 2, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(dv, hv.data(), hv.size() * 2, hipMemcpyHostToDevice));
  const size_t wsb = snap_compress_workspace(&p, 1, L), wsdb = snap_decode_workspace(&p, 1);
  if (!wsb || !wsdb) return 2;
  HIP_OK(hipMalloc(&ws, wsb));
  HIP_OK(hipMalloc(&wsd, wsdb));
  snap_cache c = {ck, cv, nullptr, nullptr, 1};
  SNAP_OK_(snap_compress(&p, &c, dpos, dntop, 1, dslot, dlen, L, dq, dk, dv, dsel, nullptr, ws, wsb, nullptr));
  HIP_OK(hipDeviceSynchronize());
  int32_t pos = 0, ntop = 0;
  HIP_OK(hipMemcpy(&pos, dpos, 4, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(&ntop, dntop, 4, hipMemcpyDeviceToHost));
  const int keff = std::min(std::max(L - sink - recent, 0), topk);
  if (pos != L || ntop != keff) {
    std::fprintf(stderr, "metadata: pos %d (want %d), n_topk %d (want %d)\n", pos, L, ntop, keff);
    return 1;
  }

  std::vector<uint16_t> hck((size_t)Hkv * B * D), hcv((size_t)Hkv * B * D), hout((size_t)Hq * D);
  std::vector<int32_t> gsel((size_t)Hkv * topk), osel(topk);
  HIP_OK(hipMemcpy(gsel.data(), dsel, gsel.size() * 4, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(hck.data(), ck, hck.size() * 2, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(hcv.data(), cv, hcv.size() * 2, hipMemcpyDeviceToHost));
  {
    const double sm = 1.0 / std::sqrt((double)D), tol = 1e-6;
    std::vector<double> qg((size_t)G * w * D), kg((size_t)L * D), vg((size_t)L * D), A(L), P(L);
    std::vector<double> oc((size_t)B * D), ov((size_t)B * D), ek((size_t)B * D), ev((size_t)B * D);
    int swaps = 0;
    for (int g = 0; g < Hkv; ++g) {
      for (size_t i = 0; i < qg.size(); ++i) qg[i] = from_bf16(hq[(size_t)g * G * w * D + i]);
      for (size_t i = 0; i < kg.size(); ++i) kg[i] = from_bf16(hk[(size_t)g * L * D + i]);
      for (size_t i = 0; i < vg.size(); ++i) vg[i] = from_bf16(hv[(size_t)g * L * D + i]);
      const int ok = oracle_compress_group(G, w, D, D, L, sink, recent, topk, p.pool_kernel, SNAP_POOL_MAX,
                                           SNAP_NORM_CAND, sm, qg.data(), kg.data(), vg.data(), A.data(), P.data(),
                                           osel.data(), oc.data(), ov.data());
      const int32_t* s_ = &gsel[(size_t)g * topk];
      if (ok != keff) return 1;
      std::vector<double> cand(P.begin() + sink, P.begin() + (L - recent));
      std::nth_element(cand.begin(), cand.begin() + (keff - 1), cand.end(), std::greater<double>());
      const double tau = cand[keff - 1];
      std::vector<char> kept(L, 0);
      for (int m = 0; m < topk; ++m) {
        if (m >= keff) {
          if (s_[m] != -1) return std::fprintf(stderr, "head %d: sel padding\n", g), 1;
          continue;
        }
        if (s_[m] < sink || s_[m] >= L - recent || (m && s_[m] <= s_[m - 1]))
          return std::fprintf(stderr, "head %d: sel[%d] = %d not an ascending candidate\n", g, m, s_[m]), 1;
        if (P[s_[m]] < tau * (1 - tol))
          return std::fprintf(stderr, "head %d: kept %d below the threshold\n", g, s_[m]), 1;
        kept[s_[m]] = 1;
      }
      for (int t = sink; t < L - recent; ++t)
        if (!kept[t] && P[t] > tau * (1 + tol))
          return std::fprintf(stderr, "head %d: dropped %d above the threshold\n", g, t), 1;
      for (int m = 0; m < keff; ++m) swaps += !kept[osel[m]];
      // the cache holds the oracle's assembly of the kept set, byte for byte
      oracle_assemble(L, sink, recent, topk, D, kg.data(), s_, keff, ek.data());
      oracle_assemble(L, sink, recent, topk, D, vg.data(), s_, keff, ev.data());
      for (size_t i = 0; i < (size_t)B * D; ++i)
        if (from_bf16(hck[(size_t)g * B * D + i]) != ek[i] || from_bf16(hcv[(size_t)g * B * D + i]) != ev[i])
          return std::fprintf(stderr, "head %d: cache element %zu differs from the oracle's assembly\n", g, i), 1;
    }
    std::printf("compress: L %d, kept %d per head, %d near-tie swaps vs the oracle\n", L, keff, swaps);
  }

  HIP_OK(hipMalloc(&dqd, (size_t)Hq * D * 2));
  HIP_OK(hipMalloc(&dkn, (size_t)Hkv * D * 2));
  HIP_OK(hipMalloc(&dvn, (size_t)Hkv * D * 2));
  HIP_OK(hipMalloc(&dout, (size_t)Hq * D * 2));
  std::vector<double> qd(Hq * D), ckd((size_t)B * D), cvd((size_t)B * D), ref(G * D);
  double worst = 0.0;
  for (int t = 0; t < steps; ++t) {
    auto q = normals((size_t)Hq * D), kn = normals((size_t)Hkv * D), vn = normals((size_t)Hkv * D);
    HIP_OK(hipMemcpy(dqd, q.data(), q.size() * 2, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(dkn, kn.data(), kn.size() * 2, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(dvn, vn.data(), vn.size() * 2, hipMemcpyHostToDevice));
    SNAP_OK_(snap_decode_step(&p, &c, dpos, dntop, 1, dslot, dqd, dkn, dvn, dout, SNAP_BF16, wsd, wsdb, nullptr));
    HIP_OK(hipDeviceSynchronize());
    HIP_OK(hipMemcpy(hck.data(), ck, hck.size() * 2, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(hcv.data(), cv, hcv.size() * 2, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(hout.data(), dout, hout.size() * 2, hipMemcpyDeviceToHost));
    const int64_t pt = L + t;
    const int row = oracle_slot_of(pt, sink, recent);
    for (int g = 0; g < Hkv; ++g) {
      // the appended row holds the input bytes
      if (std::memcmp(&hck[((size_t)g * B + row) * D], &kn[(size_t)g * D], D * 2) ||
          std::memcmp(&hcv[((size_t)g * B + row) * D], &vn[(size_t)g * D], D * 2)) {
        std::fprintf(stderr, "step %d head %d: appended row %d differs from the input\n", t, g, row);
        return 1;
      }
      for (size_t i = 0; i < (size_t)B * D; ++i) {
        ckd[i] = from_bf16(hck[(size_t)g * B * D + i]);
        cvd[i] = from_bf16(hcv[(size_t)g * B * D + i]);
      }
      for (int i = 0; i < G * D; ++i) qd[i] = from_bf16(q[(size_t)g * G * D + i]);
      oracle_decode_attn(G, D, D, D, D, sink, recent, pt, ntop, 1.0 / std::sqrt((double)D), qd.data(), ckd.data(),
                         cvd.data(), ref.data());
      for (int i = 0; i < G * D; ++i) {
        const double e = std::fabs(from_bf16(hout[(size_t)g * G * D + i]) - ref[i]);
        worst = e > worst ? e : worst;
      }
    }
    SNAP_OK_(snap_advance(dpos, 1, 1, dslot, nullptr));
  }
  HIP_OK(hipDeviceSynchronize());
  std::printf("decode steps %d, max abs err vs the oracle %.3e\n", steps, worst);
  if (!(worst <= 2e-2)) return 1;
  std::printf("NATIVE OK\n");
  return 0;
}
