// lds_dma.h -- direct global->LDS tile loads (global_load_lds_dwordx4, no
// VGPR staging), explicit vmcnt waits and an LDS-only workgroup barrier,
// shared by the score passes and the prefill attention kernel.  gfx950 only.
#pragma once

#include "snap_internal.h"

namespace snap {

// LDS tile of TK keys (64, or 32 for 576-wide rows) stored chunk-major: the
// 16-byte chunk c of key k sits at slot c*TK + k.  A fragment read by 16
// consecutive keys of one chunk is 256 contiguous bytes, and every tile load
// instruction covers 64 consecutive slots (lane i -> slot base + i).  (A
// row-major tile with a swizzled chunk index, whose loads read contiguous
// memory, measured slower for both row widths.)
template <int TK>
__device__ __forceinline__ int tile_slot(int key, int c) { return c * TK + key; }

typedef __attribute__((address_space(3))) void* lds_void_ptr;

// One wave-instruction of global -> LDS copy: lane i's 16 bytes at g land at
// LDS byte lds_wave_base + 16*i.  Issued through inline asm so that the only
// ordering with later LDS reads is the explicit vmcnt wait + barrier of the
// caller (the compiler's own LDS-DMA tracking would otherwise wait for every
// tile in flight).  M0 (the LDS base of the DMA) is saved and restored, with
// the one wait state an M0 write needs before an LDS DMA.
__device__ __forceinline__ void dma16(const void* g, const void* lds_wave_base) {
  // wave-uniform by construction; readfirstlane keeps it in a scalar register
  // whatever the compiler's uniformity analysis concludes
  const uint32_t la = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_void_ptr)lds_wave_base);
  uint32_t saved;
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

// Issue this wave's share of one key tile: the tile is CPR*TK/64
// wave-instructions, each moving 64 x 16 bytes straight into LDS (no VGPRs);
// wave w issues instructions w, w+NW, ...  Keys past c1 read key c1-1
// instead, so a wave always issues the same number of loads per tile (those
// bytes are never used).
template <int CPR, int NW, int TK>
__device__ __forceinline__ void issue_tile(const unsigned char* kbase, size_t row_bytes, int t0, int c1,
                                           unsigned char* buf, int wave, int lane) {
  constexpr int NI = CPR * TK / 64;
  constexpr int KMAX = (NI + NW - 1) / NW;  // loads of the busiest wave
  static_assert(CPR * TK % 64 == 0, "a tile is a whole number of wave-instructions");
  const int w = __builtin_amdgcn_readfirstlane(wave);
  if constexpr (TK == 64) {
    // one key per lane: a single row pointer, chunk c = instruction index
    int j = t0 + lane;
    j = j < c1 ? j : c1 - 1;
    const unsigned char* rowp = kbase + (size_t)j * row_bytes;
#pragma unroll
    for (int k = 0; k < KMAX; ++k) {
      const int c = w + k * NW;
      if (NI % NW != 0 && c >= NI) break;  // wave-uniform
      dma16(rowp + c * 16, buf + (size_t)c * 1024);
    }
  } else {
    // 64 / TK chunks per instruction: lane -> (chunk, key)
    const unsigned ul = (unsigned)lane;
#pragma unroll
    for (int k = 0; k < KMAX; ++k) {
      const int ii = w + k * NW;
      if (NI % NW != 0 && ii >= NI) break;  // wave-uniform
      const unsigned slot = (unsigned)ii * 64u + ul;
      const int c = (int)(slot / TK), key = (int)(slot % TK);
      int j = t0 + key;
      j = j < c1 ? j : c1 - 1;
      dma16(kbase + (size_t)j * row_bytes + c * 16, buf + (size_t)ii * 1024);
    }
  }
}
// this wave's loads per tile
template <int CPR, int NW, int TK>
__device__ __forceinline__ int tile_loads(int wave) {
  constexpr int NI = CPR * TK / 64;
  return (NI - wave + NW - 1) / NW;
}

// Wait until at most N vector-memory operations of this wave are in flight.
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N < 64, "vmcnt field");
  // gfx9 s_waitcnt: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt_hi[15:14]
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}
// vmcnt <= n for a wave-uniform n (a switch over the encodings; n > 24
// falls back to waiting for everything, which is always safe)
__device__ __forceinline__ void wait_vm_dyn(int n) {
  switch (n) {
#define SNAP_WAIT_CASE(N) \
  case N:                 \
    wait_vm<N>();         \
    break;
    SNAP_WAIT_CASE(0) SNAP_WAIT_CASE(1) SNAP_WAIT_CASE(2) SNAP_WAIT_CASE(3) SNAP_WAIT_CASE(4)
    SNAP_WAIT_CASE(5) SNAP_WAIT_CASE(6) SNAP_WAIT_CASE(7) SNAP_WAIT_CASE(8) SNAP_WAIT_CASE(9)
    SNAP_WAIT_CASE(10) SNAP_WAIT_CASE(11) SNAP_WAIT_CASE(12) SNAP_WAIT_CASE(13) SNAP_WAIT_CASE(14)
    SNAP_WAIT_CASE(15) SNAP_WAIT_CASE(16) SNAP_WAIT_CASE(17) SNAP_WAIT_CASE(18) SNAP_WAIT_CASE(19)
    SNAP_WAIT_CASE(20) SNAP_WAIT_CASE(21) SNAP_WAIT_CASE(22) SNAP_WAIT_CASE(23) SNAP_WAIT_CASE(24)
#undef SNAP_WAIT_CASE
    default:
      wait_vm<0>();
      break;
  }
}

// Workgroup barrier that waits only for this wave's LDS traffic (not for its
// in-flight global->LDS tile loads, which are counted separately), and keeps
// the compiler from moving memory accesses across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0); vmcnt, expcnt untouched
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

}  // namespace snap
