// Test infrastructure: the library's hardware E4M3 conversion (e4m3x4_hw)
// against its bit-exact software encoder (f32_to_e4m3), both from the
// library's own header, on every fp32 bit pattern in every one of the four
// byte positions: input b is converted together with b rotated by 8, 16 and
// 24 bits, so each pattern also meets each position.  A bounded grid-stride
// loop over 2^32 patterns; prints the mismatch count and the first few.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>

#include "snap_internal.h"

using snap::e4m3x4_hw;
using snap::f32_to_e4m3;

__device__ __forceinline__ uint32_t rot(uint32_t x, int k) { return (x << k) | (x >> (32 - k)); }

__global__ void check(unsigned long long* count, uint32_t* first) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < (1ull << 32); i += stride) {
    const uint32_t b[4] = {(uint32_t)i, rot((uint32_t)i, 8), rot((uint32_t)i, 16), rot((uint32_t)i, 24)};
    const uint32_t hw = e4m3x4_hw(__uint_as_float(b[0]), __uint_as_float(b[1]), __uint_as_float(b[2]),
                                  __uint_as_float(b[3]));
    for (int k = 0; k < 4; ++k) {
      const uint32_t sw = f32_to_e4m3(__uint_as_float(b[k])), h = (hw >> (8 * k)) & 0xffu;
      if (sw != h) {
        const unsigned long long n = atomicAdd(count, 1ull);
        if (n < 8) {
          first[4 * n] = b[k];
          first[4 * n + 1] = (uint32_t)k;
          first[4 * n + 2] = sw;
          first[4 * n + 3] = h;
        }
      }
    }
  }
}

int main() {
  unsigned long long* count = nullptr;
  uint32_t* first = nullptr;
  if (hipMalloc(&count, sizeof(*count)) != hipSuccess || hipMalloc(&first, 32 * sizeof(uint32_t)) != hipSuccess ||
      hipMemset(count, 0, sizeof(*count)) != hipSuccess || hipMemset(first, 0, 32 * sizeof(uint32_t)) != hipSuccess) {
    std::printf("allocation failed\n");
    return 2;
  }
  hipLaunchKernelGGL(check, dim3(8192), dim3(256), 0, 0, count, first);
  if (hipGetLastError() != hipSuccess || hipDeviceSynchronize() != hipSuccess) {
    std::printf("launch failed\n");
    return 3;
  }
  unsigned long long n = 0;
  uint32_t f[32];
  if (hipMemcpy(&n, count, sizeof(n), hipMemcpyDeviceToHost) != hipSuccess ||
      hipMemcpy(f, first, sizeof(f), hipMemcpyDeviceToHost) != hipSuccess) {
    std::printf("copy failed\n");
    return 4;
  }
  std::printf("fp8 conversion mismatches over 2^32 patterns x 4 positions: %llu\n", n);
  for (unsigned long long k = 0; k < n && k < 8; ++k)
    std::printf("  bits 0x%08x position %u: encoder 0x%02x, instruction 0x%02x\n", f[4 * k], f[4 * k + 1],
                f[4 * k + 2], f[4 * k + 3]);
  (void)hipFree(count);
  (void)hipFree(first);
  return n == 0 ? 0 : 1;
}
