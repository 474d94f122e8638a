// noalloc.hip -- device memory of the decode step that allocates nothing
// (snap_decode_step_noalloc): the split-K partials and (max, sum) pairs that
// snap_decode_step keeps in the caller's workspace live instead in one
// library-owned array per GPU, reserved with the code object and held until
// the process ends.  The array's host-side name is only a stand-in for the
// symbol: its device address comes from hipGetSymbolAddress, once per device
// with that device current, and only that address is handed to kernels.
#include <atomic>
#include <mutex>

#include "snap_internal.h"

namespace snap {

static __device__ __align__(256) unsigned char scratch[SNAP_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
static std::atomic<void*> g_scratch_addr[kMaxDevices];
static std::mutex g_scratch_mu;

// Device address of the current device's scratch array (looked up on the
// first call on that device).
snap_status noalloc_scratch(void** addr) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) {
    set_error("hipGetDevice failed: %s", hipGetErrorString(hipGetLastError()));
    return SNAP_ERR_HIP;
  }
  if (dev < 0 || dev >= kMaxDevices) {
    set_error("device %d is beyond the %d devices the scratch table covers", dev, kMaxDevices);
    return SNAP_ERR_UNSUPPORTED;
  }
  void* p = g_scratch_addr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_addr[dev].load(std::memory_order_relaxed);
    if (!p) {
      const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess || !p) {
        set_error("hipGetSymbolAddress of the scratch array failed: %s", hipGetErrorString(e));
        return SNAP_ERR_HIP;
      }
      g_scratch_addr[dev].store(p, std::memory_order_release);
    }
  }
  *addr = p;
  return SNAP_OK;
}

}  // namespace snap
