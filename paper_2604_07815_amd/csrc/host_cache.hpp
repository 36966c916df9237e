// Host-side caches of per-device facts that stay fixed for the life of the
// process, so that a decode call does not ask the runtime for them again:
// the compute-unit count, and the dynamic LDS limit already granted to a
// kernel (kernels that use more than 64 KiB of LDS need the limit raised once
// per device before their first launch there).
#pragma once

#include <hip/hip_runtime.h>

#include <atomic>
#include <mutex>
#include <vector>

namespace tls {

constexpr int kHostCacheDevices = 64;

// Compute units of the current device; 256 if the runtime cannot say.
inline int device_cus() {
  static std::atomic<int> known[kHostCacheDevices];  // 0: not asked yet
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  if (dev >= 0 && dev < kHostCacheDevices) {
    const int c = known[dev].load(std::memory_order_relaxed);
    if (c > 0) return c;
  }
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1) cus = 256;
  if (dev >= 0 && dev < kHostCacheDevices) known[dev].store(cus, std::memory_order_relaxed);
  return cus;
}

// Makes sure `func` may be launched with `bytes` of dynamic LDS on the current
// device: raises its limit the first time a size above the 64 KiB default is
// asked for there (or a larger one than was granted before), and remembers
// the grant.  Returns the runtime's error if raising the limit fails.
inline hipError_t allow_dynamic_lds(const void* func, size_t bytes) {
  if (bytes <= 65536) return hipSuccess;
  struct Grant {
    const void* func;
    int dev;
    size_t bytes;
  };
  static std::mutex mu;
  static std::vector<Grant> granted;  // guarded by mu
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  Grant* slot = nullptr;
  for (Grant& g : granted)
    if (g.func == func && g.dev == dev) slot = &g;
  if (slot && slot->bytes >= bytes) return hipSuccess;
  const hipError_t e = hipFuncSetAttribute(func, hipFuncAttributeMaxDynamicSharedMemorySize, int(bytes));
  if (e != hipSuccess) return e;
  if (slot)
    slot->bytes = bytes;
  else
    granted.push_back(Grant{func, dev, bytes});
  return hipSuccess;
}

}  // namespace tls
