// Host-side helpers shared by the GEMV launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>
#include <unordered_map>

#include "../../include/bitcos.h"

// Status of the launch just enqueued on this thread.
inline int bitcos_launch_status() {
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? BITCOS_OK : BITCOS_E_HIP;
}

// Resident 256-thread blocks per CU for a kernel.  Queried once per kernel
// and remembered for the life of the process (a read-mostly cache of a
// device property, not state that changes results).
inline int bitcos_blocks_per_cu(const void* fn, int threads) {
  static std::mutex mu;
  static std::unordered_map<const void*, int> cache;
  {
    std::lock_guard<std::mutex> g(mu);
    auto it = cache.find(fn);
    if (it != cache.end()) return it->second;
  }
  int nb = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, fn, threads, 0) != hipSuccess || nb < 1) nb = 1;
  std::lock_guard<std::mutex> g(mu);
  cache[fn] = nb;
  return nb;
}

// Blocks of `threads` threads for a persistent launch over `units` work units:
// as many as the GPU keeps resident at once, and no more than one wave per
// unit.  -1 on a HIP error.
inline int64_t persistent_blocks(const void* fn, int64_t units, int threads = 256) {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return -1;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return -1;
  const int64_t resident = static_cast<int64_t>(cus) * bitcos_blocks_per_cu(fn, threads);
  const int64_t wpb = threads / 64;
  const int64_t need = (units + wpb - 1) / wpb;
  int64_t b = need < resident ? need : resident;
  return b < 1 ? 1 : b;
}
