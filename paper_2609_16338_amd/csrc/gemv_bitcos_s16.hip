// BITCOS GEMV kernels with 16 lanes per row segment (one file per segment
// width so the instantiations compile in parallel).
#include "bitcos_fast.h"
#include "bitcos_kernel.h"

namespace bitcos_k {
KernelFn pick_seg_16(int per_lane, bool bf16, bool table) { return pick_seg<16>(per_lane, bf16, table); }
FastFn pick_fast_seg_16(int per_lane, bool bf16, bool table) {
  return pick_fast_seg<16>(per_lane, bf16, table);
}
}  // namespace bitcos_k
