// 2-bit GEMV kernel instantiations (kernels in fixed_kernel.h).
#include "fixed_kernel.h"

namespace fixed_k {
KernelFn pick_bit2(int per_lane, int seg, bool bf16, bool table) {
  if (bf16)
    return table ? pick_kernel<Bit2K, bitcos::kMaxWords2Bf16, true, true>(per_lane, seg)
                 : pick_kernel<Bit2K, bitcos::kMaxWords2Bf16, true, false>(per_lane, seg);
  return table ? pick_kernel<Bit2K, bitcos::kMaxWords2I8, false, true>(per_lane, seg)
               : pick_kernel<Bit2K, bitcos::kMaxWords2I8, false, false>(per_lane, seg);
}
}  // namespace fixed_k
