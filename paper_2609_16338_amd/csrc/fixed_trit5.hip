// Five-trit GEMV kernel instantiations (kernels in fixed_kernel.h).
#include "fixed_kernel.h"

namespace fixed_k {
KernelFn pick_trit5(int per_lane, int seg, bool bf16, bool table) {
  if (seg == 20) {
    if (bf16) {
      const auto seq = std::make_integer_sequence<int, bitcos::kMaxBlocksBf16>{};
      return table ? pick_p<Trit5K, 20, true, true>(per_lane, seq) : pick_p<Trit5K, 20, true, false>(per_lane, seq);
    }
    const auto seq = std::make_integer_sequence<int, bitcos::kMaxBlocksI8>{};
    return table ? pick_p<Trit5K, 20, false, true>(per_lane, seq) : pick_p<Trit5K, 20, false, false>(per_lane, seq);
  }
  if (bf16)
    return table ? pick_kernel<Trit5K, bitcos::kMaxBlocksBf16, true, true>(per_lane, seg)
                 : pick_kernel<Trit5K, bitcos::kMaxBlocksBf16, true, false>(per_lane, seg);
  return table ? pick_kernel<Trit5K, bitcos::kMaxBlocksI8, false, true>(per_lane, seg)
               : pick_kernel<Trit5K, bitcos::kMaxBlocksI8, false, false>(per_lane, seg);
}
}  // namespace fixed_k
