// BITCOS batch-1 kernels with the multiply on the matrix cores, 4 lanes per
// row segment (one file per segment width so the instantiations compile in
// parallel).
#include "bitcos_diag.h"

namespace bitcos_k {
FastFn pick_diag_seg_4(int per_lane, bool bf16, bool table) { return pick_diag_seg<4>(per_lane, bf16, table); }
}  // namespace bitcos_k
