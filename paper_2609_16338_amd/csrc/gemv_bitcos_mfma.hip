// Launcher of the small-batch BITCOS kernel (bitcos_mfma.h): 2 <= m <= 16
// activation rows, one launch for one GEMV or a batch table.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/bitcos.h"
#include "batch.h"
#include "bitcos_mfma.h"
#include "launch_common.h"

static_assert(bitcos_k::kMfmaRows == bitcos::kMfmaUnitRows, "host and kernel agree on the unit");
static_assert(bitcos_k::kMfmaMaxBatch == BITCOS_MAX_M, "one MFMA tile holds every activation row");

namespace bitcos {

int launch_bitcos_mfma(const BatchHeader& h, const GemvDesc* table_dev, const GemvDesc& one, void* stream) {
  if (h.format != BITCOS_FMT_BITCOS || h.m < 1 || h.m > BITCOS_MAX_M) return BITCOS_E_UNSUPPORTED;
  if (h.m == 1 && !h.small_batch) return BITCOS_E_UNSUPPORTED;
  if (h.total_units < 1 || h.total_units >= (int64_t(1) << 31)) return BITCOS_E_UNSUPPORTED;
  const bool bf16 = h.x_dtype == BITCOS_X_BF16;
  bitcos_k::MfmaFn fn = bitcos_k::pick_mfma(bf16, h.any_xscale != 0, table_dev != nullptr);
  bitcos_k::KernelArgs a;
  a.table = table_dev;
  a.total_units = h.total_units;
  a.count = h.count;
  a.pad = 0;
  a.one = one;
  const int threads = bitcos_k::mfma_threads(bf16, h.any_xscale != 0);
  const int64_t blocks = persistent_blocks(reinterpret_cast<const void*>(fn), h.total_units, threads);
  if (blocks <= 0 || blocks > 0x7FFFFFFF) return BITCOS_E_HIP;
  hipLaunchKernelGGL(fn, dim3(static_cast<unsigned>(blocks)), dim3(threads), 0,
                     static_cast<hipStream_t>(stream), a);
  return bitcos_launch_status();
}

}  // namespace bitcos
