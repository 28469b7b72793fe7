// Launcher of the same-GPU baselines (five-trit and 2-bit; kernels in
// fixed_kernel.h) and their single-GEMV entry points.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/bitcos.h"
#include "batch.h"
#include "fixed_kernel.h"
#include "launch_common.h"

namespace fixed_k {
KernelFn pick_trit5(int per_lane, int seg, bool bf16, bool table);
KernelFn pick_bit2(int per_lane, int seg, bool bf16, bool table);
}  // namespace fixed_k

namespace bitcos {

int launch_fixed(const BatchHeader& h, const GemvDesc* table_dev, const GemvDesc& one, void* stream) {
  const bool bf16 = h.x_dtype == BITCOS_X_BF16;
  const bool table = table_dev != nullptr;
  fixed_k::KernelFn fn = h.format == BITCOS_FMT_TRIT5 ? fixed_k::pick_trit5(h.per_lane, h.seg, bf16, table)
                                                      : fixed_k::pick_bit2(h.per_lane, h.seg, bf16, table);
  if (!fn) return BITCOS_E_UNSUPPORTED;
  fixed_k::KernelArgs a;
  a.table = table_dev;
  a.total_units = h.total_units;
  a.count = h.count;
  a.pad = 0;
  a.one = one;
  const int threads = fixed_k::fixed_threads(h.format == BITCOS_FMT_BIT2, bf16, h.per_lane);
  const int64_t blocks = persistent_blocks(reinterpret_cast<const void*>(fn), h.total_units, threads);
  if (blocks <= 0 || blocks > 0x7FFFFFFF) return BITCOS_E_HIP;
  hipLaunchKernelGGL(fn, dim3(static_cast<unsigned>(blocks)), dim3(threads), 0,
                     static_cast<hipStream_t>(stream), a);
  return bitcos_launch_status();
}

}  // namespace bitcos

static int fixed_gemv(uint32_t fmt, const bitcos_layout* L, const void* blob_dev, int32_t m,
                      const void* x_dev, int32_t x_dtype, const float* xscale_dev, void* y_dev,
                      int32_t y_mode, void* stream) {
  if (!L || L->format != fmt) return BITCOS_E_ARG;
  if (m < 1 || m > BITCOS_MAX_M) return BITCOS_E_ARG;
  if (m > 1)
    return bitcos::gemv_rows(fmt == BITCOS_FMT_TRIT5 ? trit5_gemv : bit2_gemv, L, blob_dev, m, x_dev, x_dtype,
                             xscale_dev, y_dev, y_mode, stream);
  bitcos::GemvDesc d;
  int st = bitcos::make_desc(L, blob_dev, x_dev, xscale_dev, y_dev, x_dtype, y_mode, &d);
  if (st) return st;
  bitcos::BatchHeader h{};
  h.magic = bitcos::kBatchMagic;
  h.version = BITCOS_LAYOUT_VERSION;
  h.format = fmt;
  h.count = 1;
  h.x_dtype = x_dtype;
  h.y_mode = y_mode;
  h.m = 1;
  int rows = 0;
  st = bitcos::tile_for(L, x_dtype, &h.per_lane, &h.seg, &rows);
  if (st) return st;
  h.total_units = d.units;
  return bitcos::launch_fixed(h, nullptr, d, stream);
}

extern "C" {

int trit5_gemv(const bitcos_layout* L, const void* blob_dev, int32_t m, const void* x_dev,
               int32_t x_dtype, const float* xscale_dev, void* y_dev, int32_t y_mode,
               void* stream) {
  return fixed_gemv(BITCOS_FMT_TRIT5, L, blob_dev, m, x_dev, x_dtype, xscale_dev, y_dev, y_mode, stream);
}

int bit2_gemv(const bitcos_layout* L, const void* blob_dev, int32_t m, const void* x_dev,
              int32_t x_dtype, const float* xscale_dev, void* y_dev, int32_t y_mode,
              void* stream) {
  return fixed_gemv(BITCOS_FMT_BIT2, L, blob_dev, m, x_dev, x_dtype, xscale_dev, y_dev, y_mode, stream);
}

}  // extern "C"
