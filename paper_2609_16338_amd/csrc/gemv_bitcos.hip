// Launcher of the BITCOS GEMV kernels (kernels in bitcos_kernel.h, one
// instantiation file per lane-segment width) and the single-GEMV entry point.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/bitcos.h"
#include "batch.h"
#include "bitcos_diag.h"
#include "bitcos_fast.h"
#include "bitcos_kernel.h"
#include "launch_common.h"
#include "plan.h"

namespace bitcos_k {
KernelFn pick_seg_4(int per_lane, bool bf16, bool table);
KernelFn pick_seg_8(int per_lane, bool bf16, bool table);
KernelFn pick_seg_16(int per_lane, bool bf16, bool table);
KernelFn pick_seg_32(int per_lane, bool bf16, bool table);
KernelFn pick_seg_64(int per_lane, bool bf16, bool table);
FastFn pick_fast_seg_4(int per_lane, bool bf16, bool table);
FastFn pick_fast_seg_8(int per_lane, bool bf16, bool table);
FastFn pick_fast_seg_16(int per_lane, bool bf16, bool table);
FastFn pick_fast_seg_32(int per_lane, bool bf16, bool table);
FastFn pick_fast_seg_64(int per_lane, bool bf16, bool table);
FastFn pick_diag_seg_4(int per_lane, bool bf16, bool table);
FastFn pick_diag_seg_8(int per_lane, bool bf16, bool table);
FastFn pick_diag_seg_16(int per_lane, bool bf16, bool table);
FastFn pick_diag_seg_32(int per_lane, bool bf16, bool table);
FastFn pick_diag_seg_64(int per_lane, bool bf16, bool table);
}  // namespace bitcos_k

namespace bitcos {

static bitcos_k::KernelFn pick_bitcos(int per_lane, int seg, bool bf16, bool table) {
  switch (seg) {
    case 4: return bitcos_k::pick_seg_4(per_lane, bf16, table);
    case 8: return bitcos_k::pick_seg_8(per_lane, bf16, table);
    case 16: return bitcos_k::pick_seg_16(per_lane, bf16, table);
    case 32: return bitcos_k::pick_seg_32(per_lane, bf16, table);
    case 64: return bitcos_k::pick_seg_64(per_lane, bf16, table);
    default: return nullptr;
  }
}

static bitcos_k::FastFn pick_bitcos_fast(int per_lane, int seg, bool bf16, bool table) {
  switch (seg) {
    case 4: return bitcos_k::pick_fast_seg_4(per_lane, bf16, table);
    case 8: return bitcos_k::pick_fast_seg_8(per_lane, bf16, table);
    case 16: return bitcos_k::pick_fast_seg_16(per_lane, bf16, table);
    case 32: return bitcos_k::pick_fast_seg_32(per_lane, bf16, table);
    case 64: return bitcos_k::pick_fast_seg_64(per_lane, bf16, table);
    default: return nullptr;
  }
}

// Streaming kernel with the multiply on the matrix cores: one scale per
// tensor (or raw sums) and no activation scales.
static bitcos_k::FastFn pick_bitcos_diag(int per_lane, int seg, bool bf16, bool table) {
  switch (seg) {
    case 4: return bitcos_k::pick_diag_seg_4(per_lane, bf16, table);
    case 8: return bitcos_k::pick_diag_seg_8(per_lane, bf16, table);
    case 16: return bitcos_k::pick_diag_seg_16(per_lane, bf16, table);
    case 32: return bitcos_k::pick_diag_seg_32(per_lane, bf16, table);
    case 64: return bitcos_k::pick_diag_seg_64(per_lane, bf16, table);
    default: return nullptr;
  }
}

int launch_bitcos(const BatchHeader& h, const GemvDesc* table_dev, const GemvDesc& one, void* stream) {
  const bool bf16 = h.x_dtype == BITCOS_X_BF16;
  // Streaming kernels when every unit is one wave step (their unit counters
  // are 32-bit): on the matrix cores unless some GEMV has group or
  // activation scales (with 16 or fewer lanes per row the matrix-core kernel
  // also needs one sign offset per row).  The general kernel otherwise.
  const bool streaming = h.unit_is_step && h.total_units < (int64_t(1) << 30);
  const bool diag = streaming && !h.any_grouped && !h.any_xscale && (h.seg > 16 || h.row_offsets);
  const bool table = table_dev != nullptr;
  bitcos_k::KernelFn fn = diag        ? pick_bitcos_diag(h.per_lane, h.seg, bf16, table)
                          : streaming ? pick_bitcos_fast(h.per_lane, h.seg, bf16, table)
                                      : pick_bitcos(h.per_lane, h.seg, bf16, table);
  if (!fn) return BITCOS_E_UNSUPPORTED;
  bitcos_k::KernelArgs a;
  a.table = table_dev;
  a.total_units = h.total_units;
  a.count = h.count;
  a.pad = 0;
  a.one = one;
  const int threads = diag        ? bitcos_k::diag_threads(h.per_lane, bf16)
                      : streaming ? bitcos_k::fast_threads(h.per_lane, bf16)
                                  : (bf16 ? bitcos_k::Cfg<true>::kThreads : bitcos_k::Cfg<false>::kThreads);
  const int64_t blocks = persistent_blocks(reinterpret_cast<const void*>(fn), h.total_units, threads);
  if (blocks <= 0 || blocks > 0x7FFFFFFF) return BITCOS_E_HIP;
  hipLaunchKernelGGL(fn, dim3(static_cast<unsigned>(blocks)), dim3(threads), 0,
                     static_cast<hipStream_t>(stream), a);
  return bitcos_launch_status();
}

}  // namespace bitcos

extern "C" int bitcos_gemv(const bitcos_layout* L, const void* blob_dev, int32_t m,
                           const void* x_dev, int32_t x_dtype, const float* xscale_dev,
                           void* y_dev, int32_t y_mode, void* stream) {
  if (!L || L->format != BITCOS_FMT_BITCOS) return BITCOS_E_ARG;
  if (m < 1 || m > BITCOS_MAX_M) return BITCOS_E_ARG;
  // m > 1, or a batch-1 row longer than every batch-1 tile: the small-batch kernel.
  if (m > 1 || bitcos::batch1_on_small_batch(L, x_dtype)) {
    if (!bitcos::mfma_layout_ok(L))
      return bitcos::gemv_rows(bitcos_gemv, L, blob_dev, m, x_dev, x_dtype, xscale_dev, y_dev, y_mode, stream);
    bitcos::GemvDesc d;
    int st = bitcos::make_desc(L, blob_dev, x_dev, xscale_dev, y_dev, x_dtype, y_mode, &d, m);
    if (st) return st;
    bitcos::to_mfma_units(&d);
    bitcos::BatchHeader h{};
    h.magic = bitcos::kBatchMagic;
    h.version = BITCOS_LAYOUT_VERSION;
    h.format = BITCOS_FMT_BITCOS;
    h.count = 1;
    h.x_dtype = x_dtype;
    h.y_mode = y_mode;
    h.m = m;
    h.small_batch = m == 1;
    h.any_xscale = xscale_dev != nullptr;
    h.total_units = d.units;
    return bitcos::launch_bitcos_mfma(h, nullptr, d, stream);
  }
  bitcos::GemvDesc d;
  int st = bitcos::make_desc(L, blob_dev, x_dev, xscale_dev, y_dev, x_dtype, y_mode, &d);
  if (st) return st;
  bitcos::BatchHeader h{};
  h.magic = bitcos::kBatchMagic;
  h.version = BITCOS_LAYOUT_VERSION;
  h.format = BITCOS_FMT_BITCOS;
  h.count = 1;
  h.x_dtype = x_dtype;
  h.y_mode = y_mode;
  h.m = 1;
  h.any_xscale = (d.mode & bitcos::kModeXscale) != 0;
  h.any_grouped = (d.mode & bitcos::kModeGrouped) != 0;
  h.row_offsets = d.unit_rows == 1;
  int rows = 0;
  st = bitcos::tile_for(L, x_dtype, &h.per_lane, &h.seg, &rows);
  if (st) return st;
  h.unit_is_step = bitcos::to_step_units(&d, rows);
  h.total_units = d.units;
  return bitcos::launch_bitcos(h, nullptr, d, stream);
}
