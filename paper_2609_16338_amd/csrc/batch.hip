// Descriptor construction, tile choice and the batch entry points: a list of
// GEMVs of one format and tile run as one persistent launch.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include "../../include/bitcos.h"
#include "batch.h"
#include "launch_common.h"
#include "plan.h"

namespace bitcos {

int tile_for(const bitcos_layout* L, int32_t x_dtype, int* per_lane, int* seg, int* rows) {
  if (x_dtype != BITCOS_X_I8 && x_dtype != BITCOS_X_BF16) return BITCOS_E_ARG;
  const bool bf16 = x_dtype == BITCOS_X_BF16;
  Tile t;
  bool ok;
  switch (L->format) {
    case BITCOS_FMT_BITCOS: ok = bitcos_tile(L->k, bf16, &t); break;
    case BITCOS_FMT_TRIT5: ok = choose_tile(L->k / 128, bf16 ? kMaxBlocksBf16 : kMaxBlocksI8, &t, false, true); break;
    case BITCOS_FMT_BIT2:
      ok = (!bf16 && choose_tile(L->k / 16, kSoftWords2I8, &t)) ||
           choose_tile(L->k / 16, bf16 ? kMaxWords2Bf16 : kMaxWords2I8, &t);
      break;
    default: return BITCOS_E_ARG;
  }
  if (!ok) return BITCOS_E_UNSUPPORTED;
  *per_lane = t.per_lane;
  *seg = t.seg;
  *rows = t.rows;
  return BITCOS_OK;
}

static int check_layout(const bitcos_layout* L) {
  if (!L || L->version != BITCOS_LAYOUT_VERSION) return BITCOS_E_ARG;
  if (L->n < 1 || L->k < 32 || L->k % 32 || (L->group != 0 && L->group != 128)) return BITCOS_E_ARG;
  if (L->group == 128 && L->k % 128) return BITCOS_E_ARG;
  switch (L->format) {
    case BITCOS_FMT_BITCOS:
      if (L->unit_rows < 1) return BITCOS_E_ARG;
      if (L->nnz > 0xFFFFFFFFull) return BITCOS_E_UNSUPPORTED;
      return BITCOS_OK;
    case BITCOS_FMT_TRIT5:
    case BITCOS_FMT_BIT2:
      return L->k % 128 ? BITCOS_E_ARG : BITCOS_OK;
    default:
      return BITCOS_E_ARG;
  }
}

int make_desc(const bitcos_layout* L, const void* blob_dev, const void* x_dev, const float* xscale_dev,
              void* y_dev, int32_t x_dtype, int32_t y_mode, GemvDesc* d, int32_t m) {
  if (m < 1 || m > BITCOS_MAX_M) return BITCOS_E_ARG;
  int st = check_layout(L);
  if (st) return st;
  if (x_dtype != BITCOS_X_I8 && x_dtype != BITCOS_X_BF16) return BITCOS_E_ARG;
  if (y_mode != BITCOS_Y_F32 && y_mode != BITCOS_Y_I32_RAW && y_mode != BITCOS_Y_F32_ADD &&
      y_mode != BITCOS_Y_I32_RAW_ADD)
    return BITCOS_E_ARG;
  const bool raw_y = y_mode == BITCOS_Y_I32_RAW || y_mode == BITCOS_Y_I32_RAW_ADD;
  if (raw_y && x_dtype != BITCOS_X_I8) return BITCOS_E_ARG;
  if (!blob_dev || !x_dev || !y_dev) return BITCOS_E_ARG;
  if (xscale_dev && L->k % 128) return BITCOS_E_ARG;
  int per_lane = 0, seg = 0, rows = 0;
  if (!mfma_layout_ok(L) || (m == 1 && !batch1_on_small_batch(L, x_dtype))) {
    st = tile_for(L, x_dtype, &per_lane, &seg, &rows);  // the small-batch kernel has no tile limit on K
    if (st) return st;
  }
  memset(d, 0, sizeof(*d));
  const uint8_t* blob = static_cast<const uint8_t*>(blob_dev);
  d->sec0 = blob + L->sec_off[0];
  d->scales = reinterpret_cast<const uint16_t*>(blob + L->sec_off[BITCOS_SEC_SCALES]);
  d->x = x_dev;
  d->xscale = xscale_dev;
  d->y = y_dev;
  d->n = L->n;
  d->ngroups = L->k / 128;
  d->last_dword = static_cast<uint32_t>(L->sec_bytes[0] / 4 - 1);
  if (L->sec_bytes[0] >= 0x80000000ull || L->total_bytes >= 0x80000000ull) return BITCOS_E_UNSUPPORTED;
  d->sec0_bytes = static_cast<uint32_t>(L->sec_bytes[0]);
  d->scales_bytes = static_cast<uint32_t>(L->sec_bytes[BITCOS_SEC_SCALES]);
  const uint64_t xb = static_cast<uint64_t>(m) * L->k * (x_dtype == BITCOS_X_BF16 ? 2u : 1u);
  const uint64_t yb = static_cast<uint64_t>(m) * L->n * 4u;
  if (xb >= 0x80000000ull || yb >= 0x80000000ull) return BITCOS_E_UNSUPPORTED;
  d->x_bytes = static_cast<uint32_t>(xb);
  d->y_bytes = static_cast<uint32_t>(yb);
  d->mode = (L->group == 128 ? kModeGrouped : 0) | (xscale_dev ? kModeXscale : 0) |
            (raw_y ? kModeRaw : 0) |
            (y_mode == BITCOS_Y_F32_ADD || y_mode == BITCOS_Y_I32_RAW_ADD ? kModeAdd : 0);
  if (L->format == BITCOS_FMT_BITCOS) {
    d->signs = reinterpret_cast<const uint32_t*>(blob + L->sec_off[BITCOS_SEC_SIGNS]);
    d->signs_bytes = static_cast<uint32_t>(L->sec_bytes[BITCOS_SEC_SIGNS]);
    d->offsets = reinterpret_cast<const uint32_t*>(blob + L->sec_off[BITCOS_SEC_OFFSETS]);
    d->nnz = static_cast<uint32_t>(L->nnz);
    d->upr = L->k / 32;
    d->unit_rows = L->unit_rows;
  } else {
    d->upr = L->format == BITCOS_FMT_TRIT5 ? L->k / 128 : L->k / 16;
    d->unit_rows = rows;  // one wave step per unit
  }
  d->unit_begin = 0;
  d->units = (L->n + d->unit_rows - 1) / d->unit_rows;
  d->offset_last = static_cast<int32_t>(d->units);
  d->offset_stride = 0;
  return BITCOS_OK;
}

bool batch1_on_small_batch(const bitcos_layout* L, int32_t x_dtype) {
  if (!L || !mfma_layout_ok(L)) return false;
  int per_lane = 0, seg = 0, rows = 0;
  return tile_for(L, x_dtype, &per_lane, &seg, &rows) == BITCOS_E_UNSUPPORTED;
}

bool to_step_units(GemvDesc* d, int rows) {
  if (d->unit_rows < 1 || rows % d->unit_rows) return false;
  d->offset_stride = rows / d->unit_rows;
  d->units = (d->n + rows - 1) / rows;
  return true;
}

static int launch(const BatchHeader& h, const GemvDesc* table_dev, const GemvDesc& one, void* stream) {
  if (h.m > 1 || h.small_batch) return launch_bitcos_mfma(h, table_dev, one, stream);
  return h.format == BITCOS_FMT_BITCOS ? launch_bitcos(h, table_dev, one, stream)
                                       : launch_fixed(h, table_dev, one, stream);
}

// Batch table for m > 1 (the small-batch kernel; BITCOS layouts it runs only).
static int build_small_batch(int32_t count, int32_t m, const bitcos_layout* layouts,
                             const void* const* blobs_dev, const void* const* x_dev,
                             const float* const* xscale_dev, void* const* y_dev, BatchHeader* h,
                             GemvDesc* descs) {
  int64_t units = 0;
  for (int32_t i = 0; i < count; ++i) {
    const bitcos_layout* L = &layouts[i];
    if (L->format != BITCOS_FMT_BITCOS) return L->format == BITCOS_FMT_TRIT5 || L->format == BITCOS_FMT_BIT2
                                                   ? BITCOS_E_UNSUPPORTED
                                                   : BITCOS_E_ARG;
    const float* xs = xscale_dev ? xscale_dev[i] : nullptr;
    int st = make_desc(L, blobs_dev[i], x_dev[i], xs, y_dev[i], h->x_dtype, h->y_mode, &descs[i], m);
    if (st) return st;
    if (!mfma_layout_ok(L)) return BITCOS_E_UNSUPPORTED;
    if (xs) h->any_xscale = 1;
    to_mfma_units(&descs[i]);
    descs[i].unit_begin = units;
    units += descs[i].units;
  }
  if (units >= (int64_t(1) << 31)) return BITCOS_E_UNSUPPORTED;
  h->total_units = units;
  return BITCOS_OK;
}

}  // namespace bitcos

extern "C" {

size_t bitcos_batch_bytes(int32_t count) {
  return count < 1 ? 0 : bitcos::batch_bytes(count);
}

int bitcos_batch_build(int32_t count, int32_t m, const bitcos_layout* layouts, const void* const* blobs_dev,
                       const void* const* x_dev, const float* const* xscale_dev, void* const* y_dev,
                       int32_t x_dtype, int32_t y_mode, void* table, size_t table_bytes) {
  if (count < 1 || !layouts || !blobs_dev || !x_dev || !y_dev || !table) return BITCOS_E_ARG;
  if (m < 1 || m > BITCOS_MAX_M) return BITCOS_E_ARG;
  if (table_bytes < bitcos::batch_bytes(count)) return BITCOS_E_SPACE;
  bitcos::BatchHeader h;
  memset(&h, 0, sizeof(h));
  h.magic = bitcos::kBatchMagic;
  h.version = BITCOS_LAYOUT_VERSION;
  h.format = layouts[0].format;
  h.count = count;
  h.x_dtype = x_dtype;
  h.y_mode = y_mode;
  h.m = m;
  bitcos::GemvDesc* descs =
      reinterpret_cast<bitcos::GemvDesc*>(static_cast<uint8_t*>(table) + sizeof(bitcos::BatchHeader));
  if (m > 1 || bitcos::batch1_on_small_batch(&layouts[0], x_dtype)) {
    h.small_batch = m == 1;
    int st = bitcos::build_small_batch(count, m, layouts, blobs_dev, x_dev, xscale_dev, y_dev, &h, descs);
    if (st) return st;
    memcpy(table, &h, sizeof(h));
    return BITCOS_OK;
  }
  int64_t units = 0;
  int step_rows = 0;
  h.unit_is_step = 1;
  h.row_offsets = 1;
  for (int32_t i = 0; i < count; ++i) {
    const bitcos_layout* L = &layouts[i];
    if (L->format != h.format) return BITCOS_E_UNSUPPORTED;
    int per_lane = 0, seg = 0, rows = 0;
    int st = bitcos::tile_for(L, x_dtype, &per_lane, &seg, &rows);
    if (st) return st;
    if (i == 0) {
      h.per_lane = per_lane;
      h.seg = seg;
    } else if (per_lane != h.per_lane || seg != h.seg) {
      return BITCOS_E_UNSUPPORTED;  // different tiles: split into one batch per tile
    }
    st = bitcos::make_desc(L, blobs_dev[i], x_dev[i], xscale_dev ? xscale_dev[i] : nullptr, y_dev[i],
                           x_dtype, y_mode, &descs[i]);
    if (st) return st;
    if (descs[i].mode & bitcos::kModeXscale) h.any_xscale = 1;
    if (descs[i].mode & bitcos::kModeGrouped) h.any_grouped = 1;
    if (descs[i].unit_rows != 1) h.row_offsets = 0;
    if (h.format != BITCOS_FMT_BITCOS || rows % descs[i].unit_rows) h.unit_is_step = 0;
    step_rows = rows;
  }
  // The streaming kernel counts every GEMV in wave steps; the general kernel
  // in the layout's units.
  for (int32_t i = 0; i < count; ++i) {
    if (h.unit_is_step) bitcos::to_step_units(&descs[i], step_rows);
    descs[i].unit_begin = units;
    units += descs[i].units;
  }
  h.total_units = units;
  memcpy(table, &h, sizeof(h));
  return BITCOS_OK;
}

int bitcos_gemv_batch(const void* table_host, const void* table_dev, void* stream) {
  if (!table_host || !table_dev) return BITCOS_E_ARG;
  bitcos::BatchHeader h;
  memcpy(&h, table_host, sizeof(h));
  if (h.magic != bitcos::kBatchMagic || h.version != BITCOS_LAYOUT_VERSION || h.count < 1) return BITCOS_E_ARG;
  if (h.m < 1 || h.m > BITCOS_MAX_M) return BITCOS_E_ARG;
  if (reinterpret_cast<uintptr_t>(table_dev) % 16) return BITCOS_E_ARG;
  const bitcos::GemvDesc* descs = reinterpret_cast<const bitcos::GemvDesc*>(
      static_cast<const uint8_t*>(table_dev) + sizeof(bitcos::BatchHeader));
  const bitcos::GemvDesc* first = reinterpret_cast<const bitcos::GemvDesc*>(
      static_cast<const uint8_t*>(table_host) + sizeof(bitcos::BatchHeader));
  return bitcos::launch(h, descs, *first, stream);
}

static_assert(sizeof(bitcos_launch_info) == 40, "bitcos_launch_info is 40 bytes (the Python binding mirrors it)");

int bitcos_describe(const bitcos_layout* L, int32_t m, int32_t x_dtype, bitcos_launch_info* out) {
  if (!L || !out) return BITCOS_E_ARG;
  if (m < 1 || m > BITCOS_MAX_M) return BITCOS_E_ARG;
  int st = bitcos::check_layout(L);
  if (st) return st;
  if (x_dtype != BITCOS_X_I8 && x_dtype != BITCOS_X_BF16) return BITCOS_E_ARG;
  if (bitcos::mfma_layout_ok(L) && (m > 1 || bitcos::batch1_on_small_batch(L, x_dtype))) {
    // small-batch kernel: 4 lanes per row, one word each per group
    const int64_t units = (L->n + bitcos::kMfmaUnitRows - 1) / bitcos::kMfmaUnitRows;
    out->per_lane = 1;
    out->seg_lanes = 4;
    out->rows_per_step = bitcos::kMfmaUnitRows;
    out->lanes_used = 4;
    out->waves = units;
    out->workgroups = (units + 3) / 4;
    out->kernel = BITCOS_KERNEL_SMALL_BATCH;
    out->reserved = 0;
    return BITCOS_OK;
  }
  int per_lane = 0, seg = 0, rows = 0;
  st = bitcos::tile_for(L, x_dtype, &per_lane, &seg, &rows);
  if (st) return st;
  const int unit_rows = L->format == BITCOS_FMT_BITCOS ? L->unit_rows : rows;
  const int64_t units = (L->n + unit_rows - 1) / unit_rows;
  out->per_lane = per_lane;
  out->seg_lanes = seg;
  out->rows_per_step = rows;
  int upr = L->format == BITCOS_FMT_BITCOS ? L->k / 32 : (L->format == BITCOS_FMT_TRIT5 ? L->k / 128 : L->k / 16);
  out->lanes_used = (upr + per_lane - 1) / per_lane;
  out->waves = units;          // upper bound: persistent grids use at most the resident waves
  out->workgroups = (units + 3) / 4;
  out->reserved = 0;
  if (L->format != BITCOS_FMT_BITCOS) {
    out->kernel = BITCOS_KERNEL_FIXED;
  } else {  // the choice launch_bitcos makes (batch 1; m > 1 here runs m batch-1 calls)
    const bool streaming = rows % L->unit_rows == 0 && (L->n + rows - 1) / rows < (int64_t(1) << 30);
    const bool matrix = streaming && L->group == 0 && (seg > 16 || L->unit_rows == 1);
    out->kernel = matrix ? BITCOS_KERNEL_MATRIX : streaming ? BITCOS_KERNEL_STREAMING : BITCOS_KERNEL_GENERAL;
  }
  return BITCOS_OK;
}

}  // extern "C"
