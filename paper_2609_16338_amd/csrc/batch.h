// Descriptors shared by the host launchers and the persistent GEMV kernels.
//
// Every GEMV launch -- one matrix or a whole list of them -- runs as a
// persistent grid: the matrices' work units (a few rows each) are numbered
// consecutively across the list, and every wave takes one contiguous range of
// units, so its activations stay in registers until it crosses into the next
// matrix and its loads can be issued a step ahead.  A single GEMV passes its
// one descriptor by value; a batch passes a table in device memory.
#pragma once

#include <stdint.h>

#include "../../include/bitcos.h"

namespace bitcos {

struct GemvDesc {
  const void* sec0;         // BITCOS bitmap; five-trit / 2-bit codes
  const uint32_t* signs;    // BITCOS sign stream
  const uint32_t* offsets;  // BITCOS per-unit sign offsets
  const uint16_t* scales;   // fp16 scales
  const void* x;            // activations [k] (int8 or bf16 bits)
  const float* xscale;      // NULL or fp32 [k/128]
  void* y;                  // output [n]
  int64_t unit_begin;       // first unit of this GEMV in the launch
  int64_t units;            // units of this GEMV
  uint32_t nnz;             // BITCOS non-zeros
  uint32_t last_dword;      // last readable dword of section 0
  int32_t n;                // rows
  int32_t upr;              // per-row units: BITCOS / 2-bit words, five-trit blocks
  int32_t ngroups;          // K / 128 (0 if K % 128 != 0)
  int32_t unit_rows;        // rows per unit
  int32_t mode;             // kMode* flags
  uint32_t sec0_bytes;      // bytes of section 0
  uint32_t signs_bytes;     // bytes of the sign stream (with its zero tail)
  uint32_t scales_bytes;    // bytes of the scales
  uint32_t x_bytes;         // bytes of the activations
  uint32_t y_bytes;         // bytes of the output (4 per row)
  int32_t offset_stride;    // streaming kernel: offset entries per wave step (its unit), else 0
  int32_t offset_last;      // index of the last offset entry (= nnz)
};
static_assert(sizeof(GemvDesc) == 128, "GemvDesc is 128 bytes");

constexpr int kModeGrouped = 1;  // one scale per (row, 128-group)
constexpr int kModeXscale = 2;   // per-group activation scales
constexpr int kModeRaw = 4;      // int32 raw row sums
constexpr int kModeAdd = 8;      // add the result onto y instead of overwriting it

constexpr uint32_t kBatchMagic = 0x42435342u;  // "BSCB"

// Header of a batch table; `count` descriptors follow at offset 128.
struct BatchHeader {
  uint32_t magic;
  uint32_t version;
  uint32_t format;
  int32_t count;
  int32_t x_dtype;
  int32_t y_mode;
  int32_t per_lane;
  int32_t seg;
  int64_t total_units;
  int32_t unit_is_step;  // every GEMV's unit is one wave step (BITCOS streaming kernel)
  int32_t m;             // activation rows (> 1: the small-batch MFMA kernel)
  int32_t any_xscale;    // some GEMV has activation scales
  int32_t any_grouped;   // some GEMV has group scales
  int32_t row_offsets;   // every BITCOS GEMV stores one sign offset per row
  int32_t small_batch;   // m == 1 rows longer than any batch-1 tile: the small-batch kernel
  int32_t reserved[16];
};
static_assert(sizeof(BatchHeader) == 128, "BatchHeader is 128 bytes");

inline size_t batch_bytes(int32_t count) {
  return sizeof(BatchHeader) + sizeof(GemvDesc) * static_cast<size_t>(count);
}

// Persistent launch of one format's kernel over `total_units` units.  With
// table_dev == nullptr the single descriptor `one` is used.  Defined next to
// each format's kernels.
int launch_bitcos(const BatchHeader& h, const GemvDesc* table_dev, const GemvDesc& one, void* stream);
int launch_fixed(const BatchHeader& h, const GemvDesc* table_dev, const GemvDesc& one, void* stream);
int launch_bitcos_mfma(const BatchHeader& h, const GemvDesc* table_dev, const GemvDesc& one, void* stream);

// Small-batch (m > 1) BITCOS kernel: rows per work unit, and the layouts it
// runs (one sign offset per row, whole 128-weight groups).
constexpr int kMfmaUnitRows = 32;
inline bool mfma_layout_ok(const bitcos_layout* L) {
  return L->format == BITCOS_FMT_BITCOS && L->unit_rows == 1 && L->k % 128 == 0;
}

// m activation rows as m batch-1 calls of `gemv` (row i: x + i k, xscale +
// i k / 128, y + i n), for layouts the small-batch kernel does not take.
// The first call validates everything the others would, so an error
// enqueues nothing.
using GemvEntry = int (*)(const bitcos_layout*, const void*, int32_t, const void*, int32_t, const float*, void*,
                          int32_t, void*);
inline int gemv_rows(GemvEntry gemv, const bitcos_layout* L, const void* blob_dev, int32_t m, const void* x_dev,
                     int32_t x_dtype, const float* xscale_dev, void* y_dev, int32_t y_mode, void* stream) {
  const size_t xrow = static_cast<size_t>(L->k) * (x_dtype == BITCOS_X_BF16 ? 2u : 1u);
  for (int32_t i = 0; i < m; ++i) {
    const void* x = x_dev ? static_cast<const uint8_t*>(x_dev) + i * xrow : nullptr;
    const float* xs = xscale_dev ? xscale_dev + static_cast<size_t>(i) * (L->k / 128) : nullptr;
    void* y = y_dev ? static_cast<uint8_t*>(y_dev) + static_cast<size_t>(i) * L->n * 4u : nullptr;
    const int st = gemv(L, blob_dev, 1, x, x_dtype, xs, y, y_mode, stream);
    if (st) return st;
  }
  return BITCOS_OK;
}

// Batch-1 layouts with rows longer than any batch-1 tile (the activations
// of a lane live in VGPRs: bf16 K > 16384, int8 K > 32768) run the
// small-batch kernel with one activation row, when it takes the layout.
bool batch1_on_small_batch(const bitcos_layout* L, int32_t x_dtype);

// Count a descriptor in the small-batch kernel's steps: units of 32 rows,
// each K / 512 steps (four 128-weight groups per step).  The kernel splits a
// launch's steps evenly over its waves.
inline void to_mfma_units(GemvDesc* d) {
  d->units = static_cast<int64_t>((d->n + kMfmaUnitRows - 1) / kMfmaUnitRows) * ((d->ngroups + 3) / 4);
}

// Tile (per-lane units, lanes per row) the given layout runs with.
int tile_for(const bitcos_layout* L, int32_t x_dtype, int* per_lane, int* seg, int* rows);

// Count the descriptor's units in wave steps of `rows` rows for the
// streaming BITCOS kernel; possible when the layout's unit divides the step.
bool to_step_units(GemvDesc* d, int rows);

// Fill one descriptor from a layout and device pointers (unit_begin = 0);
// m activation rows ([m][k] in, [m][n] out).
int make_desc(const bitcos_layout* L, const void* blob_dev, const void* x_dev, const float* xscale_dev,
              void* y_dev, int32_t x_dtype, int32_t y_mode, GemvDesc* d, int32_t m = 1);

}  // namespace bitcos
