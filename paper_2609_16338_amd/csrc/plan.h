// Host-side kernel planning shared by the packers (default unit size) and the
// GEMV launchers (tile choice).  Pure C++; no HIP types.
#pragma once

#include <cstdint>

namespace bitcos {

// A GEMV wave covers `rows` = 64 / seg rows per step (rounded down).  Each row
// is split over `lanes` <= seg lanes; every lane owns `per_lane` consecutive
// units of the row (32-weight words for BITCOS, 128-weight blocks for
// five-trit, 16-weight words for 2-bit).  `seg` is a power of two, so a row's
// partial sums reduce with butterflies inside an aligned lane segment, except
// for the five-trit kernel's 20-lane segment (three rows, 60 lanes).
struct Tile {
  int per_lane = 0;
  int seg = 0;
  int rows = 0;
  int lanes = 0;
};

// Largest per-lane count that has a compiled kernel, by activation type.
constexpr int kMaxWordsI8 = 16;    // BITCOS: x in VGPRs, 8 dwords per 32-weight word
constexpr int kMaxWordsBf16 = 8;   // BITCOS: 16 dwords per word
constexpr int kMaxBlocksI8 = 4;    // five-trit: 32 dwords per 128-weight block (five blocks spill)
constexpr int kMaxBlocksBf16 = 2;  // five-trit: 64 dwords per block
constexpr int kMaxWords2I8 = 32;   // 2-bit: 4 dwords per 16-weight word
// 2-bit with int8 activations takes at most this many words per lane when a
// tile fits (27 words at K = 6912 hold about 250 registers, two waves per
// SIMD, and measured 6 % slower per BitNet-like step than 7 words), and up to
// kMaxWords2I8 only for rows no such tile covers.
constexpr int kSoftWords2I8 = 16;
constexpr int kMaxWords2Bf16 = 16; // 2-bit: 8 dwords per word

// Pick the tile that leaves the fewest lanes of the wave idle for
// `units_per_row` units split into chunks of at most `max_per_lane`; ties go
// to the smaller per-lane count (fewer registers), or with `wide` to the
// larger one (more rows per wave step).  `seg20` also offers the 20-lane
// segment: the five-trit kernel holds at most two (bf16) or four (int8)
// blocks' activations per lane, so rows of 20 or 40 blocks (K = 2560, 5120)
// would otherwise leave up to 3/8 of the lanes idle.  Returns false if no
// tile fits.
inline bool choose_tile(int units_per_row, int max_per_lane, Tile* t, bool wide = false, bool seg20 = false) {
  double best = -1.0;
  Tile pick;
  constexpr int kSegs[6] = {64, 32, 20, 16, 8, 4};
  for (int seg : kSegs) {
    if (seg == 20 && !seg20) continue;
    int per_lane = (units_per_row + seg - 1) / seg;
    if (per_lane < 1) per_lane = 1;
    if (per_lane > max_per_lane) continue;
    int lanes = (units_per_row + per_lane - 1) / per_lane;
    double util = double(units_per_row) * double(64 / seg) / double(64 * per_lane);
    bool better = util > best + 1e-12 ||
                  (util > best - 1e-12 && (wide ? per_lane > pick.per_lane : per_lane < pick.per_lane));
    if (better) {
      best = util;
      pick.per_lane = per_lane;
      pick.seg = seg;
      pick.rows = 64 / seg;
      pick.lanes = lanes;
    }
  }
  if (best < 0) return false;
  *t = pick;
  return true;
}

// BITCOS tile for (K, activation type): words of 32 weights.  Among the
// tiles of up to 8 words per lane that leave the fewest lanes idle, the
// widest: a wave step then covers more rows and each lane more words, over
// which the step's fixed work (prefix of the row's counts, sign offsets,
// row sums) is spread; at K = 4096 eight words per lane on 16-lane rows run
// the Qwen3-8B-like set 16 % (int8) and 8 % (bf16) faster than two words on
// 64-lane rows, and sixteen words per lane are slower again.  bf16 takes the
// widest of those tiles with at most 5 words per lane when there is one
// (its kernels then run 3 waves per SIMD instead of 2): 4 words on 32-lane
// rows at K = 4096 and on 64-lane rows at K = 8192 measured 4-6 % faster
// than 8 words.  Longer rows (int8 K > 16384) take up to 16 words.
inline bool bitcos_tile(int k, bool bf16, Tile* t) {
  constexpr int kWideWords = 8;
  constexpr int kWordsAt3Waves = 5;  // bf16: most words per lane at 3 waves per SIMD
  Tile wide;
  if (!choose_tile(k / 32, kWideWords, &wide, true))
    return choose_tile(k / 32, bf16 ? kMaxWordsBf16 : kMaxWordsI8, t);
  Tile narrow;
  const auto idle_free = [&](const Tile& x) { return double(k / 32) / double(x.seg * x.per_lane); };
  if (bf16 && choose_tile(k / 32, kWordsAt3Waves, &narrow, true) && idle_free(narrow) > idle_free(wide) - 1e-12) {
    *t = narrow;
    return true;
  }
  *t = wide;
  return true;
}

// Default rows per sign offset: one, so every kernel (any rows per wave step,
// the batched MFMA kernel's 16-row tiles) finds each row's entry point; 4
// bytes of metadata per row.
inline int bitcos_default_unit_rows(int n, int k) {
  (void)n;
  (void)k;
  return 1;
}

// BITCOS layout (section placement, sizes, payload bits) of an n x k matrix
// with `nnz` non-zeros; unit_rows 0 = the default.  Shared by the host and
// device packers so both place every section identically.  Defined in
// host.cpp.
int bitcos_layout_for(int32_t n, int32_t k, int32_t group, int32_t unit_rows, uint64_t nnz,
                      struct bitcos_layout* out);

}  // namespace bitcos
