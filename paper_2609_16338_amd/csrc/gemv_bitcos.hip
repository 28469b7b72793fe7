// BITCOS ternary GEMV for gfx950 (MI355X): y = (S (.) W) x at batch 1.
//
// Layout (Sec. II-A of "Breaking the 1.58-bit Barrier for Ternary LLMs"): a
// presence bitmap with one bit per weight and a sign stream with one bit per
// non-zero, both in row-major order.  The paper's x86 kernels scatter the
// compact signs with pdep and its Xe2 kernel with a nibble lookup table
// (Sec. II-B..D).  CDNA has neither pdep nor the Xe2 block loads, so this
// kernel is organised around the wavefront instead:
//
//   * Work split.  A wave step covers R = 64 / SEG consecutive rows; a row is
//     split over SEG lanes and every lane owns W consecutive 32-weight words
//     of it, so its activations stay in VGPRs for the whole kernel.
//   * Sign cursor.  Rows are consecutive in the sign stream and lanes are in
//     row-major order, so one wavefront prefix sum of the lanes' non-zero
//     counts (DPP) gives every lane its entry point; the unit offset stored in
//     the blob gives the wave's.  Inside a lane, each word's window starts at
//     the lane's entry plus the popcounts of its earlier words (Sec. II-D
//     keeps the block count separate from the per-group count for the same
//     reason: the address depends on one count per word, not on a chain).
//   * Deposit without pdep.  Per presence byte m, the 8 activations are
//     compacted onto the present positions with one v_perm_b32 pair (selector
//     table SEL[m]: byte q = position of the q-th set bit, else zero), and the
//     next 8 compact sign bits s become +-1 bytes (T[s]); one v_dot4 pair then
//     gives sum_j (1 - 2 s_j) x_{pos_j}, i.e. Eq. (2) w = p - 2n applied to
//     the activations instead of the weights.  The cursor moves by
//     popcount(m).  bf16 activations instead build +-0.5 bf16 weights with
//     v_perm_b32 from (SELB[m], TH[s]) and use v_dot2_f32_bf16; the 0.5 is
//     undone exactly at the end.
//   * Scales.  int8 dot products accumulate exactly in int32; each scale group
//     of 128 weights is multiplied once in fp32 (Sec. II-C); with one scale
//     per tensor the full int32 row sum is multiplied once.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

#include "../../include/bitcos.h"
#include "device_common.h"
#include "launch_common.h"
#include "plan.h"

namespace {

using namespace bitcos_dev;

constexpr int kModeGrouped = 1;   // one scale per (row, 128-group)
constexpr int kModeXscale = 2;    // per-group activation scales
constexpr int kModeRaw = 4;       // int32 raw row sums

struct BitcosArgs {
  const uint32_t* bitmap;
  const uint32_t* signs;
  const uint32_t* offsets;
  const uint16_t* scales;
  const void* x;
  const float* xscale;
  void* y;
  uint32_t nnz;
  int32_t n;
  int32_t nw;        // 32-weight words per row
  int32_t ngroups;   // 128-groups per row (K / 128), 0 if K % 128 != 0
  int32_t unit_rows;
  int32_t nunits;
  int32_t mode;
};

// Decode tables, one entry per byte value e.
//   sel[e]  int8 path: byte q (< popcount e) = bit position of the q-th set
//           bit of e; other bytes 0x0C (v_perm_b32 writes zero).
//   tsg[e]  int8 path: byte q = 0xFF if bit q of e is set, else 0x01.
//   selb[e] bf16 path: 16 selector bytes for 8 bf16 outputs; output b has
//           low byte 0x0C (zero) and high byte = rank of b in e if present.
//   tsh[e]  bf16 path: byte q = 0xBF if bit q of e is set, else 0x3F (the
//           high byte of -0.5 / +0.5).
struct Tables {
  uint2 sel[256];
  uint2 tsg[256];
  uint4 selb[256];
  uint2 tsh[256];
};

template <bool BF16>
__device__ __forceinline__ void build_tables(Tables& t, int e) {
  uint32_t sb[8];
  int q = 0;
#pragma unroll
  for (int b = 0; b < 8; ++b) sb[b] = 0x0C;
#pragma unroll
  for (int b = 0; b < 8; ++b)
    if (e >> b & 1) sb[q++] = b;
  uint32_t g[8];
#pragma unroll
  for (int b = 0; b < 8; ++b) g[b] = (e >> b & 1) ? (BF16 ? 0xBF : 0xFF) : (BF16 ? 0x3F : 0x01);
  if (!BF16) {
    t.sel[e] = make_uint2(bytes4(sb[0], sb[1], sb[2], sb[3]), bytes4(sb[4], sb[5], sb[6], sb[7]));
    t.tsg[e] = make_uint2(bytes4(g[0], g[1], g[2], g[3]), bytes4(g[4], g[5], g[6], g[7]));
  } else {
    uint32_t hi[8];
    int r = 0;
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      hi[b] = (e >> b & 1) ? uint32_t(r) : 0x0Cu;
      r += e >> b & 1;
    }
    t.selb[e] = make_uint4(bytes4(0x0C, hi[0], 0x0C, hi[1]), bytes4(0x0C, hi[2], 0x0C, hi[3]),
                           bytes4(0x0C, hi[4], 0x0C, hi[5]), bytes4(0x0C, hi[6], 0x0C, hi[7]));
    t.tsh[e] = make_uint2(bytes4(g[0], g[1], g[2], g[3]), bytes4(g[4], g[5], g[6], g[7]));
  }
}

// One 32-weight word, int8 activations: P presence word, S the compact signs
// of P's non-zeros (bit 0 = first non-zero), x[8] the 32 activations.
__device__ __forceinline__ int word_i8(uint32_t P, uint32_t S, const uint32_t* x, int acc,
                                       const Tables& t) {
  uint32_t r = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t m = (P >> (8 * i)) & 0xFFu;
    const uint32_t s = (S >> r) & 0xFFu;
    const uint2 sv = t.sel[m];
    const uint2 tv = t.tsg[s];
    const uint32_t c0 = __builtin_amdgcn_perm(x[2 * i + 1], x[2 * i], sv.x);
    const uint32_t c1 = __builtin_amdgcn_perm(x[2 * i + 1], x[2 * i], sv.y);
    acc = sdot4(c0, tv.x, acc);
    acc = sdot4(c1, tv.y, acc);
    r += __builtin_popcount(m);
  }
  return acc;
}

// Same word with bf16 activations (x[16] = 32 bf16): weights as +-0.5 bf16.
__device__ __forceinline__ float word_bf16(uint32_t P, uint32_t S, const uint32_t* x, float acc,
                                           const Tables& t) {
  uint32_t r = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t m = (P >> (8 * i)) & 0xFFu;
    const uint32_t s = (S >> r) & 0xFFu;
    const uint4 sb = t.selb[m];
    const uint2 th = t.tsh[s];
    acc = bdot2(__builtin_amdgcn_perm(th.y, th.x, sb.x), x[4 * i + 0], acc);
    acc = bdot2(__builtin_amdgcn_perm(th.y, th.x, sb.y), x[4 * i + 1], acc);
    acc = bdot2(__builtin_amdgcn_perm(th.y, th.x, sb.z), x[4 * i + 2], acc);
    acc = bdot2(__builtin_amdgcn_perm(th.y, th.x, sb.w), x[4 * i + 3], acc);
    r += __builtin_popcount(m);
  }
  return acc;
}

template <int W, int SEG, bool BF16>
__global__ void __launch_bounds__(kBlock) bitcos_gemv_kernel(const BitcosArgs a) {
  __shared__ Tables tab;
  build_tables<BF16>(tab, threadIdx.x);
  __syncthreads();

  const int lane = threadIdx.x & 63;
  const int wave = blockIdx.x * (kBlock / kWave) + (threadIdx.x >> 6);
  if (wave >= a.nunits) return;

  constexpr int R = kWave / SEG;
  constexpr int NX = BF16 ? 16 : 8;  // activation dwords per 32-weight word
  using Acc = typename std::conditional<BF16, float, int>::type;
  using Ends = GroupEnds<W, 4>;

  const int rho = lane / SEG;
  const int j = lane % SEG;
  const int w0 = j * W;
  const int nwl = max(0, min(W, a.nw - w0));

  uint32_t xr[W][NX];
  const uint32_t* x32 = static_cast<const uint32_t*>(a.x);
#pragma unroll
  for (int w = 0; w < W; ++w)
#pragma unroll
    for (int d = 0; d < NX; ++d) xr[w][d] = (w < nwl) ? x32[(w0 + w) * NX + d] : 0u;

  const int ph = Ends::kAligned ? 0 : (w0 & 3);
  const int g0 = w0 >> 2;
  float xs[Ends::kNQ];
#pragma unroll
  for (int q = 0; q < Ends::kNQ; ++q) {
    int g = min(g0 + q, max(a.ngroups - 1, 0));
    xs[q] = (a.mode & kModeXscale) ? a.xscale[g] : 1.0f;
  }
  const float tensor_scale = half_bits_to_float(a.scales[0]);

  const int r0 = wave * a.unit_rows;
  const int r1 = min(r0 + a.unit_rows, a.n);
  uint32_t cursor = a.offsets[wave];

  for (int rb = r0; rb < r1; rb += R) {
    const int row = rb + rho;
    const bool act = row < r1 && nwl > 0;
    const uint32_t* bm = a.bitmap + static_cast<size_t>(act ? row : 0) * a.nw + w0;
    uint32_t P[W];
    int pc[W];
    int cnt = 0;
#pragma unroll
    for (int w = 0; w < W; ++w) {
      P[w] = (act && w < nwl) ? bm[w] : 0u;
      pc[w] = cnt;
      cnt += __builtin_popcount(P[w]);
    }
    const int incl = wave_incl_scan(cnt);
    const uint32_t base = cursor + static_cast<uint32_t>(incl - cnt);
    cursor += static_cast<uint32_t>(lane63(incl));

    Acc run[W];
    Acc acc = Acc(0);
#pragma unroll
    for (int w = 0; w < W; ++w) {
      const uint32_t b = min(base + static_cast<uint32_t>(pc[w]), a.nnz);
      const uint32_t* sp = a.signs + (b >> 5);
      const uint32_t S = __builtin_amdgcn_alignbit(sp[1], sp[0], b & 31);
      if constexpr (BF16)
        acc = word_bf16(P[w], S, xr[w], acc, tab);
      else
        acc = word_i8(P[w], S, xr[w], acc, tab);
      run[w] = acc;
    }

    if (!BF16 && (a.mode & kModeRaw)) {
      const int tot = seg_sum<SEG>(static_cast<int>(run[W - 1]));
      if (j == 0 && row < r1) static_cast<int*>(a.y)[row] = tot;
      continue;
    }
    float part;
    if (!(a.mode & (kModeGrouped | kModeXscale))) {
      // One scale per tensor: reduce the exact row sum, multiply once.
      if constexpr (BF16) {
        part = seg_sum<SEG>(static_cast<float>(run[W - 1]));
        part = tensor_scale * (2.0f * part);
      } else {
        const int tot = seg_sum<SEG>(static_cast<int>(run[W - 1]));
        part = tensor_scale * static_cast<float>(tot);
      }
    } else {
      float f = 0.0f;
      Acc prev = Acc(0);
#pragma unroll
      for (int q = 0; q < Ends::kNQ; ++q) {
        const Acc e = Ends::pick(run, q, ph);
        const Acc grp = e - prev;
        prev = e;
        const int g = min(g0 + q, a.ngroups - 1);
        const float s = (a.mode & kModeGrouped)
                            ? half_bits_to_float(a.scales[static_cast<size_t>(act ? row : 0) * a.ngroups + g])
                            : tensor_scale;
        f += s * xs[q] * static_cast<float>(grp);
      }
      part = seg_sum<SEG>(BF16 ? 2.0f * f : f);
    }
    if (j == 0 && row < r1) static_cast<float*>(a.y)[row] = part;
  }
}

using KernelFn = void (*)(const BitcosArgs);

template <int SEG, bool BF16, int... Ws>
KernelFn pick_w(int w, std::integer_sequence<int, Ws...>) {
  KernelFn fn = nullptr;
  ((w == Ws + 1 ? (fn = bitcos_gemv_kernel<Ws + 1, SEG, BF16>, 0) : 0), ...);
  return fn;
}

template <bool BF16>
KernelFn pick_kernel(int per_lane, int seg) {
  constexpr int kMax = BF16 ? bitcos::kMaxWordsBf16 : bitcos::kMaxWordsI8;
  auto seq = std::make_integer_sequence<int, kMax>{};
  switch (seg) {
    case 4: return pick_w<4, BF16>(per_lane, seq);
    case 8: return pick_w<8, BF16>(per_lane, seq);
    case 16: return pick_w<16, BF16>(per_lane, seq);
    case 32: return pick_w<32, BF16>(per_lane, seq);
    case 64: return pick_w<64, BF16>(per_lane, seq);
    default: return nullptr;
  }
}

int bitcos_check(const bitcos_layout* L, int32_t m, int32_t x_dtype, int32_t y_mode,
                 bitcos::Tile* tile) {
  if (!L || L->version != BITCOS_LAYOUT_VERSION || L->format != BITCOS_FMT_BITCOS) return BITCOS_E_ARG;
  if (L->n < 1 || L->k < 32 || L->k % 32 || L->unit_rows < 1) return BITCOS_E_ARG;
  if (L->group != 0 && L->group != 128) return BITCOS_E_ARG;
  if (L->group == 128 && L->k % 128) return BITCOS_E_ARG;
  if (x_dtype != BITCOS_X_I8 && x_dtype != BITCOS_X_BF16) return BITCOS_E_ARG;
  if (y_mode != BITCOS_Y_F32 && y_mode != BITCOS_Y_I32_RAW) return BITCOS_E_ARG;
  if (y_mode == BITCOS_Y_I32_RAW && x_dtype != BITCOS_X_I8) return BITCOS_E_ARG;
  if (m != 1) return m < 1 ? BITCOS_E_ARG : BITCOS_E_UNSUPPORTED;
  if (L->nnz > 0xFFFFFFFFull) return BITCOS_E_UNSUPPORTED;
  if (!bitcos::bitcos_tile(L->k, x_dtype == BITCOS_X_BF16, tile)) return BITCOS_E_UNSUPPORTED;
  return BITCOS_OK;
}

}  // namespace

extern "C" int bitcos_gemv(const bitcos_layout* L, const void* blob_dev, int32_t m,
                           const void* x_dev, int32_t x_dtype, const float* xscale_dev,
                           void* y_dev, int32_t y_mode, void* stream) {
  bitcos::Tile tile;
  int st = bitcos_check(L, m, x_dtype, y_mode, &tile);
  if (st) return st;
  if (!blob_dev || !x_dev || !y_dev) return BITCOS_E_ARG;
  if (xscale_dev && L->k % 128) return BITCOS_E_ARG;
  const bool bf16 = x_dtype == BITCOS_X_BF16;
  KernelFn fn = bf16 ? pick_kernel<true>(tile.per_lane, tile.seg)
                     : pick_kernel<false>(tile.per_lane, tile.seg);
  if (!fn) return BITCOS_E_UNSUPPORTED;

  const uint8_t* blob = static_cast<const uint8_t*>(blob_dev);
  BitcosArgs a;
  a.bitmap = reinterpret_cast<const uint32_t*>(blob + L->sec_off[BITCOS_SEC_BITMAP]);
  a.signs = reinterpret_cast<const uint32_t*>(blob + L->sec_off[BITCOS_SEC_SIGNS]);
  a.offsets = reinterpret_cast<const uint32_t*>(blob + L->sec_off[BITCOS_SEC_OFFSETS]);
  a.scales = reinterpret_cast<const uint16_t*>(blob + L->sec_off[BITCOS_SEC_SCALES]);
  a.x = x_dev;
  a.xscale = xscale_dev;
  a.y = y_dev;
  a.nnz = static_cast<uint32_t>(L->nnz);
  a.n = L->n;
  a.nw = L->k / 32;
  a.ngroups = L->k / 128;
  a.unit_rows = L->unit_rows;
  a.nunits = (L->n + L->unit_rows - 1) / L->unit_rows;
  a.mode = (L->group == 128 ? kModeGrouped : 0) | (xscale_dev ? kModeXscale : 0) |
           (y_mode == BITCOS_Y_I32_RAW ? kModeRaw : 0);
  const int waves_per_block = kBlock / kWave;
  const int blocks = (a.nunits + waves_per_block - 1) / waves_per_block;
  hipLaunchKernelGGL(fn, dim3(blocks), dim3(kBlock), 0, static_cast<hipStream_t>(stream), a);
  return bitcos_launch_status();
}

extern "C" int bitcos_describe_bitcos(const bitcos_layout* L, int32_t m, int32_t x_dtype,
                                      bitcos_launch_info* out) {
  bitcos::Tile tile;
  int st = bitcos_check(L, m, x_dtype, BITCOS_Y_F32, &tile);
  if (st) return st;
  const int64_t nunits = (L->n + L->unit_rows - 1) / L->unit_rows;
  out->per_lane = tile.per_lane;
  out->seg_lanes = tile.seg;
  out->rows_per_step = tile.rows;
  out->lanes_used = tile.lanes;
  out->waves = nunits;
  out->workgroups = (nunits + 3) / 4;
  return BITCOS_OK;
}
