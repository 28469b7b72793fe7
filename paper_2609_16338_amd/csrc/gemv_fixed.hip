// Same-GPU baselines for the BITCOS GEMV: five trits per byte (26 bytes per
// 128 weights, Sec. I of "Breaking the 1.58-bit Barrier for Ternary LLMs")
// and 2 bits per weight (Table I's 2-bit column).  Both use the BITCOS
// kernel's work split (a wave step covers 64 / SEG rows; each lane owns
// consecutive units of a row with its activations in VGPRs) so the three
// kernels differ only in how they turn bytes into weights.
//
//   five-trit  per byte, one LDS lookup gives its five weights as int8 (or
//              bf16); four lookup tables hold the same five values shifted by
//              0..3 bytes so that four consecutive bytes (20 weights) OR
//              together into five dot4 operands without any shuffling.
//   2-bit      code c = w + 1 sits in bit pairs laid out so that
//              (word >> 2t) & 0x03030303 are four consecutive codes: one
//              v_dot4 each, minus the activation sum once per word.  bf16
//              activations look up four bf16 weights per code byte.
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

constexpr int kModeGrouped = 1;
constexpr int kModeXscale = 2;
constexpr int kModeRaw = 4;

constexpr int kMaxBlocksI8 = 5;    // five-trit: 128-weight blocks per lane
constexpr int kMaxBlocksBf16 = 2;
constexpr int kMaxWords2I8 = 32;   // 2-bit: 16-weight words per lane
constexpr int kMaxWords2Bf16 = 16;

struct FixedArgs {
  const uint8_t* codes;
  const uint16_t* scales;
  const void* x;
  const float* xscale;
  void* y;
  int32_t n;
  int32_t units;      // units per row (five-trit blocks or 2-bit words)
  int32_t ngroups;    // K / 128
  int32_t rows_per_wave;
  int32_t nwaves;
  int32_t mode;
  uint32_t last_dword;  // last readable dword index of the code section
};

// Common epilogue: reduce the lane partials of one row and store.
template <int SEG, bool BF16, int PER, int UPG, class Acc>
__device__ __forceinline__ void finish_row(const FixedArgs& a, const Acc (&run)[PER], int row,
                                           bool live, int j, int ph, int g0, const float* xs,
                                           float tensor_scale, float wscale) {
  using Ends = GroupEnds<PER, UPG>;
  if (!BF16 && (a.mode & kModeRaw)) {
    const int tot = seg_sum<SEG>(static_cast<int>(run[PER - 1]));
    if (j == 0 && live) static_cast<int*>(a.y)[row] = tot;
    return;
  }
  float part;
  if (!(a.mode & (kModeGrouped | kModeXscale))) {
    if constexpr (BF16) {
      part = tensor_scale * (wscale * seg_sum<SEG>(static_cast<float>(run[PER - 1])));
    } else {
      part = tensor_scale * static_cast<float>(seg_sum<SEG>(static_cast<int>(run[PER - 1])));
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
                          ? half_bits_to_float(a.scales[static_cast<size_t>(live ? row : 0) * a.ngroups + g])
                          : tensor_scale;
      f += s * xs[q] * static_cast<float>(grp);
    }
    part = seg_sum<SEG>(wscale * f);
  }
  if (j == 0 && live) static_cast<float*>(a.y)[row] = part;
}

// ---------------------------------------------------------------------------
// Five-trit
// ---------------------------------------------------------------------------

// tab[p][v]: the five weights of byte value v (digits base 3, digit = w + 1,
// first weight in the lowest digit) as int8, placed at byte offset p of an
// 8-byte entry.  Values 243..255 are not produced by the packer: all zero.
struct Trit5TablesI8 {
  uint2 t[4][256];
};
// bf16 variant: five bf16 weights starting at element 0 or 1 of a 16-byte
// entry (an even byte of a block starts on a dword, an odd one half-way in).
struct Trit5TablesBf16 {
  uint4 t[2][256];
};

__device__ __forceinline__ void trit5_digits(int v, int (&w)[5]) {
  bool ok = v < 243;
#pragma unroll
  for (int t = 0; t < 5; ++t) {
    w[t] = ok ? (v % 3) - 1 : 0;
    v /= 3;
  }
}

__device__ __forceinline__ void build_trit5_i8(Trit5TablesI8& tb, int v) {
  int w[5];
  trit5_digits(v, w);
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    uint32_t b[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int t = 0; t < 5; ++t) b[p + t] = uint32_t(w[t]) & 0xFF;
    tb.t[p][v] = make_uint2(bytes4(b[0], b[1], b[2], b[3]), bytes4(b[4], b[5], b[6], b[7]));
  }
}

__device__ __forceinline__ void build_trit5_bf16(Trit5TablesBf16& tb, int v) {
  int w[5];
  trit5_digits(v, w);
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    uint32_t h[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int t = 0; t < 5; ++t) h[p + t] = w[t] == 0 ? 0u : (w[t] > 0 ? 0x3F80u : 0xBF80u);
    tb.t[p][v] = make_uint4(h[0] | h[1] << 16, h[2] | h[3] << 16, h[4] | h[5] << 16, h[6] | h[7] << 16);
  }
}

// Byte i of the lane's aligned code stream A.
template <int NA>
__device__ __forceinline__ uint32_t code_byte(const uint32_t (&A)[NA], int i) {
  return (A[i >> 2] >> (8 * (i & 3))) & 0xFFu;
}

template <int BK, int SEG, bool BF16>
__global__ void __launch_bounds__(kBlock) trit5_gemv_kernel(const FixedArgs a) {
  using Tables = typename std::conditional<BF16, Trit5TablesBf16, Trit5TablesI8>::type;
  __shared__ Tables tab;
  if constexpr (BF16)
    build_trit5_bf16(tab, threadIdx.x);
  else
    build_trit5_i8(tab, threadIdx.x);
  __syncthreads();

  const int lane = threadIdx.x & 63;
  const int wave = blockIdx.x * (kBlock / kWave) + (threadIdx.x >> 6);
  if (wave >= a.nwaves) return;

  constexpr int R = kWave / SEG;
  constexpr int NX = BF16 ? 64 : 32;             // activation dwords per block
  constexpr int ND = (2 + 26 * BK + 3) / 4 + 1;  // code dwords loaded per lane
  using Acc = typename std::conditional<BF16, float, int>::type;

  const int rho = lane / SEG;
  const int j = lane % SEG;
  const int b0 = j * BK;
  const int nbl = max(0, min(BK, a.units - b0));

  uint32_t xr[BK][NX];
  const uint32_t* x32 = static_cast<const uint32_t*>(a.x);
#pragma unroll
  for (int t = 0; t < BK; ++t)
#pragma unroll
    for (int d = 0; d < NX; ++d) xr[t][d] = (t < nbl) ? x32[(b0 + t) * NX + d] : 0u;

  float xs[BK];
#pragma unroll
  for (int t = 0; t < BK; ++t) {
    int g = min(b0 + t, a.ngroups - 1);
    xs[t] = (a.mode & kModeXscale) ? a.xscale[g] : 1.0f;
  }
  const float tensor_scale = half_bits_to_float(a.scales[0]);

  const int r0 = wave * a.rows_per_wave;
  const int r1 = min(r0 + a.rows_per_wave, a.n);
  for (int rb = r0; rb < r1; rb += R) {
    const int row = rb + rho;
    const bool live = row < r1;
    const bool act = live && nbl > 0;
    const uint64_t start = (static_cast<uint64_t>(act ? row : 0) * a.units + b0) * 26u;
    const uint32_t o = static_cast<uint32_t>(start & 3u);
    const uint32_t d0 = static_cast<uint32_t>(start >> 2);
    const uint32_t* c32 = reinterpret_cast<const uint32_t*>(a.codes);
    uint32_t cw[ND];
#pragma unroll
    for (int d = 0; d < ND; ++d) cw[d] = act ? c32[min(d0 + d, a.last_dword)] : 0u;
    uint32_t A[ND - 1];
#pragma unroll
    for (int d = 0; d < ND - 1; ++d) A[d] = __builtin_amdgcn_alignbyte(cw[d + 1], cw[d], o);

    Acc run[BK];
    Acc acc = Acc(0);
#pragma unroll
    for (int t = 0; t < BK; ++t) {
      const uint32_t* x = xr[t];
      if constexpr (!BF16) {
#pragma unroll
        for (int c = 0; c < 6; ++c) {
          const uint2 e0 = tab.t[0][code_byte(A, 26 * t + 4 * c + 0)];
          const uint2 e1 = tab.t[1][code_byte(A, 26 * t + 4 * c + 1)];
          const uint2 e2 = tab.t[2][code_byte(A, 26 * t + 4 * c + 2)];
          const uint2 e3 = tab.t[3][code_byte(A, 26 * t + 4 * c + 3)];
          acc = sdot4(e0.x, x[5 * c + 0], acc);
          acc = sdot4(e0.y | e1.x, x[5 * c + 1], acc);
          acc = sdot4(e1.y | e2.x, x[5 * c + 2], acc);
          acc = sdot4(e2.y | e3.x, x[5 * c + 3], acc);
          acc = sdot4(e3.y, x[5 * c + 4], acc);
        }
        const uint2 e0 = tab.t[0][code_byte(A, 26 * t + 24)];
        const uint2 e1 = tab.t[1][code_byte(A, 26 * t + 25)];
        acc = sdot4(e0.x, x[30], acc);
        acc = sdot4(e0.y | e1.x, x[31], acc);
      } else {
#pragma unroll
        for (int c = 0; c < 13; ++c) {
          const uint4 e0 = tab.t[0][code_byte(A, 26 * t + 2 * c + 0)];
          const uint4 e1 = tab.t[1][code_byte(A, 26 * t + 2 * c + 1)];
          acc = bdot2(e0.x, x[5 * c + 0], acc);
          acc = bdot2(e0.y, x[5 * c + 1], acc);
          acc = bdot2(e0.z | e1.x, x[5 * c + 2], acc);
          acc = bdot2(e1.y, x[5 * c + 3], acc);
          if (c < 12) acc = bdot2(e1.z, x[5 * c + 4], acc);  // weights 128, 129 do not exist
        }
      }
      run[t] = acc;
    }
    finish_row<SEG, BF16, BK, 1>(a, run, row, live, j, 0, b0, xs, tensor_scale, 1.0f);
  }
}

// ---------------------------------------------------------------------------
// 2-bit
// ---------------------------------------------------------------------------

// bf16 table: code byte v holds weights k0+b, k0+4+b, k0+8+b, k0+12+b (bit
// pairs 0..3); entry = those four weights as bf16, pairs (t0,t1), (t2,t3).
struct Bit2TablesBf16 {
  uint2 t[256];
};

__device__ __forceinline__ void build_bit2_bf16(Bit2TablesBf16& tb, int v) {
  uint32_t h[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    int c = (v >> (2 * t)) & 3;
    h[t] = c == 0 ? 0xBF80u : (c == 2 ? 0x3F80u : 0u);
  }
  tb.t[v] = make_uint2(h[0] | h[1] << 16, h[2] | h[3] << 16);
}

template <int WB, int SEG, bool BF16>
__global__ void __launch_bounds__(kBlock) bit2_gemv_kernel(const FixedArgs a) {
  __shared__ Bit2TablesBf16 tab;
  if constexpr (BF16) {
    build_bit2_bf16(tab, threadIdx.x);
    __syncthreads();
  }

  const int lane = threadIdx.x & 63;
  const int wave = blockIdx.x * (kBlock / kWave) + (threadIdx.x >> 6);
  if (wave >= a.nwaves) return;

  constexpr int R = kWave / SEG;
  constexpr int NX = BF16 ? 8 : 4;  // activation dwords per 16-weight word
  using Acc = typename std::conditional<BF16, float, int>::type;
  using Ends = GroupEnds<WB, 8>;

  const int rho = lane / SEG;
  const int j = lane % SEG;
  const int u0 = j * WB;
  const int nul = max(0, min(WB, a.units - u0));

  // int8: x in natural order; the per-word activation sum corrects c = w + 1.
  // bf16: x permuted to match the code bytes: dword 2b + h holds
  // (x[k0 + 8h + b], x[k0 + 8h + 4 + b]).
  uint32_t xr[WB][NX];
  int xsum[WB];
#pragma unroll
  for (int w = 0; w < WB; ++w) {
    const bool ok = w < nul;
    if constexpr (!BF16) {
      const uint32_t* x32 = static_cast<const uint32_t*>(a.x) + (u0 + w) * 4;
      int s = 0;
#pragma unroll
      for (int d = 0; d < 4; ++d) {
        xr[w][d] = ok ? x32[d] : 0u;
        s = sdot4(xr[w][d], 0x01010101u, s);
      }
      xsum[w] = s;
    } else {
      const uint16_t* x16 = static_cast<const uint16_t*>(a.x) + (u0 + w) * 16;
#pragma unroll
      for (int b = 0; b < 4; ++b)
#pragma unroll
        for (int h = 0; h < 2; ++h)
          xr[w][2 * b + h] = ok ? (uint32_t(x16[8 * h + b]) | uint32_t(x16[8 * h + 4 + b]) << 16) : 0u;
      xsum[w] = 0;
    }
  }

  const int ph = Ends::kAligned ? 0 : (u0 & 7);
  const int g0 = u0 >> 3;
  float xs[Ends::kNQ];
#pragma unroll
  for (int q = 0; q < Ends::kNQ; ++q) {
    int g = min(g0 + q, a.ngroups - 1);
    xs[q] = (a.mode & kModeXscale) ? a.xscale[g] : 1.0f;
  }
  const float tensor_scale = half_bits_to_float(a.scales[0]);

  const uint32_t* c32 = reinterpret_cast<const uint32_t*>(a.codes);
  const int r0 = wave * a.rows_per_wave;
  const int r1 = min(r0 + a.rows_per_wave, a.n);
  for (int rb = r0; rb < r1; rb += R) {
    const int row = rb + rho;
    const bool live = row < r1;
    const bool act = live && nul > 0;
    const uint32_t* cp = c32 + static_cast<size_t>(act ? row : 0) * a.units + u0;
    Acc run[WB];
    Acc acc = Acc(0);
#pragma unroll
    for (int w = 0; w < WB; ++w) {
      const uint32_t c = (act && w < nul) ? cp[w] : 0x55555555u;  // code 1 = weight 0
      if constexpr (!BF16) {
        acc -= xsum[w];
        acc = sdot4(c & 0x03030303u, xr[w][0], acc);
        acc = sdot4((c >> 2) & 0x03030303u, xr[w][1], acc);
        acc = sdot4((c >> 4) & 0x03030303u, xr[w][2], acc);
        acc = sdot4((c >> 6) & 0x03030303u, xr[w][3], acc);
      } else {
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const uint2 e = tab.t[(c >> (8 * b)) & 0xFFu];
          acc = bdot2(e.x, xr[w][2 * b + 0], acc);
          acc = bdot2(e.y, xr[w][2 * b + 1], acc);
        }
      }
      run[w] = acc;
    }
    finish_row<SEG, BF16, WB, 8>(a, run, row, live, j, ph, g0, xs, tensor_scale, 1.0f);
  }
}

// ---------------------------------------------------------------------------
// Launch plumbing
// ---------------------------------------------------------------------------

using KernelFn = void (*)(const FixedArgs);

template <template <int, int, bool> class K, int SEG, bool BF16, int... Ps>
KernelFn pick_p(int p, std::integer_sequence<int, Ps...>) {
  KernelFn fn = nullptr;
  ((p == Ps + 1 ? (fn = K<Ps + 1, SEG, BF16>::fn, 0) : 0), ...);
  return fn;
}

template <int BK, int SEG, bool BF16>
struct Trit5K {
  static constexpr KernelFn fn = trit5_gemv_kernel<BK, SEG, BF16>;
};
template <int WB, int SEG, bool BF16>
struct Bit2K {
  static constexpr KernelFn fn = bit2_gemv_kernel<WB, SEG, BF16>;
};

template <template <int, int, bool> class K, bool BF16, int MAX>
KernelFn pick_kernel(int per_lane, int seg) {
  auto seq = std::make_integer_sequence<int, MAX>{};
  switch (seg) {
    case 4: return pick_p<K, 4, BF16>(per_lane, seq);
    case 8: return pick_p<K, 8, BF16>(per_lane, seq);
    case 16: return pick_p<K, 16, BF16>(per_lane, seq);
    case 32: return pick_p<K, 32, BF16>(per_lane, seq);
    case 64: return pick_p<K, 64, BF16>(per_lane, seq);
    default: return nullptr;
  }
}

int fixed_check(const bitcos_layout* L, uint32_t fmt, int32_t m, int32_t x_dtype, int32_t y_mode,
                bitcos::Tile* tile) {
  if (!L || L->version != BITCOS_LAYOUT_VERSION || L->format != fmt) return BITCOS_E_ARG;
  if (L->n < 1 || L->k < 128 || L->k % 128) return BITCOS_E_ARG;
  if (L->group != 0 && L->group != 128) return BITCOS_E_ARG;
  if (x_dtype != BITCOS_X_I8 && x_dtype != BITCOS_X_BF16) return BITCOS_E_ARG;
  if (y_mode != BITCOS_Y_F32 && y_mode != BITCOS_Y_I32_RAW) return BITCOS_E_ARG;
  if (y_mode == BITCOS_Y_I32_RAW && x_dtype != BITCOS_X_I8) return BITCOS_E_ARG;
  if (m != 1) return m < 1 ? BITCOS_E_ARG : BITCOS_E_UNSUPPORTED;
  const bool bf16 = x_dtype == BITCOS_X_BF16;
  bool ok;
  if (fmt == BITCOS_FMT_TRIT5)
    ok = bitcos::choose_tile(L->k / 128, bf16 ? kMaxBlocksBf16 : kMaxBlocksI8, tile);
  else
    ok = bitcos::choose_tile(L->k / 16, bf16 ? kMaxWords2Bf16 : kMaxWords2I8, tile);
  return ok ? BITCOS_OK : BITCOS_E_UNSUPPORTED;
}

// Rows per wave: one wave step, as for the BITCOS default unit.
int fixed_rows_per_wave(const bitcos::Tile& t) { return t.rows; }

int fixed_gemv(uint32_t fmt, const bitcos_layout* L, const void* blob_dev, int32_t m,
               const void* x_dev, int32_t x_dtype, const float* xscale_dev, void* y_dev,
               int32_t y_mode, void* stream) {
  bitcos::Tile tile;
  int st = fixed_check(L, fmt, m, x_dtype, y_mode, &tile);
  if (st) return st;
  if (!blob_dev || !x_dev || !y_dev) return BITCOS_E_ARG;
  const bool bf16 = x_dtype == BITCOS_X_BF16;
  KernelFn fn;
  if (fmt == BITCOS_FMT_TRIT5)
    fn = bf16 ? pick_kernel<Trit5K, true, kMaxBlocksBf16>(tile.per_lane, tile.seg)
              : pick_kernel<Trit5K, false, kMaxBlocksI8>(tile.per_lane, tile.seg);
  else
    fn = bf16 ? pick_kernel<Bit2K, true, kMaxWords2Bf16>(tile.per_lane, tile.seg)
              : pick_kernel<Bit2K, false, kMaxWords2I8>(tile.per_lane, tile.seg);
  if (!fn) return BITCOS_E_UNSUPPORTED;
  const uint8_t* blob = static_cast<const uint8_t*>(blob_dev);
  FixedArgs a;
  a.codes = blob + L->sec_off[BITCOS_SEC_CODES];
  a.scales = reinterpret_cast<const uint16_t*>(blob + L->sec_off[BITCOS_SEC_SCALES]);
  a.x = x_dev;
  a.xscale = xscale_dev;
  a.y = y_dev;
  a.n = L->n;
  a.units = fmt == BITCOS_FMT_TRIT5 ? L->k / 128 : L->k / 16;
  a.ngroups = L->k / 128;
  a.rows_per_wave = fixed_rows_per_wave(tile);
  a.nwaves = (L->n + a.rows_per_wave - 1) / a.rows_per_wave;
  a.mode = (L->group == 128 ? kModeGrouped : 0) | (xscale_dev ? kModeXscale : 0) |
           (y_mode == BITCOS_Y_I32_RAW ? kModeRaw : 0);
  a.last_dword = static_cast<uint32_t>(L->sec_bytes[BITCOS_SEC_CODES] / 4 - 1);
  const int blocks = (a.nwaves + 3) / 4;
  hipLaunchKernelGGL(fn, dim3(blocks), dim3(kBlock), 0, static_cast<hipStream_t>(stream), a);
  return bitcos_launch_status();
}

int fixed_describe(uint32_t fmt, const bitcos_layout* L, int32_t m, int32_t x_dtype,
                   bitcos_launch_info* out) {
  bitcos::Tile tile;
  int st = fixed_check(L, fmt, m, x_dtype, BITCOS_Y_F32, &tile);
  if (st) return st;
  const int rpw = fixed_rows_per_wave(tile);
  const int64_t waves = (L->n + rpw - 1) / rpw;
  out->per_lane = tile.per_lane;
  out->seg_lanes = tile.seg;
  out->rows_per_step = tile.rows;
  out->lanes_used = tile.lanes;
  out->waves = waves;
  out->workgroups = (waves + 3) / 4;
  return BITCOS_OK;
}

}  // namespace

extern "C" int bitcos_describe_bitcos(const bitcos_layout* L, int32_t m, int32_t x_dtype,
                                      bitcos_launch_info* out);

extern "C" {

int trit5_gemv(const bitcos_layout* L, const void* blob_dev, int32_t m, const void* x_dev,
               int32_t x_dtype, const float* xscale_dev, void* y_dev, int32_t y_mode,
               void* stream) {
  return fixed_gemv(BITCOS_FMT_TRIT5, L, blob_dev, m, x_dev, x_dtype, xscale_dev, y_dev, y_mode,
                    stream);
}

int bit2_gemv(const bitcos_layout* L, const void* blob_dev, int32_t m, const void* x_dev,
              int32_t x_dtype, const float* xscale_dev, void* y_dev, int32_t y_mode,
              void* stream) {
  return fixed_gemv(BITCOS_FMT_BIT2, L, blob_dev, m, x_dev, x_dtype, xscale_dev, y_dev, y_mode,
                    stream);
}

int bitcos_describe(const bitcos_layout* L, int32_t m, int32_t x_dtype, bitcos_launch_info* out) {
  if (!L || !out) return BITCOS_E_ARG;
  switch (L->format) {
    case BITCOS_FMT_BITCOS: return bitcos_describe_bitcos(L, m, x_dtype, out);
    case BITCOS_FMT_TRIT5:
    case BITCOS_FMT_BIT2: return fixed_describe(L->format, L, m, x_dtype, out);
    default: return BITCOS_E_ARG;
  }
}

}  // extern "C"
