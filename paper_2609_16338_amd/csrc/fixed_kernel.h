#pragma once
// Same-GPU baselines for the BITCOS GEMV: five trits per byte (26 bytes per
// 128 weights, Sec. I of "Breaking the 1.58-bit Barrier for Ternary LLMs")
// and 2 bits per weight (Table I's 2-bit column).  Both use the BITCOS
// kernel's work split (a wave step covers 64 / SEG rows; each lane owns
// consecutive units of a row with its activations in VGPRs) so the three
// kernels differ only in how they turn bytes into weights.  Five-trit also
// has 20-lane segments (three rows per step, the last four lanes idle) for
// rows of 20 or 40 blocks, which power-of-two segments would leave up to
// 3/8 idle at the few blocks per lane its activation registers allow.
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
#include "batch.h"
#include "device_common.h"
#include "launch_common.h"
#include "plan.h"

namespace fixed_k {

using namespace bitcos_dev;
using bitcos::GemvDesc;
using bitcos::kModeGrouped;
using bitcos::kModeRaw;
using bitcos::kModeXscale;
using bitcos::kModeAdd;

struct KernelArgs {
  const GemvDesc* __restrict__ table;  // batch: descriptor table in device memory
  int64_t total_units;
  int32_t count;
  int32_t pad;
  GemvDesc one;                        // single GEMV: its descriptor
};

typedef const __attribute__((address_space(4))) GemvDesc CDesc;

template <bool TABLE>
__device__ __forceinline__ decltype(auto) desc_at(const KernelArgs& a, int di) {
  if constexpr (TABLE)
    return static_cast<CDesc&>(((CDesc*)a.table)[__builtin_amdgcn_readfirstlane(di)]);
  else
    return static_cast<const GemvDesc&>(a.one);
}

// Row range and descriptor of one unit (= one wave step of R rows).
struct Step {
  int di;
  int row0;
  int row_end;
  bool valid;
};

template <int R, bool TABLE>
struct StepGen {
  int di;
  int64_t U, Uend;

  __device__ __forceinline__ Step next(const KernelArgs& a) {
    Step s;
    s.valid = U < Uend;
    s.di = di;
    s.row0 = 0;
    s.row_end = 0;
    if (!s.valid) return s;
    if constexpr (TABLE) {
      while (di + 1 < a.count && U >= desc_at<TABLE>(a, di).unit_begin + desc_at<TABLE>(a, di).units) ++di;
      di = __builtin_amdgcn_readfirstlane(di);
    }
    const auto& g = desc_at<TABLE>(a, di);
    const int64_t u = U - g.unit_begin;
    s.di = di;
    s.row0 = static_cast<int>(u) * R;
    s.row_end = min(s.row0 + R, g.n);
    ++U;
    return s;
  }
};

// The wave's contiguous unit range of a persistent launch; returns false if empty.
template <int R, bool TABLE, int WPB = kBlock / kWave>
__device__ __forceinline__ bool wave_range(const KernelArgs& a, StepGen<R, TABLE>& gen) {
  const int wave = __builtin_amdgcn_readfirstlane(blockIdx.x * WPB + (threadIdx.x >> 6));
  const int64_t nwaves = static_cast<int64_t>(gridDim.x) * WPB;
  const int64_t per = (a.total_units + nwaves - 1) / nwaves;
  gen.U = per * wave;
  gen.Uend = min(gen.U + per, a.total_units);
  gen.di = 0;
  if constexpr (TABLE) {
    int lo = 0, hi = a.count;
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (((CDesc*)a.table)[mid].unit_begin <= gen.U) lo = mid; else hi = mid;
    }
    gen.di = __builtin_amdgcn_readfirstlane(lo);
  }
  return gen.U < gen.Uend;
}

// Common epilogue: reduce the lane partials of one row and store.  SC holds
// the row's group scales for the lane's groups (fp16 bits, grouped mode).
template <int SEG, bool BF16, int PER, int UPG, class Acc>
__device__ __forceinline__ void finish_row(int mode, void* ydst, uint32_t ybytes, const Acc (&run)[PER], int row,
                                           bool live, int j, int ph, const float* xs,
                                           const uint16_t* SC, float tensor_scale) {
  using Ends = GroupEnds<PER, UPG>;
  const bool add = (mode & kModeAdd) != 0;
  if (!BF16 && (mode & kModeRaw)) {
    const int tot = seg_sum<SEG>(static_cast<int>(run[PER - 1]));
    if (j == SEG - 1 && live) put_y(static_cast<uint32_t>(tot), make_rsrc(ydst, ybytes), 4u * row, 0, add, true);
    return;
  }
  float part;
  if (!(mode & (kModeGrouped | kModeXscale))) {
    if constexpr (BF16) {
      part = tensor_scale * seg_sum<SEG>(static_cast<float>(run[PER - 1]));
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
      const float s = (mode & kModeGrouped) ? half_bits_to_float(SC[q]) : tensor_scale;
      f += s * xs[q] * static_cast<float>(grp);
    }
    part = seg_sum<SEG>(f);
  }
  if (j == SEG - 1 && live) put_y(__builtin_bit_cast(uint32_t, part), make_rsrc(ydst, ybytes), 4u * row, 0, add, false);
}

// The lane's group scales for one row (grouped mode), else zeros.
template <int NQ, class G>
__device__ __forceinline__ void load_row_scales(const G& g, int row, bool act, int g0,
                                                uint16_t (&SC)[NQ]) {
  const bool grouped = (g.mode & kModeGrouped) != 0;
  const rsrc_t rs = make_rsrc(g.scales, g.scales_bytes);
  const uint32_t soff = (act && grouped) ? static_cast<uint32_t>(row) * g.ngroups * 2u : kOOB;
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int gi = min(g0 + q, max(g.ngroups - 1, 0));
    SC[q] = ld16(rs, soff + 2u * gi);
  }
}

template <int NQ, class G>
__device__ __forceinline__ void load_xscales(const G& g, int g0, float (&xs)[NQ]) {
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int gi = min(g0 + q, max(g.ngroups - 1, 0));
    xs[q] = (g.mode & kModeXscale) ? gp_f32(g.xscale)[gi] : 1.0f;
  }
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
// Each entry is kept in kTrit5Copies copies (copy c of value v at index
// v * kTrit5Copies + c; lane l reads copy l % kTrit5Copies): a ds_read_b128
// serves 16 lanes at a time, and 16 copies keep any 16 keys on distinct
// banks, where a single copy serialises lanes whose values share banks.
constexpr int kTrit5Copies = 16;
struct Trit5TablesBf16 {
  uint4 t[2][256 * kTrit5Copies];
};

// Workgroup size of the baselines: the five-trit bf16 kernel fills most of
// the LDS with replicated tables, so one workgroup holds a CU's waves (three
// per SIMD with one block per lane, two with two); the others run several
// 256-thread workgroups per CU.  Host and device both use it.
constexpr int fixed_threads(bool bit2, bool bf16, int per_lane) {
  return (bit2 || !bf16) ? kBlock : (per_lane == 1 ? 768 : 512);
}

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

__device__ __forceinline__ void build_trit5_bf16(Trit5TablesBf16& tb, int tid, int nthreads) {
  for (int idx = tid; idx < 256 * kTrit5Copies; idx += nthreads) {
    int w[5];
    trit5_digits(idx / kTrit5Copies, w);
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      uint32_t h[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
      for (int t = 0; t < 5; ++t) h[p + t] = w[t] == 0 ? 0u : (w[t] > 0 ? 0x3F80u : 0xBF80u);
      tb.t[p][idx] = make_uint4(h[0] | h[1] << 16, h[2] | h[3] << 16, h[4] | h[5] << 16, h[6] | h[7] << 16);
    }
  }
}

// A table entry read as one 16-byte vector.  Its fourth dword is always zero
// and unused; read through a uint4 the compiler drops it and splits the rest
// into an 8-byte and a 4-byte read, twice the LDS instructions.
typedef unsigned u32v4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ u32v4 lds_read16(const uint4* p) { return *reinterpret_cast<const u32v4*>(p); }

// Byte i of the lane's aligned code stream A.
template <int NA>
__device__ __forceinline__ uint32_t code_byte(const uint32_t (&A)[NA], int i) {
  return (A[i >> 2] >> (8 * (i & 3))) & 0xFFu;
}

template <int BK, int SEG, bool BF16, bool TABLE>
__global__ void __launch_bounds__(fixed_threads(false, BF16, BK)) trit5_gemv_kernel(const KernelArgs a) {
  using Tables = typename std::conditional<BF16, Trit5TablesBf16, Trit5TablesI8>::type;
  constexpr int WPB = fixed_threads(false, BF16, BK) / kWave;
  __shared__ Tables tab;
  if constexpr (BF16)
    build_trit5_bf16(tab, threadIdx.x, fixed_threads(false, BF16, BK));
  else
    build_trit5_i8(tab, threadIdx.x);
  __syncthreads();

  constexpr int R = kWave / SEG;
  constexpr int NX = BF16 ? 64 : 32;             // activation dwords per block
  constexpr int ND = (2 + 26 * BK + 3) / 4 + 1;  // code dwords loaded per lane
  using Acc = typename std::conditional<BF16, float, int>::type;

  StepGen<R, TABLE> gen;
  if (!wave_range<R, TABLE, WPB>(a, gen)) return;
  const int lane = threadIdx.x & 63;
  const int rho = lane / SEG;
  const int j = lane % SEG;
  const int b0 = j * BK;
  const int cpy = lane & (kTrit5Copies - 1);

  auto load_c = [&](const Step& s, uint32_t (&cw)[ND], uint32_t& o, uint16_t (&SC)[BK]) {
    const auto& g = desc_at<TABLE>(a, s.di);
    const int row = s.row0 + rho;
    const int nbl = max(0, min(BK, g.upr - b0));
    const bool act = s.valid && row < s.row_end && nbl > 0;
    const uint32_t start = (static_cast<uint32_t>(act ? row : 0) * g.upr + b0) * 26u;
    o = start & 3u;
    const uint32_t off = act ? (start & ~3u) : kOOB;
    const rsrc_t rc = make_rsrc(g.sec0, g.sec0_bytes);
#pragma unroll
    for (int d = 0; d < ND; ++d) cw[d] = ld32(rc, off + 4u * d);
    load_row_scales<BK>(g, row, act, b0, SC);
  };

  int xdi = -1;
  uint32_t xr[BK][NX];
  float xs[BK];
  float tensor_scale = 0.0f;
  int mode = 0;
  void* ydst = nullptr;
  uint32_t ybytes = 0;

  Step s1 = gen.next(a);
  uint32_t cw1[ND], o1;
  uint16_t SC1[BK];
  load_c(s1, cw1, o1, SC1);
  while (s1.valid) {
    const Step s0 = s1;
    uint32_t A[ND - 1];
#pragma unroll
    for (int d = 0; d < ND - 1; ++d) A[d] = __builtin_amdgcn_alignbyte(cw1[d + 1], cw1[d], o1);
    uint16_t SC0[BK];
#pragma unroll
    for (int t = 0; t < BK; ++t) SC0[t] = SC1[t];
    if (s0.di != xdi) {
      xdi = s0.di;
      const auto& g = desc_at<TABLE>(a, xdi);
      const int nbl = max(0, min(BK, g.upr - b0));
      const rsrc_t rx = make_rsrc(g.x, g.x_bytes);
#pragma unroll
      for (int t = 0; t < BK; ++t) {
        const uint32_t off = t < nbl ? static_cast<uint32_t>(b0 + t) * NX * 4u : kOOB;
#pragma unroll
        for (int d = 0; d < NX; ++d) xr[t][d] = ld32(rx, off + 4u * d);
      }
      load_xscales<BK>(g, b0, xs);
      tensor_scale = half_bits_to_float(gp_u16(g.scales)[0]);
      mode = g.mode;
      ydst = g.y;
      ybytes = g.y_bytes;
      wait_vmem_all();
    }
    // The next step's loads, issued after the activations of a GEMV the wave
    // enters have been waited for, so that no wait inside the step covers them.
    s1 = gen.next(a);
    if (s1.valid) load_c(s1, cw1, o1, SC1);

    const int row = s0.row0 + rho;
    const bool live = row < s0.row_end;
    Acc run[BK];
    Acc acc = Acc(0);
    // The decode burst at raised wave priority, as in the BITCOS kernels.
    __builtin_amdgcn_s_setprio(1);
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
          const u32v4 e0 = lds_read16(&tab.t[0][code_byte(A, 26 * t + 2 * c + 0) * kTrit5Copies + cpy]);
          const u32v4 e1 = lds_read16(&tab.t[1][code_byte(A, 26 * t + 2 * c + 1) * kTrit5Copies + cpy]);
          acc = bdot2(e0.x, x[5 * c + 0], acc);
          acc = bdot2(e0.y, x[5 * c + 1], acc);
          acc = bdot2(e0.z | e1.x, x[5 * c + 2], acc);
          acc = bdot2(e1.y, x[5 * c + 3], acc);
          if (c < 12) acc = bdot2(e1.z, x[5 * c + 4], acc);  // weights 128, 129 do not exist
          // Unscheduled, the compiler hoists all 26 table reads of a block
          // (4 registers each) and the one-block variants spill; a fence every
          // six pairs bounds the reads in flight.
          if (c % 6 == 5) __builtin_amdgcn_sched_barrier(0);
        }
      }
      run[t] = acc;
    }
    __builtin_amdgcn_s_setprio(0);
    finish_row<SEG, BF16, BK, 1>(mode, ydst, ybytes, run, row, live, j, 0, xs, SC0, tensor_scale);
  }
}

// ---------------------------------------------------------------------------
// 2-bit
// ---------------------------------------------------------------------------

// bf16 table: code byte v holds weights k0+b, k0+4+b, k0+8+b, k0+12+b (bit
// pairs 0..3); entry = those four weights as bf16, pairs (t0,t1), (t2,t3).
// Kept in kBit2Copies copies (copy c of v at index v * kBit2Copies + c, lane
// l reads copy l % kBit2Copies): a ds_read_b64 serves 32 lanes at a time;
// 16 copies (32 KB) leave room for four 256-thread workgroups per CU, which
// measured faster than 32 conflict-free copies with one 512-thread
// workgroup.
constexpr int kBit2Copies = 16;
struct Bit2TablesBf16 {
  uint2 t[256 * kBit2Copies];
};

__device__ __forceinline__ void build_bit2_bf16(Bit2TablesBf16& tb, int tid, int nthreads) {
  for (int idx = tid; idx < 256 * kBit2Copies; idx += nthreads) {
    const int v = idx / kBit2Copies;
    uint32_t h[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      int c = (v >> (2 * t)) & 3;
      h[t] = c == 0 ? 0xBF80u : (c == 2 ? 0x3F80u : 0u);
    }
    tb.t[idx] = make_uint2(h[0] | h[1] << 16, h[2] | h[3] << 16);
  }
}

template <int WB, int SEG, bool BF16, bool TABLE>
__global__ void __launch_bounds__(fixed_threads(true, BF16, WB)) bit2_gemv_kernel(const KernelArgs a) {
  constexpr int WPB = fixed_threads(true, BF16, WB) / kWave;
  __shared__ typename std::conditional<BF16, Bit2TablesBf16, char>::type tab;
  if constexpr (BF16) {
    build_bit2_bf16(tab, threadIdx.x, fixed_threads(true, BF16, WB));
    __syncthreads();
  }

  constexpr int R = kWave / SEG;
  constexpr int NX = BF16 ? 8 : 4;  // activation dwords per 16-weight word
  using Acc = typename std::conditional<BF16, float, int>::type;
  using Ends = GroupEnds<WB, 8>;
  constexpr int NQ = Ends::kNQ;

  StepGen<R, TABLE> gen;
  if (!wave_range<R, TABLE, WPB>(a, gen)) return;
  const int lane = threadIdx.x & 63;
  const int rho = lane / SEG;
  const int j = lane % SEG;
  const int u0 = j * WB;
  const int cpy = lane & (kBit2Copies - 1);
  const int ph = Ends::kAligned ? 0 : (u0 & 7);
  const int g0 = u0 >> 3;

  auto load_c = [&](const Step& s, uint32_t (&cw)[WB], uint16_t (&SC)[NQ]) {
    const auto& g = desc_at<TABLE>(a, s.di);
    const int row = s.row0 + rho;
    const int nul = max(0, min(WB, g.upr - u0));
    const bool act = s.valid && row < s.row_end && nul > 0;
    const rsrc_t rc = make_rsrc(g.sec0, g.sec0_bytes);
    const uint32_t off = act ? (static_cast<uint32_t>(row) * g.upr + u0) * 4u : kOOB;
#pragma unroll
    for (int w = 0; w < WB; ++w) {
      const uint32_t v = ld32(rc, off + 4u * w);
      cw[w] = w < nul ? v : 0x55555555u;  // code 1 = weight 0
    }
    load_row_scales<NQ>(g, row, act, g0, SC);
  };

  // int8: x in natural order; the per-word activation sum corrects c = w + 1.
  // bf16: x permuted to match the code bytes: dword 2b + h holds
  // (x[k0 + 8h + b], x[k0 + 8h + 4 + b]).
  int xdi = -1;
  uint32_t xr[WB][NX];
  int xsum[WB];
  float xs[NQ];
  float tensor_scale = 0.0f;
  int mode = 0;
  void* ydst = nullptr;
  uint32_t ybytes = 0;

  Step s1 = gen.next(a);
  uint32_t cw1[WB];
  uint16_t SC1[NQ];
  load_c(s1, cw1, SC1);
  while (s1.valid) {
    const Step s0 = s1;
    uint32_t cw0[WB];
    uint16_t SC0[NQ];
#pragma unroll
    for (int w = 0; w < WB; ++w) cw0[w] = cw1[w];
#pragma unroll
    for (int q = 0; q < NQ; ++q) SC0[q] = SC1[q];
    if (s0.di != xdi) {
      xdi = s0.di;
      const auto& g = desc_at<TABLE>(a, xdi);
      const int nul = max(0, min(WB, g.upr - u0));
#pragma unroll
      for (int w = 0; w < WB; ++w) {
        const bool ok = w < nul;
        const rsrc_t rx = make_rsrc(g.x, g.x_bytes);
        if constexpr (!BF16) {
          const uint32_t off = ok ? static_cast<uint32_t>(u0 + w) * 16u : kOOB;
          int s = 0;
#pragma unroll
          for (int d = 0; d < 4; ++d) {
            xr[w][d] = ld32(rx, off + 4u * d);
            s = sdot4(xr[w][d], 0x01010101u, s);
          }
          xsum[w] = s;
        } else {
          const uint32_t off = ok ? static_cast<uint32_t>(u0 + w) * 32u : kOOB;
#pragma unroll
          for (int b = 0; b < 4; ++b)
#pragma unroll
            for (int h = 0; h < 2; ++h)
              xr[w][2 * b + h] = uint32_t(ld16(rx, off + 2u * (8 * h + b))) |
                                 uint32_t(ld16(rx, off + 2u * (8 * h + 4 + b))) << 16;
          xsum[w] = 0;
        }
      }
      load_xscales<NQ>(g, g0, xs);
      tensor_scale = half_bits_to_float(gp_u16(g.scales)[0]);
      mode = g.mode;
      ydst = g.y;
      ybytes = g.y_bytes;
      wait_vmem_all();
    }
    // The next step's loads, issued after the activations of a GEMV the wave
    // enters have been waited for, so that no wait inside the step covers them.
    s1 = gen.next(a);
    if (s1.valid) load_c(s1, cw1, SC1);

    const int row = s0.row0 + rho;
    const bool live = row < s0.row_end;
    Acc run[WB];
    Acc acc = Acc(0);
    // The decode burst at raised wave priority, as in the BITCOS kernels.
    __builtin_amdgcn_s_setprio(1);
    if constexpr (!BF16) {
#pragma unroll
      for (int w = 0; w < WB; ++w) {
        const uint32_t c = cw0[w];
        acc -= xsum[w];
        acc = sdot4(c & 0x03030303u, xr[w][0], acc);
        acc = sdot4((c >> 2) & 0x03030303u, xr[w][1], acc);
        acc = sdot4((c >> 4) & 0x03030303u, xr[w][2], acc);
        acc = sdot4((c >> 6) & 0x03030303u, xr[w][3], acc);
        run[w] = acc;
      }
    } else {
      // The next word's four lookups are issued before this word's products,
      // so a word waits on lookups issued a word earlier, not just before use.
      auto look = [&](uint32_t c, uint2 (&e)[4]) {
#pragma unroll
        for (int b = 0; b < 4; ++b) e[b] = tab.t[((c >> (8 * b)) & 0xFFu) * kBit2Copies + cpy];
      };
      uint2 e[2][4];
      look(cw0[0], e[0]);
#pragma unroll
      for (int w = 0; w < WB; ++w) {
        if (w + 1 < WB) look(cw0[w + 1], e[(w + 1) & 1]);
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          acc = bdot2(e[w & 1][b].x, xr[w][2 * b + 0], acc);
          acc = bdot2(e[w & 1][b].y, xr[w][2 * b + 1], acc);
        }
        run[w] = acc;
      }
    }
    __builtin_amdgcn_s_setprio(0);
    finish_row<SEG, BF16, WB, 8>(mode, ydst, ybytes, run, row, live, j, ph, xs, SC0, tensor_scale);
  }
}

using KernelFn = void (*)(const KernelArgs);

template <int P, int SEG, bool BF16, bool TABLE>
struct Trit5K {
  static constexpr KernelFn fn = trit5_gemv_kernel<P, SEG, BF16, TABLE>;
};
template <int P, int SEG, bool BF16, bool TABLE>
struct Bit2K {
  static constexpr KernelFn fn = bit2_gemv_kernel<P, SEG, BF16, TABLE>;
};

template <template <int, int, bool, bool> class K, int SEG, bool BF16, bool TABLE, int... Ps>
KernelFn pick_p(int p, std::integer_sequence<int, Ps...>) {
  KernelFn fn = nullptr;
  ((p == Ps + 1 ? (fn = K<Ps + 1, SEG, BF16, TABLE>::fn, 0) : 0), ...);
  return fn;
}

template <template <int, int, bool, bool> class K, int MAX, bool BF16, bool TABLE>
KernelFn pick_kernel(int per_lane, int seg) {
  auto seq = std::make_integer_sequence<int, MAX>{};
  switch (seg) {
    case 4: return pick_p<K, 4, BF16, TABLE>(per_lane, seq);
    case 8: return pick_p<K, 8, BF16, TABLE>(per_lane, seq);
    case 16: return pick_p<K, 16, BF16, TABLE>(per_lane, seq);
    case 32: return pick_p<K, 32, BF16, TABLE>(per_lane, seq);
    case 64: return pick_p<K, 64, BF16, TABLE>(per_lane, seq);
    default: return nullptr;
  }
}

}  // namespace fixed_k
