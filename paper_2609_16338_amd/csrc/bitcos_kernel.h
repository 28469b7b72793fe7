// BITCOS ternary GEMV for gfx950 (MI355X): y = (S (.) W) x at batch 1.
//
// Layout (Sec. II-A of "Breaking the 1.58-bit Barrier for Ternary LLMs"): a
// presence bitmap with one bit per weight and a sign stream with one bit per
// non-zero, both in row-major order.  The paper's x86 kernels scatter the
// compact signs with pdep and its Xe2 kernel with a nibble lookup table
// (Sec. II-B..D).  CDNA has neither pdep nor the Xe2 block loads, so this
// kernel is organised around the 64-wide wavefront instead:
//
//   * Work split.  A wave step covers R = 64 / SEG consecutive rows; a row is
//     split over SEG lanes and every lane owns W consecutive 32-weight words
//     of it, so its activations stay in VGPRs.  Units (groups of rows with a
//     stored sign offset) of one or many matrices are numbered in one list
//     and every wave of a persistent grid takes a contiguous range of it.
//   * Sign cursor.  Rows are consecutive in the sign stream and lanes are in
//     row-major order, so one wavefront prefix sum of the lanes' non-zero
//     counts (DPP) gives every lane its entry point; the unit offset stored in
//     the blob (or the previous step's total) gives the wave's.  Inside a
//     lane, each word's window starts at the lane's entry plus the popcounts
//     of its earlier words (Sec. II-D also keeps the address count apart from
//     the per-group count, to keep the dependent chain short).
//   * Deposit without pdep.  Per presence byte m, the 8 activations are
//     compacted onto the present positions with one v_perm_b32 pair (selector
//     table SEL[m]: byte q = position of the q-th set bit, else zero), and the
//     next 8 compact sign bits s become +-1 bytes (T[s]); one v_dot4 pair then
//     gives sum_j (1 - 2 s_j) x_{pos_j}, i.e. Eq. (2) w = p - 2n applied to
//     the activations instead of the weights.  The cursor moves by
//     popcount(m).  bf16 activations instead build +-0.5 bf16 weights with
//     v_perm_b32 from (SELB[m], TH[s]) and use v_dot2_f32_bf16; the factor
//     0.5 is undone exactly at the end.
//   * Pipelining.  While step i is decoded, the sign windows of step i+1 and
//     the presence words (and group scales) of step i+2 are in flight.
//   * Scales.  int8 dot products accumulate exactly in int32; each scale group
//     of 128 weights is multiplied once in fp32 (Sec. II-C); with one scale
//     per tensor the full int32 row sum is multiplied once.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

#include "../../include/bitcos.h"
#include "batch.h"
#include "device_common.h"
#include "launch_common.h"
#include "plan.h"

namespace bitcos_k {

using namespace bitcos_dev;
using bitcos::GemvDesc;
using bitcos::kModeGrouped;
using bitcos::kModeRaw;
using bitcos::kModeXscale;
using bitcos::kModeAdd;

struct KernelArgs {
  const GemvDesc* __restrict__ table;  // batch: descriptor table in device memory
  int64_t total_units;
  int32_t count;                       // descriptors in the table
  int32_t pad;
  GemvDesc one;                        // single GEMV: its descriptor
};

// Decode tables, one entry per byte value e, each kept in NC copies: lane l
// reads copy l % NC, and copy c of every entry sits c entries past the start
// of the entry's group of copies, so lanes that read the same cycle hit
// different LDS banks whatever keys they look up.
//   sel[e]  int8 path: byte q (< popcount e) = bit position of the q-th set
//           bit of e; other bytes 0x0C (v_perm_b32 writes zero).
//   tsg[e]  int8 path: byte q = 0xFF if bit q of e is set, else 0x01.
//   selb[e] bf16 path: 16 selector bytes for 8 bf16 outputs; output b has
//           low byte 0x0C (zero) and high byte = rank of b in e if present.
//   tsh[e]  bf16 path: byte q = 0xBF if bit q of e is set, else 0x3F (the
//           high byte of -0.5 / +0.5).
template <bool BF16>
struct Cfg {
  static constexpr int kThreads = 512;  // workgroup size of the general kernel
  static constexpr int kCopies = 16;    // table copies
};

template <bool BF16>
struct Tables;
template <>
struct Tables<false> {
  uint2 sel[256 * Cfg<false>::kCopies];
  uint2 tsg[256 * Cfg<false>::kCopies];
};
template <>
struct Tables<true> {
  uint4 selb[256 * Cfg<true>::kCopies];
  uint2 tsh[256 * Cfg<true>::kCopies];
};

template <bool BF16>
__device__ __forceinline__ void build_tables(Tables<BF16>& t, int tid, int nthreads) {
  constexpr int NC = Cfg<BF16>::kCopies;
  for (int idx = tid; idx < 256 * NC; idx += nthreads) {
    const int e = idx & 255;
    const int c = idx >> 8;
    uint32_t g[8];
#pragma unroll
    for (int b = 0; b < 8; ++b) g[b] = (e >> b & 1) ? (BF16 ? 0xBF : 0xFF) : (BF16 ? 0x3F : 0x01);
    const uint2 gv = make_uint2(bytes4(g[0], g[1], g[2], g[3]), bytes4(g[4], g[5], g[6], g[7]));
    if constexpr (!BF16) {
      uint32_t sb[8];
      int q = 0;
#pragma unroll
      for (int b = 0; b < 8; ++b) sb[b] = 0x0C;
#pragma unroll
      for (int b = 0; b < 8; ++b)
        if (e >> b & 1) sb[q++] = b;
      t.sel[e * NC + c] = make_uint2(bytes4(sb[0], sb[1], sb[2], sb[3]), bytes4(sb[4], sb[5], sb[6], sb[7]));
      t.tsg[e * NC + c] = gv;
    } else {
      uint32_t hi[8];
      int r = 0;
#pragma unroll
      for (int b = 0; b < 8; ++b) {
        hi[b] = (e >> b & 1) ? uint32_t(r) : 0x0Cu;
        r += e >> b & 1;
      }
      t.selb[e * NC + c] = make_uint4(bytes4(0x0C, hi[0], 0x0C, hi[1]), bytes4(0x0C, hi[2], 0x0C, hi[3]),
                                      bytes4(0x0C, hi[4], 0x0C, hi[5]), bytes4(0x0C, hi[6], 0x0C, hi[7]));
      t.tsh[e * NC + c] = gv;
    }
  }
}

// One 32-weight word, int8 activations: P presence word, S the compact signs
// of P's non-zeros (bit 0 = first non-zero), x[8] the 32 activations; `cp`
// is this lane's table copy.  The word is split into its table lookups
// (word_look_*) and its arithmetic (word_math_*) so a caller can keep the
// next word's lookups in flight while it multiplies the current one.
struct LookI8 {
  uint2 sv[4];  // sel[m] per presence byte
  uint2 tv[4];  // tsg[s] per presence byte
};

__device__ __forceinline__ LookI8 word_look_i8(uint32_t P, uint32_t S, const Tables<false>& t, int cp) {
  constexpr int NC = Cfg<false>::kCopies;
  LookI8 L;
  uint32_t r = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t m = __builtin_amdgcn_ubfe(P, 8 * i, 8);
    const uint32_t s = __builtin_amdgcn_ubfe(S, r, 8);
    if (i < 3) r = __builtin_popcount(m) + r;
    L.sv[i] = t.sel[m * NC + cp];
    L.tv[i] = t.tsg[s * NC + cp];
  }
  return L;
}

__device__ __forceinline__ int word_math_i8(const LookI8& L, const uint32_t* x, int acc) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t c0 = __builtin_amdgcn_perm(x[2 * i + 1], x[2 * i], L.sv[i].x);
    const uint32_t c1 = __builtin_amdgcn_perm(x[2 * i + 1], x[2 * i], L.sv[i].y);
    acc = sdot4(c0, L.tv[i].x, acc);
    acc = sdot4(c1, L.tv[i].y, acc);
  }
  return acc;
}

// Byte-at-a-time form (fewest live registers), for the wide tiles.
__device__ __forceinline__ int word_i8(uint32_t P, uint32_t S, const uint32_t* x, int acc,
                                       const Tables<false>& t, int cp) {
  constexpr int NC = Cfg<false>::kCopies;
  uint32_t r = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t m = __builtin_amdgcn_ubfe(P, 8 * i, 8);
    const uint32_t s = __builtin_amdgcn_ubfe(S, r, 8);
    const uint2 sv = t.sel[m * NC + cp];
    const uint2 tv = t.tsg[s * NC + cp];
    acc = sdot4(__builtin_amdgcn_perm(x[2 * i + 1], x[2 * i], sv.x), tv.x, acc);
    acc = sdot4(__builtin_amdgcn_perm(x[2 * i + 1], x[2 * i], sv.y), tv.y, acc);
    r += __builtin_popcount(m);
  }
  return acc;
}

// Same word with bf16 activations (x[16] = 32 bf16): weights as +-0.5 bf16.
struct LookBf16 {
  uint4 sb[4];  // selb[m]
  uint2 th[4];  // tsh[s]
};

__device__ __forceinline__ LookBf16 word_look_bf16(uint32_t P, uint32_t S, const Tables<true>& t, int cp) {
  constexpr int NC = Cfg<true>::kCopies;
  LookBf16 L;
  uint32_t r = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t m = __builtin_amdgcn_ubfe(P, 8 * i, 8);
    const uint32_t s = __builtin_amdgcn_ubfe(S, r, 8);
    if (i < 3) r = __builtin_popcount(m) + r;
    L.sb[i] = t.selb[m * NC + cp];
    L.th[i] = t.tsh[s * NC + cp];
  }
  return L;
}

__device__ __forceinline__ float word_math_bf16(const LookBf16& L, const uint32_t* x, float acc) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    acc = bdot2(__builtin_amdgcn_perm(L.th[i].y, L.th[i].x, L.sb[i].x), x[4 * i + 0], acc);
    acc = bdot2(__builtin_amdgcn_perm(L.th[i].y, L.th[i].x, L.sb[i].y), x[4 * i + 1], acc);
    acc = bdot2(__builtin_amdgcn_perm(L.th[i].y, L.th[i].x, L.sb[i].z), x[4 * i + 2], acc);
    acc = bdot2(__builtin_amdgcn_perm(L.th[i].y, L.th[i].x, L.sb[i].w), x[4 * i + 3], acc);
  }
  return acc;
}

__device__ __forceinline__ float word_bf16(uint32_t P, uint32_t S, const uint32_t* x, float acc,
                                           const Tables<true>& t, int cp) {
  constexpr int NC = Cfg<true>::kCopies;
  uint32_t r = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t m = __builtin_amdgcn_ubfe(P, 8 * i, 8);
    const uint32_t s = __builtin_amdgcn_ubfe(S, r, 8);
    const uint4 sb = t.selb[m * NC + cp];
    const uint2 th = t.tsh[s * NC + cp];
    acc = bdot2(__builtin_amdgcn_perm(th.y, th.x, sb.x), x[4 * i + 0], acc);
    acc = bdot2(__builtin_amdgcn_perm(th.y, th.x, sb.y), x[4 * i + 1], acc);
    acc = bdot2(__builtin_amdgcn_perm(th.y, th.x, sb.z), x[4 * i + 2], acc);
    acc = bdot2(__builtin_amdgcn_perm(th.y, th.x, sb.w), x[4 * i + 3], acc);
    r += __builtin_popcount(m);
  }
  return acc;
}

template <bool BF16>
using Look = typename std::conditional<BF16, LookBf16, LookI8>::type;

template <bool BF16>
__device__ __forceinline__ Look<BF16> word_look(uint32_t P, uint32_t S, const Tables<BF16>& t, int cp) {
  if constexpr (BF16)
    return word_look_bf16(P, S, t, cp);
  else
    return word_look_i8(P, S, t, cp);
}

template <bool BF16, class Acc>
__device__ __forceinline__ Acc word_math(const Look<BF16>& L, const uint32_t* x, Acc acc) {
  if constexpr (BF16)
    return word_math_bf16(L, x, acc);
  else
    return word_math_i8(L, x, acc);
}

// The descriptor of GEMV `di` (a wave-uniform index): from the device table
// (batch launch) or the kernel argument (single GEMV); scalar loads either way.
typedef const __attribute__((address_space(4))) GemvDesc CDesc;

template <bool TABLE>
__device__ __forceinline__ decltype(auto) desc_at(const KernelArgs& a, int di) {
  if constexpr (TABLE)
    return static_cast<CDesc&>(((CDesc*)a.table)[__builtin_amdgcn_readfirstlane(di)]);
  else
    return static_cast<const GemvDesc&>(a.one);
}

// Wave-uniform description of one step (R rows of one unit of one GEMV).
struct Step {
  int di;            // descriptor index
  int row0;          // first row of the step
  int row_end;       // end of the unit's rows
  uint32_t cursor0;  // the unit's sign offset (first step of a unit)
  bool first;        // first step of its unit
  bool valid;
};

// Walks a wave's contiguous unit range [U, Uend) step by step.
template <int R, bool TABLE>
struct StepGen {
  int di;
  int64_t U, Uend;
  int t;

  __device__ __forceinline__ Step next(const KernelArgs& a) {
    Step s;
    s.valid = false;
    s.di = 0;
    s.row0 = 0;
    s.row_end = 0;
    s.cursor0 = 0;
    s.first = false;
    while (U < Uend) {
      if constexpr (TABLE) {
        while (di + 1 < a.count && U >= desc_at<TABLE>(a, di).unit_begin + desc_at<TABLE>(a, di).units) ++di;
        di = __builtin_amdgcn_readfirstlane(di);
      }
      const auto& g = desc_at<TABLE>(a, di);
      const int64_t u = U - g.unit_begin;
      const int ur = g.unit_rows;
      const int r0 = static_cast<int>(u) * ur + t * R;
      const int rend = min(static_cast<int>(u) * ur + ur, g.n);
      if (r0 < rend) {
        s.valid = true;
        s.di = di;
        s.row0 = r0;
        s.row_end = rend;
        s.first = t == 0;
        s.cursor0 = s.first ? cp_u32(g.offsets)[u] : 0u;
        if (r0 + R < rend) {
          ++t;
        } else {
          ++U;
          t = 0;
        }
        return s;
      }
      ++U;
      t = 0;
    }
    return s;
  }
};

template <int W, int SEG, bool BF16, bool TABLE>
__global__ void __launch_bounds__(Cfg<BF16>::kThreads) bitcos_gemv_kernel(const KernelArgs a) {
  __shared__ Tables<BF16> tab;
  build_tables<BF16>(tab, threadIdx.x, Cfg<BF16>::kThreads);
  __syncthreads();

  constexpr int R = kWave / SEG;
  constexpr int NX = BF16 ? 16 : 8;  // activation dwords per 32-weight word
  constexpr int WPB = Cfg<BF16>::kThreads / kWave;
  using Acc = typename std::conditional<BF16, float, int>::type;
  using Ends = GroupEnds<W, 4>;
  constexpr int NQ = Ends::kNQ;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(blockIdx.x * WPB + (threadIdx.x >> 6));
  const int64_t nwaves = static_cast<int64_t>(gridDim.x) * WPB;
  const int64_t per = (a.total_units + nwaves - 1) / nwaves;
  const int64_t U0 = per * wave;
  const int64_t U1 = min(U0 + per, a.total_units);
  if (U0 >= U1) return;

  const int rho = lane / SEG;
  const int j = lane % SEG;
  const int w0 = j * W;
  const int ph = Ends::kAligned ? 0 : (w0 & 3);
  const int g0 = w0 >> 2;
  const int cp = lane & (Cfg<BF16>::kCopies - 1);

  StepGen<R, TABLE> gen;
  gen.di = 0;
  gen.U = U0;
  gen.Uend = U1;
  gen.t = 0;
  if constexpr (TABLE) {  // last descriptor with unit_begin <= U0
    int lo = 0, hi = a.count;
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (((CDesc*)a.table)[mid].unit_begin <= U0) lo = mid; else hi = mid;
    }
    gen.di = __builtin_amdgcn_readfirstlane(lo);
  }

  // First stage: presence words and this lane's group scales of step s.
  auto load_p = [&](const Step& s, uint32_t (&P)[W], uint16_t (&SC)[NQ]) {
    const auto& g = desc_at<TABLE>(a, s.di);
    const int row = s.row0 + rho;
    const int nwl = max(0, min(W, g.upr - w0));
    const bool act = s.valid && row < s.row_end;
    const rsrc_t rb = make_rsrc(g.sec0, g.sec0_bytes);
    const uint32_t off = act ? (static_cast<uint32_t>(row) * g.upr + w0) * 4u : kOOB;
#pragma unroll
    for (int w = 0; w < W; ++w) {
      const uint32_t v = ld32(rb, off + 4u * w);
      P[w] = w < nwl ? v : 0u;
    }
    const rsrc_t rs = make_rsrc(g.scales, g.scales_bytes);
    const bool grouped = (g.mode & kModeGrouped) != 0;
    const uint32_t soff = (act && grouped) ? static_cast<uint32_t>(row) * g.ngroups * 2u : kOOB;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int gi = min(g0 + q, max(g.ngroups - 1, 0));
      SC[q] = ld16(rs, soff + 2u * gi);
    }
  };

  // Second stage: wave prefix of the non-zero counts, then the sign windows.
  uint32_t carry = 0;
  auto load_s = [&](const Step& s, const uint32_t (&P)[W], uint32_t (&lo)[W], uint32_t (&hi)[W],
                    uint32_t (&sh)[W]) {
    const auto& g = desc_at<TABLE>(a, s.di);
    int pc[W];
    int cnt = 0;
#pragma unroll
    for (int w = 0; w < W; ++w) {
      pc[w] = cnt;
      cnt += __builtin_popcount(P[w]);
    }
    const int incl = wave_incl_scan(cnt);
    const uint32_t cursor = s.first ? s.cursor0 : carry;
    carry = cursor + static_cast<uint32_t>(lane63(incl));
    const uint32_t base = cursor + static_cast<uint32_t>(incl - cnt);
    const rsrc_t rg = make_rsrc(g.signs, g.signs_bytes);
#pragma unroll
    for (int w = 0; w < W; ++w) {
      const uint32_t b = base + static_cast<uint32_t>(pc[w]);
      const uint32_t off = (b >> 5) * 4u;
      lo[w] = ld32(rg, off);
      hi[w] = ld32(rg, off + 4u);
      sh[w] = b & 31u;
    }
  };

  // Lane state of the GEMV whose step is being decoded.
  int xdi = -1;
  uint32_t xr[W][NX];
  float xs[NQ];
  float tensor_scale = 0.0f;
  int mode = 0;
  void* ydst = nullptr;
  uint32_t ybytes = 0;

  Step s1 = gen.next(a);
  uint32_t P1[W], lo1[W], hi1[W], sh1[W];
  uint16_t SC1[NQ];
  load_p(s1, P1, SC1);
  load_s(s1, P1, lo1, hi1, sh1);
  Step s2 = gen.next(a);
  uint32_t P2[W];
  uint16_t SC2[NQ];
  load_p(s2, P2, SC2);

  while (s1.valid) {
    // Rotate: decode s0, scan s1 and fetch its signs, fetch presence of s2.
    const Step s0 = s1;
    uint32_t P0[W], lo0[W], hi0[W], sh0[W];
    uint16_t SC0[NQ];
#pragma unroll
    for (int w = 0; w < W; ++w) {
      P0[w] = P1[w];
      lo0[w] = lo1[w];
      hi0[w] = hi1[w];
      sh0[w] = sh1[w];
    }
#pragma unroll
    for (int q = 0; q < NQ; ++q) SC0[q] = SC1[q];
    s1 = s2;
#pragma unroll
    for (int w = 0; w < W; ++w) P1[w] = P2[w];
#pragma unroll
    for (int q = 0; q < NQ; ++q) SC1[q] = SC2[q];
    if (s1.valid) load_s(s1, P1, lo1, hi1, sh1);
    s2 = gen.next(a);
    if (s2.valid) load_p(s2, P2, SC2);

    if (s0.di != xdi) {  // entering another GEMV: its activations and scales
      xdi = s0.di;
      const auto& g = desc_at<TABLE>(a, xdi);
      const int nwl = max(0, min(W, g.upr - w0));
      const rsrc_t rx = make_rsrc(g.x, g.x_bytes);
#pragma unroll
      for (int w = 0; w < W; ++w) {
        const uint32_t off = w < nwl ? static_cast<uint32_t>(w0 + w) * NX * 4u : kOOB;
#pragma unroll
        for (int d = 0; d < NX; ++d) xr[w][d] = ld32(rx, off + 4u * d);
      }
      mode = g.mode;
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        const int gi = min(g0 + q, max(g.ngroups - 1, 0));
        xs[q] = (mode & kModeXscale) ? gp_f32(g.xscale)[gi] : 1.0f;
      }
      tensor_scale = half_bits_to_float(gp_u16(g.scales)[0]);
      ydst = g.y;
      ybytes = g.y_bytes;
    }

    const int row = s0.row0 + rho;
    const bool live = row < s0.row_end;
    Acc run[W];
    Acc acc = Acc(0);
#pragma unroll
    for (int w = 0; w < W; ++w) {
      const uint32_t S = __builtin_amdgcn_alignbit(hi0[w], lo0[w], sh0[w]);
      if constexpr (BF16)
        acc = word_bf16(P0[w], S, xr[w], acc, tab, cp);
      else
        acc = word_i8(P0[w], S, xr[w], acc, tab, cp);
      run[w] = acc;
    }

    if (!BF16 && (mode & kModeRaw)) {
      const int tot = seg_sum<SEG>(static_cast<int>(run[W - 1]));
      if (j == SEG - 1 && live)
        put_y(static_cast<uint32_t>(tot), make_rsrc(ydst, ybytes), 4u * row, 0, (mode & kModeAdd) != 0, true);
      continue;
    }
    float part;
    if (!(mode & (kModeGrouped | kModeXscale))) {
      // One scale per tensor: reduce the exact row sum, multiply once.
      if constexpr (BF16) {
        part = tensor_scale * (2.0f * seg_sum<SEG>(static_cast<float>(run[W - 1])));
      } else {
        part = tensor_scale * static_cast<float>(seg_sum<SEG>(static_cast<int>(run[W - 1])));
      }
    } else {
      float f = 0.0f;
      Acc prev = Acc(0);
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        const Acc e = Ends::pick(run, q, ph);
        const Acc grp = e - prev;
        prev = e;
        const float sc = (mode & kModeGrouped) ? half_bits_to_float(SC0[q]) : tensor_scale;
        f += sc * xs[q] * static_cast<float>(grp);
      }
      part = seg_sum<SEG>(BF16 ? 2.0f * f : f);
    }
    if (j == SEG - 1 && live)
      put_y(__builtin_bit_cast(uint32_t, part), make_rsrc(ydst, ybytes), 4u * row, 0, (mode & kModeAdd) != 0, false);
  }
}

using KernelFn = void (*)(const KernelArgs);

template <int SEG, bool BF16, bool TABLE, int... Ws>
KernelFn pick_w(int w, std::integer_sequence<int, Ws...>) {
  KernelFn fn = nullptr;
  ((w == Ws + 1 ? (fn = bitcos_gemv_kernel<Ws + 1, SEG, BF16, TABLE>, 0) : 0), ...);
  return fn;
}

// Kernel for (words per lane, bf16?, table?) at a fixed SEG; nullptr if none.
template <int SEG>
KernelFn pick_seg(int per_lane, bool bf16, bool table) {
  auto s8 = std::make_integer_sequence<int, bitcos::kMaxWordsBf16>{};
  auto s16 = std::make_integer_sequence<int, bitcos::kMaxWordsI8>{};
  if (bf16) return table ? pick_w<SEG, true, true>(per_lane, s8) : pick_w<SEG, true, false>(per_lane, s8);
  return table ? pick_w<SEG, false, true>(per_lane, s16) : pick_w<SEG, false, false>(per_lane, s16);
}

}  // namespace bitcos_k
