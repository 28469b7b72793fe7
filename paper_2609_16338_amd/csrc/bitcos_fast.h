// BITCOS GEMV, streaming kernel for layouts whose unit is one wave step
// (unit_rows == 64 / SEG rows, the library default).
//
// With one stored sign offset per step, the step's whole sign range
// [off[u], off[u+1]) is known before its presence words arrive, so nothing
// in the loop waits on a dependent global load:
//   * every wave runs a ring of D stages; the loads of step s+D-1 (the
//     lane's presence words and group scales, plus the step's sign block
//     read coalesced, 16 bytes per lane) are issued before step s is decoded;
//   * at decode time the sign block goes to a per-wave LDS scratch, a
//     wavefront prefix sum of the lanes' non-zero counts gives every lane its
//     bit position in the block, and each 32-weight word reads its 64-bit
//     window from LDS;
//   * the loop is unrolled by D so the ring never moves registers, and all
//     loads are unconditional (unused ones address past the buffer and read
//     zero) so the waits have fixed counts.
// The per-word decode (compacted activations x sign table, Eq. (2)) and the
// scale epilogue are those of bitcos_kernel.h.
#pragma once

#include "bitcos_kernel.h"

namespace bitcos_k {

template <int W, bool BF16>
struct FastCfg {
  static constexpr int kStages = W <= 8 ? 3 : 2;
  // 16-byte chunks per lane of the largest sign block of one step: 64 lanes x
  // W words of 32 weights, all non-zero, plus the two dwords a window may
  // read past its start.
  static constexpr int kSignChunks = (64 * W + 2 + 255) / 256;
  static constexpr int kScratchDw = kSignChunks * 256;
};

struct FastStep {
  int di;
  int row0;
  int nrows;
  uint32_t off0;  // first sign bit of the step
  uint32_t d0;    // first sign dword of the block
  bool valid;
};

template <int R, bool TABLE>
struct FastGen {
  int di;
  int64_t U, Uend;

  __device__ __forceinline__ FastStep next(const KernelArgs& a) {
    FastStep s;
    s.valid = U < Uend;
    s.di = di;
    s.row0 = 0;
    s.nrows = 0;
    s.off0 = 0;
    s.d0 = 0;
    if (!s.valid) return s;
    if constexpr (TABLE) {
      while (di + 1 < a.count && U >= desc_at<TABLE>(a, di).unit_begin + desc_at<TABLE>(a, di).units) ++di;
      di = __builtin_amdgcn_readfirstlane(di);
    }
    const auto& g = desc_at<TABLE>(a, di);
    const int u = static_cast<int>(U - g.unit_begin);
    s.di = di;
    s.row0 = u * R;
    s.nrows = min(R, g.n - s.row0);
    s.off0 = cp_u32(g.offsets)[u];
    s.d0 = s.off0 >> 5;
    ++U;
    return s;
  }
};

template <int W, int SEG, bool BF16, bool TABLE>
__global__ void __launch_bounds__(Cfg<BF16>::kThreads) bitcos_fast_kernel(const KernelArgs a) {
  constexpr int R = kWave / SEG;
  constexpr int NX = BF16 ? 16 : 8;
  constexpr int WPB = Cfg<BF16>::kThreads / kWave;
  constexpr int D = FastCfg<W, BF16>::kStages;
  constexpr int NSC = FastCfg<W, BF16>::kSignChunks;
  constexpr int SCR = FastCfg<W, BF16>::kScratchDw;
  using Acc = typename std::conditional<BF16, float, int>::type;
  using Ends = GroupEnds<W, 4>;
  constexpr int NQ = Ends::kNQ;

  __shared__ Tables<BF16> tab;
  __shared__ uint4 scratch[WPB][SCR / 4];
  build_tables<BF16>(tab, threadIdx.x);
  __syncthreads();

  const int lane = threadIdx.x & 63;
  const int wv = threadIdx.x >> 6;
  const int wave = __builtin_amdgcn_readfirstlane(blockIdx.x * WPB + wv);
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
  uint4* scr = scratch[wv];
  const uint32_t* scr32 = reinterpret_cast<const uint32_t*>(scr);

  FastGen<R, TABLE> gen;
  gen.di = 0;
  gen.U = U0;
  gen.Uend = U1;
  if constexpr (TABLE) {
    int lo = 0, hi = a.count;
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (((CDesc*)a.table)[mid].unit_begin <= U0) lo = mid; else hi = mid;
    }
    gen.di = __builtin_amdgcn_readfirstlane(lo);
  }

  // Ring of stages.
  FastStep st[D];
  uint32_t P[D][W];
  uint4 SV[D][NSC];
  uint16_t SC[D][NQ];

  auto issue = [&](auto stage_c) {
    constexpr int k = decltype(stage_c)::value;
    const FastStep& s = st[k];
    const auto& g = desc_at<TABLE>(a, s.di);
    const int row = s.row0 + rho;
    const int nwl = max(0, min(W, g.upr - w0));
    const bool act = s.valid && rho < s.nrows;
    const rsrc_t rb = make_rsrc(g.sec0, g.sec0_bytes);
    const uint32_t off = act ? (static_cast<uint32_t>(row) * g.upr + w0) * 4u : kOOB;
#pragma unroll
    for (int w = 0; w < W; ++w) {
      const uint32_t v = ld32(rb, off + 4u * w);
      P[k][w] = w < nwl ? v : 0u;
    }
    const rsrc_t rg = make_rsrc(g.signs, g.signs_bytes);
    const uint32_t soff = s.valid ? (s.d0 + 4u * lane) * 4u : kOOB;
#pragma unroll
    for (int c = 0; c < NSC; ++c) {
      SV[k][c] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rg, soff + 1024u * c, 0, 0));
    }
    const rsrc_t rs = make_rsrc(g.scales, g.scales_bytes);
    const bool grouped = (g.mode & kModeGrouped) != 0;
    const uint32_t qoff = (act && grouped) ? static_cast<uint32_t>(row) * g.ngroups * 2u : kOOB;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int gi = min(g0 + q, max(g.ngroups - 1, 0));
      SC[k][q] = ld16(rs, qoff + 2u * gi);
    }
  };

  // Lane state of the GEMV being decoded.
  int xdi = -1;
  uint32_t xr[W][NX];
  float xs[NQ];
  float tensor_scale = 0.0f;
  int mode = 0;
  void* ydst = nullptr;

  auto decode = [&](auto stage_c) {
    constexpr int k = decltype(stage_c)::value;
    const FastStep& s = st[k];
    if (s.di != xdi) {  // entering another GEMV: its activations and scales
      xdi = s.di;
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
    }
    // Sign block of the step into this wave's scratch.
#pragma unroll
    for (int c = 0; c < NSC; ++c) scr[lane + 64 * c] = SV[k][c];
    // Cursor: the step's first sign bit, relative to the block's first dword.
    int pc[W];
    int cnt = 0;
#pragma unroll
    for (int w = 0; w < W; ++w) {
      pc[w] = cnt;
      cnt += __builtin_popcount(P[k][w]);
    }
    const int incl = wave_incl_scan(cnt);
    const uint32_t base = (s.off0 & 31u) + static_cast<uint32_t>(incl - cnt);
    __builtin_amdgcn_wave_barrier();
    Acc run[W];
    Acc acc = Acc(0);
#pragma unroll
    for (int w = 0; w < W; ++w) {
      const uint32_t b = base + static_cast<uint32_t>(pc[w]);
      const uint32_t i = b >> 5;
      const uint32_t S = __builtin_amdgcn_alignbit(scr32[i + 1], scr32[i], b & 31u);
      if constexpr (BF16)
        acc = word_bf16(P[k][w], S, xr[w], acc, tab, cp);
      else
        acc = word_i8(P[k][w], S, xr[w], acc, tab, cp);
      run[w] = acc;
    }
    __builtin_amdgcn_wave_barrier();

    const int row = s.row0 + rho;
    const bool live = rho < s.nrows;
    if (!BF16 && (mode & kModeRaw)) {
      const int tot = seg_sum<SEG>(static_cast<int>(run[W - 1]));
      if (j == 0 && live) gp_i32_out(ydst)[row] = tot;
      return;
    }
    float part;
    if (!(mode & (kModeGrouped | kModeXscale))) {
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
        const float sc = (mode & kModeGrouped) ? half_bits_to_float(SC[k][q]) : tensor_scale;
        f += sc * xs[q] * static_cast<float>(grp);
      }
      part = seg_sum<SEG>(BF16 ? 2.0f * f : f);
    }
    if (j == 0 && live) gp_f32_out(ydst)[row] = part;
  };

  // Prologue: steps 0 .. D-2 in flight.
  [&]<int... Ks>(std::integer_sequence<int, Ks...>) {
    ((st[Ks] = gen.next(a), issue(std::integral_constant<int, Ks>{})), ...);
  }(std::make_integer_sequence<int, D - 1>{});

  bool more = true;
  while (more) {
    [&]<int... Ks>(std::integer_sequence<int, Ks...>) {
      // Stage Ks decodes; stage (Ks + D - 1) % D is refilled first.
      (([&] {
         if (!more) return;
         constexpr int nk = (Ks + D - 1) % D;
         st[nk] = gen.next(a);
         issue(std::integral_constant<int, nk>{});
         if (!st[Ks].valid) {
           more = false;
           return;
         }
         decode(std::integral_constant<int, Ks>{});
       }()),
       ...);
    }(std::make_integer_sequence<int, D>{});
  }
}

using FastFn = void (*)(const KernelArgs);

template <int SEG, bool BF16, bool TABLE, int... Ws>
FastFn pick_fast_w(int w, std::integer_sequence<int, Ws...>) {
  FastFn fn = nullptr;
  ((w == Ws + 1 ? (fn = bitcos_fast_kernel<Ws + 1, SEG, BF16, TABLE>, 0) : 0), ...);
  return fn;
}

template <int SEG>
FastFn pick_fast_seg(int per_lane, bool bf16, bool table) {
  auto s8 = std::make_integer_sequence<int, bitcos::kMaxWordsBf16>{};
  auto s16 = std::make_integer_sequence<int, bitcos::kMaxWordsI8>{};
  if (bf16) return table ? pick_fast_w<SEG, true, true>(per_lane, s8) : pick_fast_w<SEG, true, false>(per_lane, s8);
  return table ? pick_fast_w<SEG, false, true>(per_lane, s16) : pick_fast_w<SEG, false, false>(per_lane, s16);
}

}  // namespace bitcos_k
