// BITCOS GEMV, streaming kernel for layouts whose unit divides one wave step
// of 64 / SEG rows (the library default is one sign offset per row).
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
// Each word is decoded by two LDS table lookups per presence byte in deposit
// form (FastTables below) and multiplied on the VALU (v_dot2 bf16 / v_dot4
// int8); the scale epilogue is that of bitcos_kernel.h.
#pragma once

#include "bitcos_kernel.h"
#include "tables.h"

namespace bitcos_k {

// Workgroup size of the streaming kernel: one workgroup per CU holding as
// many waves per SIMD as the tile's registers allow (4: <= 128 VGPRs,
// 3: <= 168, 2: <= 256; the bounds follow the register counts of each
// instantiation so none spills).  Host and device both use it.
constexpr int fast_waves_per_simd(int w, bool bf16) {
  return bf16 ? (w <= 3 ? 4 : w <= 5 ? 3 : 2) : (w <= 5 ? 4 : w <= 8 ? 3 : 2);
}
constexpr int fast_threads(int w, bool bf16) { return 256 * fast_waves_per_simd(w, bf16); }

template <int W, bool BF16>
struct FastCfg {
  // Prefetch ring depth: one step ahead.  Two steps ahead (which fits the
  // int8 tiles up to five words per lane) measured no faster.
  static constexpr int kStages = 2;
  // Next word's lookups in flight during the current word's arithmetic
  // (costs one word of lookup registers: 16 int8, 24 bf16).
  static constexpr bool kPipelined = !BF16 && W <= 8;
  // Bytes per wave of a stage buffer: the largest sign block of one step
  // (64 lanes x W words of 32 weights, all non-zero: 64 W dwords) plus the
  // two dwords a window may read past its start, fetched in 16-byte pieces
  // from a dword-aligned start: at most 16 W + 1 pieces.
  static constexpr int kStageBytes = (16 * W + 1) * 16;
  static constexpr int kSignChunks = (16 * W + 1 + 63) / 64;
  static constexpr int kScratchDw = kStageBytes / 4;
  // Sign-table copies: 32 (a conflict-free 8-byte lookup for any 32 keys)
  // when the tables and stage buffers fit the LDS, else 16, else 8.
  static constexpr int kWaves = fast_threads(W, BF16) / 64;
  static constexpr int lds_bytes(int ct) { return 65536 + 2048 * ct + kStages * kWaves * kStageBytes; }
  static constexpr int kSignCopies = lds_bytes(32) <= kLdsBytes ? 32 : lds_bytes(16) <= kLdsBytes ? 16 : 8;
  static_assert(lds_bytes(kSignCopies) <= kLdsBytes, "streaming kernel LDS");
};

// Wave-uniform description of one step (the R rows of one unit).
struct FastStep {
  int di;         // descriptor
  int row0;       // first row
  uint32_t off0;  // first sign bit of the step
  uint32_t off1;  // first sign bit of the next step
  bool valid;
};

// Walks a wave's contiguous unit range.  The fields of the current GEMV are
// read once when the range enters it, not per step.
template <int R, bool TABLE>
struct FastGen {
  int di;
  int U, Uend;           // the launch's units fit in 31 bits (checked on the host)
  int begin, end;        // unit range of GEMV di in the launch
  const uint32_t* offs;  // its unit offsets
  int stride, last;      // offset entries per step; index of the last entry

  __device__ __forceinline__ void enter(const KernelArgs& a, int d) {
    di = __builtin_amdgcn_readfirstlane(d);
    const auto& g = desc_at<TABLE>(a, di);
    begin = static_cast<int>(g.unit_begin);
    end = static_cast<int>(g.unit_begin + g.units);
    offs = g.offsets;
    stride = g.offset_stride;
    last = g.offset_last;
  }

  __device__ __forceinline__ FastStep next(const KernelArgs& a) {
    FastStep s;
    s.valid = U < Uend;
    s.di = di;
    s.row0 = 0;
    s.off0 = 0;
    s.off1 = 0;
    if (!s.valid) return s;
    if constexpr (TABLE) {
      while (U >= end) enter(a, di + 1);  // ends: the last GEMV's end is the total
    }
    const int u = U - begin;
    s.di = di;
    s.row0 = u * R;
    s.off0 = cp_u32(offs)[u * stride];
    s.off1 = cp_u32(offs)[min((u + 1) * stride, last)];
    ++U;
    return s;
  }
};

template <int W, int SEG, bool BF16, bool TABLE>
__global__ void __launch_bounds__(fast_threads(W, BF16)) bitcos_fast_kernel(const KernelArgs a) {
  constexpr int R = kWave / SEG;
  constexpr int NX = BF16 ? 16 : 8;
  constexpr int WPB = fast_threads(W, BF16) / kWave;
  constexpr int D = FastCfg<W, BF16>::kStages;
  constexpr int NSC = FastCfg<W, BF16>::kSignChunks;
  constexpr int SCR = FastCfg<W, BF16>::kScratchDw;
  using Acc = typename std::conditional<BF16, float, int>::type;
  using Ends = GroupEnds<W, 4>;
  constexpr int NQ = Ends::kNQ;

  // Decode tables, and one sign-block buffer per ring stage (each wave owns
  // SCR dwords of every buffer).  The stage buffers are separate objects so
  // the compiler can tell that a read of one does not wait on the fetch into
  // another.
  constexpr int CT = FastCfg<W, BF16>::kSignCopies;
  __shared__ FastTables<BF16, CT> tab;
  __shared__ uint4 sbuf0[WPB * SCR / 4];
  __shared__ uint4 sbuf1[WPB * SCR / 4];
  __shared__ uint4 sbuf2[D > 2 ? WPB * SCR / 4 : 1];
  build_fast_tables<BF16, CT>(tab, threadIdx.x, fast_threads(W, BF16));
  __syncthreads();
  const auto look = [&](uint32_t Pv, uint32_t Sv, const FastLane& f) { return fast_look<BF16, CT>(Pv, Sv, tab, f); };
  const auto math = [&](const Look<BF16>& Lk, const uint32_t* xv, Acc acc0) -> Acc {
    if constexpr (BF16)
      return word_math_bf16(Lk, xv, acc0);
    else
      return fast_math_i8(Lk, xv, acc0);
  };

  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wave = __builtin_amdgcn_readfirstlane(blockIdx.x * WPB + wv);
  const int total = static_cast<int>(a.total_units);
  const int nwaves = static_cast<int>(gridDim.x) * WPB;
  const int per = (total + nwaves - 1) / nwaves;
  const int U0 = per * wave;
  const int U1 = min(U0 + per, total);
  if (U0 >= U1) return;

  const int rho = lane / SEG;
  const int j = lane % SEG;
  const int w0 = j * W;
  const int ph = Ends::kAligned ? 0 : (w0 & 3);
  const int g0 = w0 >> 2;
  const FastLane fl = fast_lane<BF16, CT>(lane);
  auto stage_buf = [&](auto stage_c) -> uint4* {
    constexpr int k = decltype(stage_c)::value;
    if constexpr (k == 0) return sbuf0;
    else if constexpr (k == 1) return sbuf1;
    else return sbuf2;
  };
  // Offset of the wave's part of a stage buffer, in bits.
  const uint32_t wave_bits = static_cast<uint32_t>(wv) * SCR * 32u;

  FastGen<R, TABLE> gen;
  gen.U = U0;
  gen.Uend = U1;
  {
    int lo = 0;
    if constexpr (TABLE) {  // last descriptor with unit_begin <= U0
      int hi = a.count;
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (((CDesc*)a.table)[mid].unit_begin <= U0) lo = mid; else hi = mid;
      }
    }
    gen.enter(a, lo);
  }

  // Ring of stages.
  FastStep st[D];
  uint32_t P[D][W];
  uint16_t SC[D][NQ];

  // Fetch side: buffer resources and lane offsets of the GEMV being fetched.
  // Per step only the wave-uniform row offset changes (soffset); rows past
  // the end of a matrix fall outside its resource and read zero.
  int idi = -1;
  rsrc_t rb = make_rsrc(nullptr, 0), rg = rb, rs = rb;
  uint32_t row_bytes = 0, row_scale_bytes = 0;
  bool grouped = false;
  uint32_t voff_p = 0;
  uint32_t voff_q[NQ];
#pragma unroll
  for (int q = 0; q < NQ; ++q) voff_q[q] = 0;
  const uint32_t voff_s = 16u * static_cast<uint32_t>(lane);

  auto fetch_enter = [&](int d) {
    idi = d;
    const auto& g = desc_at<TABLE>(a, d);
    rb = make_rsrc(g.sec0, g.sec0_bytes);
    rg = make_rsrc(g.signs, g.signs_bytes);
    rs = make_rsrc(g.scales, g.scales_bytes);
    row_bytes = static_cast<uint32_t>(g.upr) * 4u * R;
    row_scale_bytes = static_cast<uint32_t>(g.ngroups) * 2u * R;
    grouped = (g.mode & kModeGrouped) != 0;
    voff_p = (__umul24(static_cast<uint32_t>(rho), static_cast<uint32_t>(g.upr)) + static_cast<uint32_t>(w0)) * 4u;
    const int glast = max(g.ngroups - 1, 0);
#pragma unroll
    for (int q = 0; q < NQ; ++q)
      voff_q[q] = (__umul24(static_cast<uint32_t>(rho), static_cast<uint32_t>(g.ngroups)) +
                   static_cast<uint32_t>(min(g0 + q, glast))) * 2u;
  };

  auto issue = [&](auto stage_c) {
    constexpr int k = decltype(stage_c)::value;
    const FastStep& s = st[k];
    if (s.valid && s.di != idi) fetch_enter(s.di);
    const uint32_t unit = static_cast<uint32_t>(s.row0 / R);
    const uint32_t soff_p = __builtin_amdgcn_readfirstlane(s.valid ? unit * row_bytes : kOOB);
#pragma unroll
    for (int w = 0; w < W; ++w) P[k][w] = __builtin_amdgcn_raw_buffer_load_b32(rb, voff_p + 4u * w, soff_p, 0);
    // The step's sign block: dwords [off0 / 32, off1 / 32 + 1] are the most
    // any window reads.  Only the 16-byte pieces of that range are fetched,
    // straight into this wave's part of the stage buffer (lane l of chunk c
    // lands at byte 1024 c + 16 l); LDS past it keeps stale bits no window
    // uses.
    const uint32_t d0 = s.off0 >> 5;
    const int pieces = static_cast<int>((((s.off1 >> 5) + 2u - d0) * 4u + 15u) >> 4);
    uint4* dst = stage_buf(stage_c) + wv * (SCR / 4);
#pragma unroll
    for (int c = 0; c < NSC; ++c) {
      const int lanes_c = __builtin_amdgcn_readfirstlane(pieces - 64 * c);
      if (s.valid && lanes_c > 0) {
        const uint32_t soff_s = __builtin_amdgcn_readfirstlane(d0 * 4u + 1024u * c);
        if (lane < lanes_c)
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rg, (__attribute__((address_space(3))) void*)(dst + 64 * c), 16,
                                                   voff_s, soff_s, 0, 0);
      }
    }
    const uint32_t soff_q = __builtin_amdgcn_readfirstlane((s.valid && grouped) ? unit * row_scale_bytes : kOOB);
#pragma unroll
    for (int q = 0; q < NQ; ++q) SC[k][q] = __builtin_amdgcn_raw_buffer_load_b16(rs, voff_q[q], soff_q, 0);
  };

  // Decode side: lane state of the GEMV whose steps are being decoded.
  int xdi = -1;
  uint32_t xr[W][NX];
  float xs[NQ];
  float tensor_scale = 0.0f;
  int mode = 0;
  bool ragged = false;
  int nwl = W;
  rsrc_t ry = make_rsrc(nullptr, 0);
  const uint32_t voff_y = 4u * static_cast<uint32_t>(rho);

  // A step's output store is issued at the start of the next step, after
  // its wait (so that wait never waits on the store).
  bool pend = false;
  uint32_t pend_bits = 0, pend_soff = kOOB;
  int pend_mode = 0;
  rsrc_t pend_ry = ry;
  auto flush_store = [&] {
    if (pend) put_y(pend_bits, pend_ry, voff_y, pend_soff, (pend_mode & kModeAdd) != 0, (pend_mode & kModeRaw) != 0);
    pend = false;
  };

  // Decode of one step; `next` issues the following step's loads right after
  // this step's wait.  The step's loads (presence words, scales
  // and the sign block staged into LDS) are waited for all at once: a sign
  // block's LDS-DMA may complete after vector-memory loads issued behind it,
  // so a counted vmcnt wait does not cover it.  With the next step's loads
  // issued only after this wait, only this step's loads are outstanding
  // here, issued a whole step earlier; the next step's sign block goes to
  // the other stage buffer.
  auto decode = [&](auto stage_c, auto&& next) {
    constexpr int k = decltype(stage_c)::value;
    const FastStep& s = st[k];
    wait_vmem_all();
    flush_store();
    // Entering another GEMV: its activations and scales, loaded and waited
    // for before the next step's loads are issued, so that no wait inside
    // the step covers those loads.
    if (s.di != xdi) {
      xdi = s.di;
      const auto& g = desc_at<TABLE>(a, xdi);
      nwl = g.upr - w0;
      ragged = g.upr != SEG * W;
      const int nx = max(0, min(W, nwl));
      const rsrc_t rx = make_rsrc(g.x, g.x_bytes);
#pragma unroll
      for (int w = 0; w < W; ++w) {
        const uint32_t off = w < nx ? static_cast<uint32_t>(w0 + w) * NX * 4u : kOOB;
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
      ry = make_rsrc(g.y, g.y_bytes);
      wait_vmem_all();
    }
    next();
    // LDS byte address of the stage buffer, in bits, so a window's dword
    // address is one shift and mask of its bit cursor.
    using LdsU32 = const __attribute__((address_space(3))) uint32_t;
    const uint32_t stage_bits =
        static_cast<uint32_t>(reinterpret_cast<size_t>((LdsU32*)stage_buf(stage_c))) * 8u;
    // Words past the end of a row (ragged tiles only) count as empty.
    if (ragged) {
#pragma unroll
      for (int w = 0; w < W; ++w)
        if (w >= nwl) P[k][w] = 0u;
    }
    const uint32_t (&Pw)[W] = P[k];
    // Cursor: the step's first sign bit, relative to the block's first dword.
    int pc[W];
    int cnt = 0;
#pragma unroll
    for (int w = 0; w < W; ++w) {
      pc[w] = cnt;
      cnt += __builtin_popcount(Pw[w]);
    }
    const int incl = wave_incl_scan(cnt);
    const uint32_t base = stage_bits + wave_bits + (s.off0 & 31u) + static_cast<uint32_t>(incl - cnt);
    __builtin_amdgcn_wave_barrier();
    // Decode burst at raised wave priority (as in the matrix-core kernel).
    __builtin_amdgcn_s_setprio(1);
    // Software pipeline over the lane's words: the table lookups of word w+1
    // are in flight while word w is multiplied.
    Acc run[W];
    Acc acc = Acc(0);
    // A word's 64-bit window of the sign block, aligned to its first sign.
    auto window = [&](int w) {
      const uint32_t b = base + static_cast<uint32_t>(pc[w]);
      LdsU32* wp = (LdsU32*)static_cast<size_t>((b >> 3) & ~3u);
      return __builtin_amdgcn_alignbit(wp[1], wp[0], b);
    };
    if constexpr (FastCfg<W, BF16>::kPipelined) {
      Look<BF16> L = look(Pw[0], window(0), fl);
#pragma unroll
      for (int w = 0; w < W; ++w) {
        Look<BF16> Ln;
        if (w + 1 < W) Ln = look(Pw[w + 1], window(w + 1), fl);
        acc = math(L, xr[w], acc);
        run[w] = acc;
        if (w + 1 < W) L = Ln;
      }
    } else if constexpr (W <= 8) {
      // Every word's window is read before the first word is decoded, so a
      // word waits on one LDS round trip (its lookups), not two.
      uint32_t S[W];
#pragma unroll
      for (int w = 0; w < W; ++w) S[w] = window(w);
#pragma unroll
      for (int w = 0; w < W; ++w) {
        acc = math(look(Pw[w], S[w], fl), xr[w], acc);
        run[w] = acc;
      }
    } else {  // wide tiles: one word's lookups at a time
#pragma unroll
      for (int w = 0; w < W; ++w) {
        acc = math(look(Pw[w], window(w), fl), xr[w], acc);
        run[w] = acc;
      }
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_s_setprio(0);

    // One lane per row stores; rows past the end are outside ry and dropped.
    const uint32_t soff_y = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(s.row0) * 4u);
    if (!BF16 && (mode & kModeRaw)) {
      const int tot = seg_sum<SEG>(static_cast<int>(run[W - 1]));
      pend = j == SEG - 1;
      pend_bits = static_cast<uint32_t>(tot);
      pend_soff = soff_y;
      pend_mode = mode;
      pend_ry = ry;
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
    pend = j == SEG - 1;
    pend_bits = __builtin_bit_cast(uint32_t, part);
    pend_soff = soff_y;
    pend_mode = mode;
    pend_ry = ry;
  };

  // Prologue: steps 0 .. D-2 in flight.
  [&]<int... Ks>(std::integer_sequence<int, Ks...>) {
    ((st[Ks] = gen.next(a), issue(std::integral_constant<int, Ks>{})), ...);
  }(std::make_integer_sequence<int, D - 1>{});

  bool more = true;
  while (more) {
    [&]<int... Ks>(std::integer_sequence<int, Ks...>) {
      // Stage Ks decodes; stage (Ks + D - 1) % D is refilled after its wait.
      (([&] {
         if (!more) return;
         if (!st[Ks].valid) {
           more = false;
           return;
         }
         constexpr int nk = (Ks + D - 1) % D;
         decode(std::integral_constant<int, Ks>{}, [&] {
           st[nk] = gen.next(a);
           issue(std::integral_constant<int, nk>{});
         });
       }()),
       ...);
    }(std::make_integer_sequence<int, D>{});
  }
  flush_store();
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
