// BITCOS GEMV at batch 1 with the multiply on the matrix cores, for layouts
// with one scale per tensor (or raw int32 sums) and no activation scales.
//
// The decode is the streaming kernel's (bitcos_fast.h): presence words and
// the step's whole sign block are fetched one step ahead, a wavefront prefix
// sum of the lanes' non-zero counts places every lane in the sign block, and
// each presence byte m with its next 8 compact signs s becomes 8 weights in
// position order through two LDS tables, perm(T[s], E[m]) -- Eq. (2)
// w = p - 2n with the deposit of Sec. II-B done by the table.  What changes
// is the multiply: instead of v_dot4 / v_dot2 (the int8 one runs at half
// rate on gfx950) every lane hands its 8 (bf16) or 16 (int8) decoded weights
// and the matching activations to one v_mfma_f32_16x16x32_bf16 /
// v_mfma_i32_16x16x64_i8 and keeps only the diagonal of the product.
//
// A 16 x 16 MFMA sums, for output element (i, j), lane (i + 16 q)'s A slice
// against lane (j + 16 q)'s B slice over q = 0..3.  With A = each lane's own
// activations and B = its own weights, the diagonal element (i, i) is the dot
// product of lanes i, i+16, i+32, i+48 -- so those four lanes must work on
// the same output row.  The lanes are therefore laid out by i = lane % 16:
// row rho = i / (SEG/4) of the step, row segment j = i % (SEG/4) + (SEG/4) q,
// and a segment's W words (with their activations, held in VGPRs for the
// whole GEMV) are words [W j, W j + W) of the row.  The off-diagonal products
// are never read.
//
// The sign-cursor prefix must follow the row-major (row, segment) order, not
// the lane order: one ds_bpermute moves every lane's count to its row-major
// position, the usual DPP wave scan runs there, and a second ds_bpermute
// brings each lane its exclusive prefix back (none for one row per step).
//
// Epilogue per step: lane 16 (i/4) + i holds diagonal element i in
// accumulator register i % 4; a row's SEG/4 diagonal elements are summed with
// quad DPP moves (and an LDS-crossbar swizzle or a readlane for 32 / 64 lanes
// per row), the int32 (or fp32) row sum is multiplied once by the tensor
// scale (Sec. II-C), and one lane per row stores it.
#pragma once

#include "bitcos_fast.h"
#include "mfma_common.h"
#include "tables.h"

namespace bitcos_k {

// Row sums of the diagonal elements.  Lane 16 (i/4) + i holds element i in
// accumulator register i % 4, so in every quad on the diagonal (lanes 20a ..
// 20a + 3) lane 20a + t holds register t.  Returns the row's total in the lane
// that stores it (`store` set, `row` = row within the step); other lanes'
// values are unspecified.
template <int SEG, class T>
__device__ __forceinline__ T diag_row_sum(T c0, T c1, T c2, T c3, int lane, bool& store, int& row) {
  static_assert(SEG == 4 || SEG == 8 || SEG == 16 || SEG == 32 || SEG == 64, "segment");
  const int i16 = lane & 15;
  const bool on_diag = (i16 >> 2) == (lane >> 4);
  if constexpr (SEG == 4) {  // one element per row: lane 20a + t keeps register t
    const T lo = (lane & 1) ? c1 : c0;
    const T hi = (lane & 1) ? c3 : c2;
    store = on_diag;
    row = i16;
    return (lane & 2) ? hi : lo;
  } else if constexpr (SEG == 8) {  // pairs: lane 20a adds register 1 of lane 20a + 1, lane 20a + 2 register 3 of 20a + 3
    const T lo = c0 + qperm<0x55>(c1);  // quad_perm [1,1,1,1]
    const T hi = c2 + qperm<0xFF>(c3);  // quad_perm [3,3,3,3]
    store = on_diag && (lane & 1) == 0;
    row = i16 >> 1;
    const uint32_t m = lane_mask((lane & 2) != 0);
    return bits_as<T>((as_bits(hi) & m) | (as_bits(lo) & ~m));
  } else {
    // Quad total in lane 20a: registers 1, 2, 3 of lanes 20a + 1, + 2, + 3.
    const T q = c0 + qperm<0x55>(c1) + qperm<0xAA>(c2) + qperm<0xFF>(c3);
    if constexpr (SEG == 16) {
      store = on_diag && (lane & 3) == 0;  // lanes 0, 20, 40, 60
      row = lane >> 4;
      return q;
    } else {
      // Rows of 32 lanes: quad totals in lanes 0, 20 (row 0) and 40, 60
      // (row 1); swap lane 0 <-> 20 and 40 <-> 60 within each 32-lane half.
      constexpr int kXor20 = 0x1F | (20 << 10);  // ds_swizzle bitmask mode: and 0x1F, or 0, xor 20
      const T d = q + bits_as<T>(static_cast<uint32_t>(__builtin_amdgcn_ds_swizzle(static_cast<int>(as_bits(q)), kXor20)));
      if constexpr (SEG == 32) {
        store = lane == 0 || lane == 40;
        row = lane >> 5;
        return d;
      } else {
        const T hi = bits_as<T>(static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(as_bits(d)), 40)));
        store = lane == 0;
        row = 0;
        return d + hi;
      }
    }
  }
}

// Decode tables: the deposit-form tables of tables.h (E[m] turns compact
// values into position order, T[s] holds the compact values), addressed by
// one v_perm_b32 per lookup.
// Workgroup size of the diag kernel: one workgroup per CU with as many waves
// per SIMD as the tile's registers allow without spilling (bf16 tiles hold
// the next word's lookups too).  Host and device both use it.
constexpr int diag_waves_per_simd(int w, bool bf16) {
  return bf16 ? (w <= 2 ? 4 : w <= 5 ? 3 : 2) : (w <= 5 ? 4 : w <= 8 ? 3 : 2);
}
constexpr int diag_threads(int w, bool bf16) { return 256 * diag_waves_per_simd(w, bf16); }

// Sign-table copies of the diag kernel for (words per lane, bf16?): 16
// (32, conflict-free, measured no faster on the BitNet-like set), or 8 when
// 16 do not fit beside the stage buffers (int8, 16 words per lane).
constexpr int diag_sign_dwords(int w) { return 64 * w + 4; }
constexpr int diag_sign_copies(int w, bool bf16) {
  return 65536 + 2048 * 16 + 2 * (diag_threads(w, bf16) / 64) * diag_sign_dwords(w) * 4 <= kLdsBytes ? 16 : 8;
}

// Prefetch ring depth: loads one step ahead.  Two steps ahead (with the
// third sign buffer paid for by 16-copy sign tables) measured no faster on
// the BitNet-like set: the decode, not the HBM latency, bounds the kernel.
constexpr int diag_stages(int w, bool bf16) {
  (void)w;
  (void)bf16;
  return 2;
}

// The word's weights (perm) multiplied against its activations x (32 bf16 in
// 16 dwords or 32 int8 in 8) on the matrix cores, into two accumulators.
template <bool BF16, class CV>
__device__ __forceinline__ void diag_math(const Look<BF16>& L, const uint32_t* x, CV (&c)[2]) {
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    if constexpr (BF16) {
      const uint2 t = L.th[b];
      const uint4 e = L.sb[b];
      const u32x4_t wt = {__builtin_amdgcn_perm(t.y, t.x, e.x), __builtin_amdgcn_perm(t.y, t.x, e.y),
                          __builtin_amdgcn_perm(t.y, t.x, e.z), __builtin_amdgcn_perm(t.y, t.x, e.w)};
      const u32x4_t xv = {x[4 * b], x[4 * b + 1], x[4 * b + 2], x[4 * b + 3]};
      c[b & 1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, xv),
                                                         __builtin_bit_cast(bf16x8_t, wt), c[b & 1], 0, 0, 0);
    } else if (b & 1) {
      const uint2 t0 = L.tv[b - 1], e0 = L.sv[b - 1], t1 = L.tv[b], e1 = L.sv[b];
      const u32x4_t wt = {__builtin_amdgcn_perm(t0.y, t0.x, e0.x), __builtin_amdgcn_perm(t0.y, t0.x, e0.y),
                          __builtin_amdgcn_perm(t1.y, t1.x, e1.x), __builtin_amdgcn_perm(t1.y, t1.x, e1.y)};
      const int h = b >> 1;
      const u32x4_t xv = {x[4 * h], x[4 * h + 1], x[4 * h + 2], x[4 * h + 3]};
      c[h] = __builtin_amdgcn_mfma_i32_16x16x64_i8(__builtin_bit_cast(i32x4_t, xv), __builtin_bit_cast(i32x4_t, wt),
                                                   c[h], 0, 0, 0);
    }
  }
}

// Conditions of the in-row prefix below as bits of one opaque per-lane word
// (computed once per kernel; each use sign-extends one bit into a mask):
// bit 0 / 1 = the lane is at least 1 / 2 places into its S4-lane group,
// bit 2 / 3 = bits 0 / 1 of the lane's q group.
template <int S4>
__device__ __forceinline__ uint32_t row_prefix_bits(int lane) {
  const int k = lane & (S4 - 1);
  const int q = lane >> 4;
  uint32_t b = (k >= 1 ? 1u : 0u) | (k >= 2 ? 2u : 0u) | static_cast<uint32_t>(q & 3) << 2;
  asm volatile("" : "+v"(b));
  return b;
}
__device__ __forceinline__ uint32_t bit_mask(uint32_t bits, int i) {
  return static_cast<uint32_t>(__builtin_amdgcn_sbfe(static_cast<int>(bits), i, 1));
}

// Exclusive prefix of the lanes' counts over the segments of their row, in
// segment order j = i % S4 + S4 q, for S4 = SEG / 4 <= 4 lanes of a row in
// each 16-lane q group: a prefix inside the S4-lane group (quad DPP moves),
// then over the four q groups (permlane swaps between 16-lane rows, no LDS).
template <int S4>
__device__ __forceinline__ int row_prefix(int cnt, uint32_t pbits) {
  static_assert(S4 == 1 || S4 == 2 || S4 == 4, "lanes of a row per q group");
  uint32_t incl = static_cast<uint32_t>(cnt);  // inclusive prefix inside the S4-lane group
  if constexpr (S4 >= 2) incl += qperm<0x90>(incl) & bit_mask(pbits, 0);  // quad_perm [0,0,1,2]: lane k-1
  if constexpr (S4 == 4) incl += qperm<0x40>(incl) & bit_mask(pbits, 1);  // quad_perm [0,0,0,1]: lane k-2
  uint32_t own = incl;  // the group's total, in every lane of the group
  if constexpr (S4 == 2) own = qperm<0xF5>(incl);  // quad_perm [1,1,3,3]
  if constexpr (S4 == 4) own = qperm<0xFF>(incl);  // quad_perm [3,3,3,3]
  // Totals of the other q groups.  permlane16_swap exchanges 16-lane rows
  // between the pairs (0,1) and (2,3), permlane32_swap the halves (rows 0,1
  // against 2,3); with the same value in both operands the two results hold
  // this row's and the partner's value, so partner = sum - own either way.
  const auto p16 = __builtin_amdgcn_permlane16_swap(own, own, false, false);
  const uint32_t partner = p16[0] + p16[1] - own;
  const uint32_t pair = own + partner;
  const auto p32 = __builtin_amdgcn_permlane32_swap(pair, pair, false, false);
  const uint32_t other = p32[0] + p32[1] - pair;
  return static_cast<int>((partner & bit_mask(pbits, 2)) + (other & bit_mask(pbits, 3)) + incl - static_cast<uint32_t>(cnt));
}

template <int W, int SEG, bool BF16, bool TABLE>
__global__ void __launch_bounds__(diag_threads(W, BF16)) bitcos_diag_kernel(const KernelArgs a) {
  constexpr int R = kWave / SEG;
  constexpr int S4 = SEG / 4;  // lanes of one row among the 16 lanes of a q group
  constexpr int NX = BF16 ? 16 : 8;
  constexpr int WPB = diag_threads(W, BF16) / kWave;
  constexpr int D = diag_stages(W, BF16);
  // Sign buffer of one wave and stage: the largest step block (64 lanes x W
  // words, all non-zero) plus the dword a window reads past its start and
  // the step's in-dword offset, rounded to 16 bytes.  It is filled in
  // 1 KB chunks (16 bytes per lane), of which only the lanes inside the
  // step's block load.
  constexpr int SCR = diag_sign_dwords(W);
  constexpr int NSC = (SCR + 255) / 256;
  using Acc = typename std::conditional<BF16, float, int>::type;
  using CV = typename std::conditional<BF16, f32x4_t, i32x4_t>::type;

  constexpr int CT = diag_sign_copies(W, BF16);
  __shared__ FastTables<BF16, CT> tab;
  __shared__ uint4 sbuf0[WPB * SCR / 4];
  __shared__ uint4 sbuf1[WPB * SCR / 4];
  __shared__ uint4 sbuf2[D > 2 ? WPB * SCR / 4 : 1];
  static_assert(sizeof(tab) + 2 * sizeof(sbuf0) <= kLdsBytes, "diag kernel LDS");
  build_fast_tables<BF16, CT>(tab, threadIdx.x, diag_threads(W, BF16));
  __syncthreads();

  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wave = __builtin_amdgcn_readfirstlane(blockIdx.x * WPB + wv);
  const int total = static_cast<int>(a.total_units);
  const int nwaves = static_cast<int>(gridDim.x) * WPB;
  const int per = (total + nwaves - 1) / nwaves;
  const int U0 = per * wave;
  const int U1 = min(U0 + per, total);
  if (U0 >= U1) return;
  const FastLane fl = fast_lane<BF16, CT>(lane);

  // Lane layout: i = lane % 16 picks the row, the q group a quarter of its segments.
  const int i16 = lane & 15;
  const int qg = lane >> 4;
  const int rho = i16 / S4;
  const int j = (i16 % S4) + S4 * qg;
  const int w0 = j * W;
  // Row-major position of this lane in the step, and the lane that holds
  // row-major position `lane` (byte addresses for ds_bpermute).
  const int nat_addr = (rho * SEG + j) * 4;
  const uint32_t pbits = row_prefix_bits<(S4 < 4 ? S4 : 4)>(lane);
  const int src_addr = (16 * ((lane % SEG) / S4) + (lane / SEG) * S4 + (lane % SEG) % S4) * 4;

  auto stage_buf = [&](auto stage_c) -> uint4* {
    constexpr int k = decltype(stage_c)::value;
    if constexpr (k == 0) return sbuf0;
    else if constexpr (k == 1) return sbuf1;
    else return sbuf2;
  };
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

  FastStep st[D];
  uint32_t P[D][W];
  uint32_t ROFF[D];  // sign offset of the lane's row (layouts with one offset per row)
  constexpr bool kRowOffsets = SEG <= 16;

  // Fetch side (as in the streaming kernel, without group scales).
  int idi = -1;
  rsrc_t rb = make_rsrc(nullptr, 0), rg = rb, ro = rb;
  uint32_t row_bytes = 0;
  uint32_t voff_p = 0;
  const uint32_t voff_s = 16u * static_cast<uint32_t>(lane);

  auto fetch_enter = [&](int d) {
    idi = d;
    const auto& g = desc_at<TABLE>(a, d);
    rb = make_rsrc(g.sec0, g.sec0_bytes);
    rg = make_rsrc(g.signs, g.signs_bytes);
    ro = make_rsrc(g.offsets, static_cast<uint32_t>(g.offset_last + 1) * 4u);
    row_bytes = static_cast<uint32_t>(g.upr) * 4u * R;
    voff_p = (__umul24(static_cast<uint32_t>(rho), static_cast<uint32_t>(g.upr)) + static_cast<uint32_t>(w0)) * 4u;
  };

  auto issue = [&](auto stage_c) {
    constexpr int k = decltype(stage_c)::value;
    const FastStep& s = st[k];
    if (s.valid && s.di != idi) fetch_enter(s.di);
    const uint32_t unit = static_cast<uint32_t>(s.row0 / R);
    const uint32_t soff_p = __builtin_amdgcn_readfirstlane(s.valid ? unit * row_bytes : kOOB);
    // The lane's words: the first four in one 16-byte load (dword-aligned;
    // dwords past the section read zero), the rest one by one.
    if constexpr (W >= 4) {
      const u32x4_t v = ld128_s(rb, voff_p, soff_p);
#pragma unroll
      for (int w = 0; w < 4; ++w) P[k][w] = v[w];
#pragma unroll
      for (int w = 4; w < W; ++w) P[k][w] = __builtin_amdgcn_raw_buffer_load_b32(rb, voff_p + 4u * w, soff_p, 0);
    } else {
#pragma unroll
      for (int w = 0; w < W; ++w) P[k][w] = __builtin_amdgcn_raw_buffer_load_b32(rb, voff_p + 4u * w, soff_p, 0);
    }
    if constexpr (kRowOffsets) {  // rows past the matrix end read the last entry (nnz)
      const int e = min(static_cast<int>(unit) * gen.stride + rho, gen.last);
      ROFF[k] = ld32(ro, s.valid ? static_cast<uint32_t>(e) * 4u : kOOB);
    }
    // The step's sign block: dwords [off0 / 32, off1 / 32 + 1] are the most
    // any window reads.  Only the 16-byte pieces of that range are fetched
    // (lane l of chunk c lands at byte 1024 c + 16 l of the wave's buffer);
    // LDS past it keeps stale bits no window uses.
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
  };

  // Decode side.
  int xdi = -1;
  uint32_t xr[W][NX];
  float tensor_scale = 0.0f;
  int mode = 0;
  bool ragged = false;
  int nwl = W;
  rsrc_t ry = make_rsrc(nullptr, 0);

  // A step's output store is issued at the start of the next step, after
  // its wait (so that wait never waits on the store).
  bool pend = false;
  uint32_t pend_bits = 0, pend_voff = 0, pend_soff = kOOB;
  int pend_mode = 0;
  rsrc_t pend_ry = ry;
  auto flush_store = [&] {
    if (pend) put_y(pend_bits, pend_ry, pend_voff, pend_soff, (pend_mode & kModeAdd) != 0, (pend_mode & kModeRaw) != 0);
    pend = false;
  };

  // Decode of one step; `next` issues the following step's loads right after
  // this step's wait (and the activations of a GEMV the wave enters).  The step's loads (presence words, row offsets and the
  // sign block staged into LDS) are waited for all at once: a sign block's
  // LDS-DMA may complete after vector-memory loads issued behind it, so a
  // counted vmcnt wait does not cover it.  With the next step's loads issued
  // only after this wait, only this step's loads are outstanding here,
  // issued a whole step earlier; the next step's sign block goes to the
  // other stage buffer.
  auto decode = [&](auto stage_c, auto&& next) {
    constexpr int k = decltype(stage_c)::value;
    const FastStep& s = st[k];
    wait_vmem_all();
    flush_store();
    // Entering another GEMV: its activations, loaded and waited for before
    // the next step's loads are issued, so that no wait inside the step
    // covers those loads.
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
      tensor_scale = half_bits_to_float(gp_u16(g.scales)[0]);
      ry = make_rsrc(g.y, g.y_bytes);
      wait_vmem_all();
    }
    next();
    // LDS byte address of the stage buffer, in bits (cursors below count from
    // LDS address 0, so a window's dword address is one shift and mask).
    using LdsU32 = const __attribute__((address_space(3))) uint32_t;
    const uint32_t stage_bits =
        static_cast<uint32_t>(reinterpret_cast<size_t>((LdsU32*)stage_buf(stage_c))) * 8u + wave_bits;
    if (ragged) {
#pragma unroll
      for (int w = 0; w < W; ++w)
        if (w >= nwl) P[k][w] = 0u;
    }
    const uint32_t (&Pw)[W] = P[k];
    int pc[W];
    int cnt = 0;
#pragma unroll
    for (int w = 0; w < W; ++w) {
      pc[w] = cnt;
      cnt += __builtin_popcount(Pw[w]);
    }
    // The lane's first sign bit, relative to the step's sign block (which
    // starts at the dword holding the step's first sign): its row's offset
    // plus the counts of the row's earlier segments; or, with two or more
    // q groups per row, an exclusive prefix in row-major (row, segment) order.
    uint32_t base;
    if constexpr (kRowOffsets) {
      base = stage_bits + (ROFF[k] - (s.off0 & ~31u)) + static_cast<uint32_t>(row_prefix<S4>(cnt, pbits));
    } else if constexpr (SEG == 64) {
      base = stage_bits + (s.off0 & 31u) + static_cast<uint32_t>(wave_incl_scan(cnt) - cnt);
    } else {
      const int nc = __builtin_amdgcn_ds_bpermute(src_addr, cnt);
      const int excl = __builtin_amdgcn_ds_bpermute(nat_addr, wave_incl_scan(nc) - nc);
      base = stage_bits + (s.off0 & 31u) + static_cast<uint32_t>(excl);
    }
    __builtin_amdgcn_wave_barrier();
    // The windows, lookups and multiplies of the step at raised wave
    // priority: a wave whose loads have landed gets the SIMD's issue slots
    // for its whole decode burst ahead of waves still in their step
    // prologue, which keeps the VALU, LDS and matrix cores fed back to back
    // (6-7 % faster on the BitNet-like K = 2560 launch).
    __builtin_amdgcn_s_setprio(1);

    // Windows: 64 bits at each word's first sign.  The lane's cursor is
    // clamped once so that every window stays in the wave's own buffer (a
    // valid cursor never needs it; a word's offset in the lane is < 32 W).
    uint32_t S[W];
    const uint32_t bclamp = min(base, stage_bits + (SCR - 2 - W) * 32u);
#pragma unroll
    for (int w = 0; w < W; ++w) {
      const uint32_t b = bclamp + static_cast<uint32_t>(pc[w]);
      LdsU32* sp = (LdsU32*)static_cast<size_t>((b >> 3) & ~3u);
      S[w] = __builtin_amdgcn_alignbit(sp[1], sp[0], b);
    }
    // Two accumulators, alternating, so consecutive MFMAs do not wait on each
    // other; word w + 1's lookups are in flight while word w is multiplied
    // (except on the widest int8 tiles, whose registers go to activations).
    CV acc[2] = {CV{0, 0, 0, 0}, CV{0, 0, 0, 0}};
    if constexpr (BF16 || W <= 12) {
      Look<BF16> L = fast_look<BF16, CT>(Pw[0], S[0], tab, fl);
#pragma unroll
      for (int w = 0; w < W; ++w) {
        Look<BF16> Ln;
        if (w + 1 < W) Ln = fast_look<BF16, CT>(Pw[w + 1], S[w + 1], tab, fl);
        diag_math<BF16>(L, xr[w], acc);
        if (w + 1 < W) L = Ln;
      }
    } else {
#pragma unroll
      for (int w = 0; w < W; ++w) diag_math<BF16>(fast_look<BF16, CT>(Pw[w], S[w], tab, fl), xr[w], acc);
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_s_setprio(0);

    bool store = false;
    int row = 0;
    const Acc tot = diag_row_sum<SEG, Acc>(acc[0][0] + acc[1][0], acc[0][1] + acc[1][1], acc[0][2] + acc[1][2],
                                           acc[0][3] + acc[1][3], lane, store, row);
    uint32_t bits;
    if (!BF16 && (mode & kModeRaw)) {
      bits = static_cast<uint32_t>(tot);
    } else if constexpr (BF16) {
      bits = __builtin_bit_cast(uint32_t, tensor_scale * (2.0f * static_cast<float>(tot)));
    } else {
      bits = __builtin_bit_cast(uint32_t, tensor_scale * static_cast<float>(tot));
    }
    // Rows past the end of the matrix fall outside ry and are dropped.
    pend = store;
    pend_bits = bits;
    pend_voff = 4u * static_cast<uint32_t>(row);
    pend_soff = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(s.row0) * 4u);
    pend_mode = mode;
    pend_ry = ry;
  };

  [&]<int... Ks>(std::integer_sequence<int, Ks...>) {
    ((st[Ks] = gen.next(a), issue(std::integral_constant<int, Ks>{})), ...);
  }(std::make_integer_sequence<int, D - 1>{});

  bool more = true;
  while (more) {
    [&]<int... Ks>(std::integer_sequence<int, Ks...>) {
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

template <int SEG, bool BF16, bool TABLE, int... Ws>
FastFn pick_diag_w(int w, std::integer_sequence<int, Ws...>) {
  FastFn fn = nullptr;
  ((w == Ws + 1 ? (fn = bitcos_diag_kernel<Ws + 1, SEG, BF16, TABLE>, 0) : 0), ...);
  return fn;
}

template <int SEG>
FastFn pick_diag_seg(int per_lane, bool bf16, bool table) {
  auto s8 = std::make_integer_sequence<int, bitcos::kMaxWordsBf16>{};
  auto s16 = std::make_integer_sequence<int, bitcos::kMaxWordsI8>{};
  if (bf16) return table ? pick_diag_w<SEG, true, true>(per_lane, s8) : pick_diag_w<SEG, true, false>(per_lane, s8);
  return table ? pick_diag_w<SEG, false, true>(per_lane, s16) : pick_diag_w<SEG, false, false>(per_lane, s16);
}

}  // namespace bitcos_k
