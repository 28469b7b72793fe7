// BITCOS GEMV for a small batch of activation rows (2 <= M <= 16) on the
// matrix cores.  Decode cost per weight is the same at any batch size, so a
// batch of M activation rows multiplies every decoded weight M times: one
// MFMA takes a decoded weight tile against all (up to 16) rows at once.  It
// also runs batch 1 (M = 1) for rows longer than the batch-1 kernels' tiles,
// whose activations must fit a lane's registers; here they are read per
// step, so K has no limit.
//
// Work unit: 32 output rows (two 16-row MFMA tiles) over the whole of K; a
// wave walks its units in steps of four 128-weight scale groups.  A launch
// counts its GEMVs in steps (a unit of a K-long row is K / 512 steps), and
// each wave takes the units that start inside its equal share of the steps,
// so GEMVs of different K in one launch leave no wave with several times the
// others' work.
//   * Lane l works on row n = l % 16 of each tile and, in every group, on its
//     32-weight word g = l / 16, so the four lane groups of a row cover one
//     group together and an MFMA never mixes two scale groups.
//   * B operand (weights, K x 16 rows): per presence byte of the lane's word
//     the 8 weights come out of two LDS table lookups (tables.h) keyed by the
//     presence byte m and the next 8 compact sign bits s, combined by
//     v_perm_b32 (Eq. (2) w = p - 2n, with the deposit of Sec. II-B done by
//     the table): int8 +-1 bytes for v_mfma_i32_16x16x64_i8, bf16 +-0.5 for
//     v_mfma_f32_16x16x32_bf16 (the 0.5 is undone exactly at the end).
//   * A operand (activations, 16 batch rows x K): lane (m, g) holds batch row
//     m's activations at the positions its B partner decodes; rows m >= M
//     read zero through the buffer range check, so one kernel serves every M
//     (loads whose rows are all past M are skipped).  Loaded in whole 16-byte
//     pieces per batch row and handed to the lanes through a per-wave LDS
//     transpose buffer.
//   * C (16 batch rows x 16 output rows): lane l holds batch rows
//     4 (l / 16) + i of output row l % 16.  Every group's C is scaled into
//     fp32 accumulators (fp16 group scale x activation scale, Sec. II-C), or
//     summed exactly in int32 when the scale is per tensor.
// Sign cursors: every row's entry comes from its offset entry (one per row);
// in a step the four lanes of a row exchange their words' popcounts (one
// byte per group, by permlane swaps between 16-lane rows) to place each
// word.  A row's signs for one step (at most 512 bits, starting anywhere in
// a dword) are fetched as 20 dwords, staged in the wave's LDS block and read
// as 64-bit windows.
// Loads: the kernel is bound by the count of its loads more than by their
// bytes, so each row's data of a step comes in as few as possible: its
// presence words in one 16-byte load per lane (group g, then transposed
// across the row's four lanes), its four group scales in one 12-byte load,
// the activation scales in one 16-byte load per lane shared across quads.
// Pipeline: the presence words, group scales and sign dwords of step t+1 are
// issued at the start of step t (the sign range of step t+1 follows from the
// popcounts of step t).  Activations of step t+1 are issued during step t,
// group by group as step t's MFMAs release their registers, so that waiting
// for them never waits on a prefetch issued after them.  Inside a step the
// table lookups of group q + 1 are in flight while group q's weights are
// built and multiplied, and the two tiles' MFMA chains alternate.
#pragma once

#include "mfma_common.h"
#include "tables.h"

namespace bitcos_k {

constexpr int kMfmaTile = 16;                   // output rows per MFMA tile
constexpr int kMfmaRT = 2;                      // tiles per work unit
constexpr int kMfmaRows = kMfmaTile * kMfmaRT;  // rows per work unit
// Workgroup size: one workgroup per CU (the decode tables fill most of the
// LDS), 2 waves per SIMD: the group lookahead below holds about 240
// registers (bf16).  int8 at 3 waves per SIMD and without the lookahead
// spills with activation scales and measured slower.  Host and device both
// use it.
constexpr int mfma_threads(bool bf16, bool xs) {
  (void)bf16;
  (void)xs;
  return 512;
}
constexpr int kMfmaMaxBatch = 16;
constexpr int kSignStride = 21;  // LDS dwords per staged sign row (20 used; odd spreads banks)
// The table lookups of group q + 1 are issued before group q's arithmetic.
constexpr bool mfma_lookahead(bool bf16) {
  (void)bf16;
  return true;
}
// Activation loads: each load reads whole 16-byte pieces of a few batch
// rows in order (fully used cache lines) and the wave's transpose buffer in
// LDS hands every lane its MFMA operand.  Loading each lane's operand
// directly (16 bytes of batch row m at the lane's word: every load touches
// 16 rows x 2 cache lines) measured slower at every M (8 Qwen3-32B-like
// layers, us per step, bf16 / int8: 597 / 576 against 573 / 576 at M = 4,
// 843 / 670 against 651 / 611 at M = 16).
constexpr int mfma_xrow(bool bf16) { return (bf16 ? 256 : 128) + 16; }  // one group's activations of a batch row, padded
constexpr int mfma_xbuf_bytes(bool bf16) { return 16 * mfma_xrow(bf16); }
// Sign-table copies (tables.h): 32 when the tables and the waves' sign
// stages fit the LDS, else 16.
constexpr int mfma_sign_copies(bool bf16) {
  return 65536 + 2048 * 32 + (mfma_threads(bf16, false) / 64) * (kMfmaRows * kSignStride * 4 + mfma_xbuf_bytes(bf16)) <=
                 kLdsBytes
             ? 32
             : 16;
}

// Wave-uniform position of one step.
struct MStep {
  int di;      // descriptor
  int unit;    // unit within the GEMV
  int c;       // step within the unit
  bool last;   // last step of the unit
  bool valid;
};

template <bool BF16, bool XS, bool TABLE>
__global__ void __launch_bounds__(mfma_threads(BF16, XS)) bitcos_mfma_kernel(const KernelArgs a) {
  constexpr int CT = mfma_sign_copies(BF16);
  constexpr int THREADS = mfma_threads(BF16, XS);
  constexpr int WPB = THREADS / kWave;
  constexpr int RT = kMfmaRT;
  constexpr int ELEM = BF16 ? 2 : 1;  // bytes per activation
  constexpr int NA = BF16 ? 4 : 2;    // MFMAs (16-byte activation pieces) per word
  using CV = typename std::conditional<BF16, f32x4_t, i32x4_t>::type;

  __shared__ FastTables<BF16, CT> tab;
  __shared__ uint32_t sstage[WPB * kMfmaRows * kSignStride];
  __shared__ uint4 xbufs[WPB * mfma_xbuf_bytes(BF16) / 16];
  static_assert(sizeof(tab) + sizeof(sstage) + sizeof(xbufs) <= kLdsBytes, "small-batch kernel LDS");
  build_fast_tables<BF16, CT>(tab, threadIdx.x, THREADS);
  __syncthreads();

  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wave = __builtin_amdgcn_readfirstlane(blockIdx.x * WPB + wv);
  // The wave's share of the launch's steps: [S0, S1).
  const int total = static_cast<int>(a.total_units);
  const int nwaves = static_cast<int>(gridDim.x) * WPB;
  const int per = (total + nwaves - 1) / nwaves;
  const int S0 = per * wave;
  const int U1 = min(S0 + per, total);
  if (S0 >= U1) return;

  const int nr = lane & 15;
  const int g = lane >> 4;
  const uint32_t gm1 = lane_mask((g & 1) != 0), gm2 = lane_mask((g & 2) != 0);
  const FastLane fl = fast_lane<BF16, CT>(lane);
  uint32_t* const stage = sstage + wv * (kMfmaRows * kSignStride);
  uint8_t* const xbuf = reinterpret_cast<uint8_t*>(xbufs) + wv * mfma_xbuf_bytes(BF16);
  constexpr int XROW = mfma_xrow(BF16);
  constexpr int XLR = BF16 ? 16 : 8;  // lanes per batch row in a coalesced load (16-byte pieces)

  // ---- fetch side: the GEMV whose step is being fetched; fbeg / fend: its
  // first step in the launch and one past its last, fC: steps per unit.
  int fdi = 0, fbeg = 0, fend = 0, fC = 1, fG = 1, fk = 0, fupr = 0, fM = 0;
  rsrc_t rb = make_rsrc(nullptr, 0), rg = rb, rs = rb, rx = rb, rxs = rb;
  auto fetch_enter = [&](int d) {
    fdi = __builtin_amdgcn_readfirstlane(d);
    const auto& D = desc_at<TABLE>(a, fdi);
    fbeg = static_cast<int>(D.unit_begin);
    fend = static_cast<int>(D.unit_begin + D.units);
    fG = D.ngroups;
    fC = (fG + 3) >> 2;
    fk = D.upr * 32;
    fM = static_cast<int>(D.x_bytes / (static_cast<uint32_t>(fk) * ELEM));  // activation rows
    fupr = D.upr;
    rb = make_rsrc(D.sec0, D.sec0_bytes);
    rg = make_rsrc(D.signs, D.signs_bytes);
    // Scales are read three dwords at a time; a dword past the section reads
    // zero, so the range is rounded up to whole dwords (at most two padding
    // bytes of the blob, whose size is a multiple of 256).
    rs = make_rsrc(D.scales, (D.mode & kModeGrouped) ? (D.scales_bytes + 3u) & ~3u : 0u);
    rx = make_rsrc(D.x, D.x_bytes);
    const bool xs = XS && (D.mode & kModeXscale);
    rxs = make_rsrc(xs ? D.xscale : nullptr, xs ? D.x_bytes / (32u * ELEM) : 0u);
  };
  // Sign offsets of the lane's rows in the unit starting at row0 of GEMV d
  // (nothing when `in` is false).
  auto load_offsets = [&](int d, int row0, bool in, uint32_t (&o)[RT]) {
    const auto& D = desc_at<TABLE>(a, d);
    const rsrc_t ro = make_rsrc(D.offsets, static_cast<uint32_t>(D.n + 1) * 4u);
#pragma unroll
    for (int r = 0; r < RT; ++r)
      o[r] = ld32(ro, in ? static_cast<uint32_t>(row0 + kMfmaTile * r + nr) * 4u : kOOB);
  };
  // ... of the unit after unit u of the GEMV being fetched: unit u + 1, or the
  // next GEMV's first unit; read only if that unit starts inside the wave's
  // share (past the wave's last unit, u may be stale: nothing is read then,
  // or rows of a unit of the same GEMV, inside its buffer, that go unused).
  auto next_unit_offsets = [&](int u, uint32_t (&o)[RT]) {
    const int start = fbeg + (u + 1) * fC;
    const bool same = start < fend;
    load_offsets(same ? fdi : min(fdi + 1, a.count - 1), same ? (u + 1) * kMfmaRows : 0, start < U1, o);
  };

  // First unit: the first one of the launch to start at or after S0.
  int u0 = 0;
  {
    int lo = 0;
    if constexpr (TABLE) {  // last descriptor with unit_begin <= S0
      int hi = a.count;
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (((CDesc*)a.table)[mid].unit_begin <= S0) lo = mid; else hi = mid;
      }
    }
    fetch_enter(lo);
    u0 = (S0 - fbeg + fC - 1) / fC;
    if (fbeg + u0 * fC >= fend) {  // no unit of this GEMV starts in the share
      if (fend >= U1) return;
      fetch_enter(fdi + 1);
      u0 = 0;
    }
    if (fbeg + u0 * fC >= U1) return;
  }

  // Step data: presence words, fp16 group scales and sign dwords of the
  // lane's row in each tile, and the row's sign position at the step start.
  struct Slot {
    uint32_t P[RT][4];
    uint32_t SC[RT][3];  // the dwords holding the row's four fp16 group scales of the step
    uint32_t SSH[RT];    // bit offset of the first scale in SC
    u32x4_t SA[RT];
    uint32_t SB[RT];
    uint32_t pos[RT];
  };
  // Every load splits its offset into a lane part (voffset) and a
  // wave-uniform part (soffset: the unit's rows, the step, the group), so the
  // addresses cost scalar instructions; a load with nothing to read gets
  // soffset kOOB.
  auto issue = [&](const MStep& s, Slot& d) {
    const uint32_t c = static_cast<uint32_t>(s.valid ? s.c : 0);
    const uint32_t row0 = static_cast<uint32_t>(s.unit * kMfmaRows);
    // Presence: lane (nr, g) reads group g of the step (its four words, 16
    // bytes); place() transposes the four lanes' groups so that each lane
    // holds its word g of every group.
    const uint32_t lp = (static_cast<uint32_t>(nr) * static_cast<uint32_t>(fupr) + 4u * g) * 4u;
    const bool okg = s.valid && static_cast<int>(4 * c + g) < fG;
    const uint32_t ls = __umul24(static_cast<uint32_t>(nr), static_cast<uint32_t>(fG)) * 2u;
#pragma unroll
    for (int r = 0; r < RT; ++r) {
      const uint32_t rowr = row0 + kMfmaTile * r;
      const uint32_t sp = (rowr * static_cast<uint32_t>(fupr) + 16u * c) * 4u;
      const uint32_t ss = (rowr * static_cast<uint32_t>(fG) + 4u * c) * 2u;
      const u32x4_t pv = ld128_s(rb, okg ? lp : kOOB, __builtin_amdgcn_readfirstlane(s.valid ? sp : kOOB));
#pragma unroll
      for (int q = 0; q < 4; ++q) d.P[r][q] = pv[q];
      // The step's four scales of the row (8 bytes at a 2-byte aligned
      // offset) in one load of the three dwords that hold them.  Groups past
      // the row's last (last step of a unit) read scales of the next row or
      // zero; their products are zero.
      const uint32_t sa = ls + ss;
      const auto v3 = __builtin_amdgcn_raw_buffer_load_b96(rs, sa & ~3u, __builtin_amdgcn_readfirstlane(s.valid ? 0u : kOOB), 0);
      d.SC[r][0] = v3[0];
      d.SC[r][1] = v3[1];
      d.SC[r][2] = v3[2];
      d.SSH[r] = (sa & 2u) << 3;
      const uint32_t sdw = d.pos[r] >> 5;
      const uint32_t sv = __builtin_amdgcn_readfirstlane(s.valid ? 0u : kOOB);
      d.SA[r] = ld128_s(rg, (sdw + 4u * g) * 4u, sv);
      d.SB[r] = __builtin_amdgcn_raw_buffer_load_b32(rg, (sdw + 16u + g) * 4u, sv, 0);
    }
  };
  // Activations of group q of a step: 32 of batch row nr at the lane's word
  // (and with XS, the activation scales of batch rows 4 g + i).
  u32x4_t A[4][NA];
  // Activation scales of the step (XS): lane (nr, g) holds batch row
  // 4 g + nr % 4 at the step's four groups; a lane takes batch row 4 g + i's
  // from lane i of its quad.
  u32x4_t XV = {0u, 0u, 0u, 0u};
  auto issue_x = [&](const MStep& s, int q) {
    const uint32_t gi = static_cast<uint32_t>(4 * (s.valid ? s.c : 0) + q);
    const bool ok = s.valid && static_cast<int>(gi) < fG;
    const uint32_t ukk = static_cast<uint32_t>(fk);
    // Load jj covers batch rows (64 / XLR) jj .. of the group, each row's 128
    // activations as contiguous 16-byte pieces (lane l: row (64 / XLR) jj +
    // l / XLR, piece l % XLR).
    const uint32_t lx = static_cast<uint32_t>(lane / XLR) * ukk * ELEM + 16u * static_cast<uint32_t>(lane % XLR);
    // Loads whose batch rows are all past M are skipped: those rows' MFMA
    // results are never stored, so stale registers there are harmless.
#pragma unroll
    for (int jj = 0; jj < NA; ++jj) {
      const uint32_t so = (static_cast<uint32_t>((64 / XLR) * jj) * ukk + 128u * gi) * ELEM;
      if (jj == 0 || (64 / XLR) * jj < fM) A[q][jj] = ld128_s(rx, lx, __builtin_amdgcn_readfirstlane(ok ? so : kOOB));
    }
    if constexpr (XS) {
      if (q == 3) {  // after the step's last group: all four groups' scales in one load
        const uint32_t la = static_cast<uint32_t>(4 * g + (nr & 3)) * static_cast<uint32_t>(fG) * 4u;
        XV = ld128_s(rxs, la, __builtin_amdgcn_readfirstlane(s.valid ? 16u * static_cast<uint32_t>(s.c) : kOOB));
      }
    }
  };
  auto advance = [&](const MStep& s) {
    MStep n = s;
    if (s.c + 1 < fC) {
      n.c = s.c + 1;
    } else {  // the next unit: u + 1, or the next GEMV's first; it is the wave's if it starts before U1
      const int start = fbeg + (s.unit + 1) * fC;
      const bool same = start < fend;
      n.valid = start < U1;
      if (n.valid && !same) fetch_enter(fdi + 1);
      n.di = fdi;
      n.unit = same ? s.unit + 1 : 0;
      n.c = 0;
    }
    n.last = n.c + 1 == fC;
    return n;
  };

  // ---- decode side: output of the GEMV whose step is being decoded
  int ddi = -1, dn = 0;
  // scaled: per-group fp32 accumulation; dxs: the GEMV has activation scales
  bool grouped = false, raw = false, scaled = false, dxs = false, dadd = false;
  float tscale = 0.0f;
  rsrc_t ry = make_rsrc(nullptr, 0);

  // Accumulators: batch rows 4 g + i of output row nr of each tile.
  float acc[RT][4];
  int iacc[RT][4];
#pragma unroll
  for (int r = 0; r < RT; ++r)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      acc[r][i] = 0.0f;
      iacc[r][i] = 0;
    }

  // ---- prologue
  MStep fs;
  fs.di = fdi;
  fs.unit = u0;
  fs.c = 0;
  fs.last = fC == 1;
  fs.valid = true;
  Slot cur, nxt;
  uint32_t offn[RT];
  load_offsets(fdi, u0 * kMfmaRows, true, cur.pos);
  issue(fs, cur);
  next_unit_offsets(u0, offn);
#pragma unroll
  for (int q = 0; q < 4; ++q) issue_x(fs, q);

  // A step's word positions and staged signs are prepared at the end of the
  // step before it (the prologue for the first), while that step's MFMAs
  // drain, so a step starts with its window reads.
  // Word positions: popcounts exchanged among the four lanes of each row.
  uint32_t rel[RT][4];
  uint32_t stot[RT];
  auto place = [&](Slot& sl) {
#pragma unroll
    for (int r = 0; r < RT; ++r) {
      transpose_lanes16(sl.P[r]);
      uint32_t v = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) v |= static_cast<uint32_t>(__builtin_popcount(sl.P[r][q])) << (8 * q);
      const uint32_t b = xor16(v);
      const uint32_t pair = v + b;
      const uint32_t c2 = xor32(pair);
      const uint32_t excl = (b & gm1) + (c2 & gm2);
      const uint32_t tot = pair + c2;  // bytes <= 128
      uint32_t cum = sl.pos[r] & 31u;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        rel[r][q] = cum + __builtin_amdgcn_ubfe(excl, 8 * q, 8);
        cum += __builtin_amdgcn_ubfe(tot, 8 * q, 8);
      }
      stot[r] = cum - (sl.pos[r] & 31u);
    }
  };
  // A step's sign dwords into the wave's LDS block (the previous step's
  // window reads have all returned: their lookups fed its MFMAs).
  auto stage_signs = [&](const Slot& sl) {
#pragma unroll
    for (int r = 0; r < RT; ++r) {
      uint32_t* row = stage + (kMfmaTile * r + nr) * kSignStride;
#pragma unroll
      for (int j = 0; j < 4; ++j) row[4 * g + j] = sl.SA[r][j];
      row[16 + g] = sl.SB[r];
    }
    __builtin_amdgcn_wave_barrier();
  };
  place(cur);
  stage_signs(cur);

  for (;;) {
    const MStep cs = fs;
    if (!cs.valid) break;
    if (cs.di != ddi) {
      ddi = cs.di;
      const auto& D = desc_at<TABLE>(a, ddi);
      dn = D.n;
      grouped = (D.mode & kModeGrouped) != 0;
      raw = !BF16 && (D.mode & kModeRaw);
      dadd = (D.mode & kModeAdd) != 0;
      dxs = XS && (D.mode & kModeXscale);
      scaled = !raw && (grouped || dxs);
      tscale = half_bits_to_float(gp_u16(D.scales)[0]);
      ry = make_rsrc(D.y, D.y_bytes);
    }

    // Fetch step t+1.  offn holds the offsets of the unit after step t's:
    // step t+1's own when it starts a unit.
    fs = advance(cs);
#pragma unroll
    for (int r = 0; r < RT; ++r) nxt.pos[r] = fs.c == 0 ? offn[r] : cur.pos[r] + stot[r];
    // The unit after step t+1's is read only when step t+1 ends its unit (a
    // lane-masked branch: loads under a uniform branch into this
    // loop-carried register would make the compiler copy it into place).
    if (lane_mask(fs.last)) next_unit_offsets(fs.unit, offn);
    issue(fs, nxt);

    // The groups at raised wave priority (as in the batch-1 kernels): int8
    // 9 % faster at M = 4 on the Qwen3-32B-like layers, bf16 1.5 %.
    __builtin_amdgcn_s_setprio(1);
    // Groups: the MFMAs of group q, then the epilogue of group q - 1 (whose
    // MFMAs have had a group's worth of work to finish).
    CV cg[2][RT];
    const u32x4_t xv = XV;  // this step's activation scales (the next step's load reuses XV)
    auto epilogue = [&](int q, const CV (&c)[RT]) {
      float xa[4] = {1.0f, 1.0f, 1.0f, 1.0f};
      if (XS && dxs) {
        xa[0] = qperm<0x00>(bits_as<float>(xv[q]));
        xa[1] = qperm<0x55>(bits_as<float>(xv[q]));
        xa[2] = qperm<0xAA>(bits_as<float>(xv[q]));
        xa[3] = qperm<0xFF>(bits_as<float>(xv[q]));
      }
#pragma unroll
      for (int r = 0; r < RT; ++r) {
        if (scaled) {
          const uint32_t pair = __builtin_amdgcn_alignbit(cur.SC[r][q / 2 + 1], cur.SC[r][q / 2], cur.SSH[r]);
          const float sc = (grouped ? half_bits_to_float(static_cast<uint16_t>(q & 1 ? pair >> 16 : pair)) : tscale) *
                           (BF16 ? 2.0f : 1.0f);
#pragma unroll
          for (int i = 0; i < 4; ++i)
            acc[r][i] = __builtin_fmaf(dxs ? sc * xa[i] : sc, static_cast<float>(c[r][i]), acc[r][i]);
        } else if constexpr (BF16) {
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[r][i] += static_cast<float>(c[r][i]);
        } else {
#pragma unroll
          for (int i = 0; i < 4; ++i) iacc[r][i] += static_cast<int>(c[r][i]);
        }
      }
    };
    // Table lookups of a group: per tile, the lane's word and its 64-bit
    // sign window from the staged block.  bf16 looks group 0 up here and, in
    // group q, group q + 1 while q's weights are built and multiplied; int8
    // looks each group up where it is used.  The two tiles' MFMA chains
    // alternate so consecutive MFMAs do not depend on each other.
    auto lookup1 = [&](int q, int r) {
      const uint32_t* srow = stage + (kMfmaTile * r + nr) * kSignStride;
      const uint32_t bpos = rel[r][q];
      const uint32_t S = __builtin_amdgcn_alignbit(srow[(bpos >> 5) + 1], srow[bpos >> 5], bpos);
      return fast_look<BF16, CT>(cur.P[r][q], S, tab, fl);
    };
    // The MFMAs of one tile's word: (bf16) 4 MFMAs of 8 weights, (int8) 2 of
    // 16, each weight dword perm(T[s], E[m]).
    auto mfma_word = [&](const Look<BF16>& L, const u32x4_t (&Aq)[NA], int j, CV c) {
      if constexpr (BF16) {
        const uint2 th = L.th[j];
        const uint4 sb = L.sb[j];
        const u32x4_t w = {__builtin_amdgcn_perm(th.y, th.x, sb.x), __builtin_amdgcn_perm(th.y, th.x, sb.y),
                           __builtin_amdgcn_perm(th.y, th.x, sb.z), __builtin_amdgcn_perm(th.y, th.x, sb.w)};
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, Aq[j]),
                                                       __builtin_bit_cast(bf16x8_t, w), c, 0, 0, 0);
      } else {
        const uint2 t0 = L.tv[2 * j], e0 = L.sv[2 * j];
        const uint2 t1 = L.tv[2 * j + 1], e1 = L.sv[2 * j + 1];
        const u32x4_t w = {__builtin_amdgcn_perm(t0.y, t0.x, e0.x), __builtin_amdgcn_perm(t0.y, t0.x, e0.y),
                           __builtin_amdgcn_perm(t1.y, t1.x, e1.x), __builtin_amdgcn_perm(t1.y, t1.x, e1.y)};
        return __builtin_amdgcn_mfma_i32_16x16x64_i8(__builtin_bit_cast(i32x4_t, Aq[j]),
                                                     __builtin_bit_cast(i32x4_t, w), c, 0, 0, 0);
      }
    };
    constexpr bool LA = mfma_lookahead(BF16);
    Look<BF16> lk[2][RT];
    if constexpr (LA) {
#pragma unroll
      for (int r = 0; r < RT; ++r) lk[0][r] = lookup1(0, r);
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (LA && q + 1 < 4) {
#pragma unroll
        for (int r = 0; r < RT; ++r) lk[(q + 1) & 1][r] = lookup1(q + 1, r);
      }
      // The group's activations in MFMA order, through the wave's transpose
      // buffer: lane (nr, g) takes batch row nr at its word's pieces.
      u32x4_t Aq[NA];
#pragma unroll
      for (int jj = 0; jj < NA; ++jj)
        *reinterpret_cast<u32x4_t*>(xbuf + ((64 / XLR) * jj + lane / XLR) * XROW + 16 * (lane % XLR)) = A[q][jj];
#pragma unroll
      for (int j = 0; j < NA; ++j) Aq[j] = *reinterpret_cast<const u32x4_t*>(xbuf + nr * XROW + 16 * (NA * g + j));
      CV c[RT];
#pragma unroll
      for (int r = 0; r < RT; ++r) c[r] = CV{0, 0, 0, 0};
      if constexpr (LA) {  // the two tiles' chains alternate
#pragma unroll
        for (int j = 0; j < NA; ++j)
#pragma unroll
          for (int r = 0; r < RT; ++r) c[r] = mfma_word(lk[q & 1][r], Aq, j, c[r]);
      } else {  // one tile's lookups live at a time
#pragma unroll
        for (int r = 0; r < RT; ++r) {
          const Look<BF16> L = lookup1(q, r);
#pragma unroll
          for (int j = 0; j < NA; ++j) c[r] = mfma_word(L, Aq, j, c[r]);
        }
      }
#pragma unroll
      for (int r = 0; r < RT; ++r) cg[q & 1][r] = c[r];
      // This group's activations are consumed: fetch step t+1's.
      issue_x(fs, q);
      if (q > 0) epilogue(q - 1, cg[(q - 1) & 1]);
    }
    epilogue(3, cg[1]);
    __builtin_amdgcn_s_setprio(0);
    __builtin_amdgcn_wave_barrier();

    if (cs.last) {  // store the unit: y[m][row]; rows past n and batch rows past M are dropped
      const int row0 = cs.unit * kMfmaRows;
#pragma unroll
      for (int r = 0; r < RT; ++r) {
        const int row = row0 + kMfmaTile * r + nr;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const uint32_t off = row < dn ? (static_cast<uint32_t>((4 * g + i) * dn) + row) * 4u : kOOB;
          float f;
          if (scaled)
            f = acc[r][i];
          else if constexpr (BF16)
            f = tscale * (2.0f * acc[r][i]);
          else
            f = tscale * static_cast<float>(iacc[r][i]);
          const uint32_t bits = raw ? static_cast<uint32_t>(iacc[r][i]) : __builtin_bit_cast(uint32_t, f);
          put_y(bits, ry, off, 0, dadd, raw);
          acc[r][i] = 0.0f;
          iacc[r][i] = 0;
        }
      }
    }
    // The next step's positions and signs (its loads were issued a step ago).
    place(nxt);
    stage_signs(nxt);
    cur = nxt;
  }
}

using MfmaFn = void (*)(const KernelArgs);

template <bool BF16, bool XS>
MfmaFn pick_mfma_t(bool table) {
  return table ? bitcos_mfma_kernel<BF16, XS, true> : bitcos_mfma_kernel<BF16, XS, false>;
}

inline MfmaFn pick_mfma(bool bf16, bool xs, bool table) {
  if (bf16) return xs ? pick_mfma_t<true, true>(table) : pick_mfma_t<true, false>(table);
  return xs ? pick_mfma_t<false, true>(table) : pick_mfma_t<false, false>(table);
}

}  // namespace bitcos_k
