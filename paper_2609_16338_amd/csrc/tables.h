// Deposit-form decode tables in LDS, shared by the BITCOS kernels that
// decode one presence byte with two table lookups and one v_perm_b32 per
// output dword (the batch-1 streaming kernel and the small-batch kernel).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "bitcos_kernel.h"

namespace bitcos_k {

// LDS of one workgroup on gfx950.
constexpr int kLdsBytes = 160 * 1024;

// Decode tables of the streaming kernel, in deposit form: perm(T[s], E[m])
// is the 8 weights of presence byte m (compact signs s) in position order,
// Eq. (2) w = p - 2n with the deposit of Sec. II-B done by the table.
//   E[m] bf16: 16 selector bytes for 8 bf16 weights (low byte 0x0C = zero,
//              high byte = rank of bit b in m, or 0x0C); int8: byte b = rank
//              of bit b, or 0x0C.
//   T[s] byte q: sign of the q-th non-zero, as the high byte of -+0.5 bf16
//              (0xBF / 0x3F) or as int8 -+1 (0xFF / 0x01).
// One LDS object laid out so that the byte offset of E[m] is one v_perm_b32
// of the presence word and a per-lane constant (m lands in byte 1, the copy
// offset in byte 0):
//   [0, 64 KB)   E: 256-byte rows, 16 copies of 16 bytes (bf16) or 32 copies
//                of 8 bytes (int8);
//   [64 KB, ...) T: 8-byte entries in CT copies (8 CT-byte rows).
// Lane l reads copy l % copies.  32 copies of an 8-byte entry keep any 32
// keys of a ds_read_b64 pass on distinct banks; a ds_read_b128 pass serves
// 16 lanes, for which 16 copies suffice.
template <bool BF16, int CT>
struct FastTables {
  static constexpr uint32_t kEsz = BF16 ? 16 : 8;
  static constexpr int kCE = 256 / kEsz;
  static constexpr uint32_t kT = 65536;
  static constexpr uint32_t kTStride = 8u * CT;
  static_assert(CT == 8 || CT == 16 || CT == 32, "sign-table copies");
  alignas(256) uint8_t bytes[kT + 256u * kTStride];
};

template <bool BF16, int CT>
__device__ __forceinline__ void build_fast_tables(FastTables<BF16, CT>& t, int tid, int nthreads) {
  using Tb = FastTables<BF16, CT>;
  // Each of the 256 entries is computed once, into the first 16 bytes of its
  // row (E: copy 0, or copies 0 and 1 of the 8-byte int8 entries; T: copies 0
  // and 1); the other copies are then 16-byte moves from there, so building
  // the tables costs every launch little next to its GEMVs.
  uint4* q = reinterpret_cast<uint4*>(t.bytes);
  if (tid < 256) {
    const uint32_t e = static_cast<uint32_t>(tid);
    uint32_t rk[8], g[8];
    uint32_t r = 0;
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const uint32_t on = e >> b & 1;
      rk[b] = on ? r : 0x0Cu;
      r += on;
      g[b] = on ? (BF16 ? 0xBFu : 0xFFu) : (BF16 ? 0x3Fu : 0x01u);
    }
    uint4 ev;
    if constexpr (BF16) {
      ev = make_uint4(bytes4(0x0C, rk[0], 0x0C, rk[1]), bytes4(0x0C, rk[2], 0x0C, rk[3]),
                      bytes4(0x0C, rk[4], 0x0C, rk[5]), bytes4(0x0C, rk[6], 0x0C, rk[7]));
    } else {
      const uint32_t lo = bytes4(rk[0], rk[1], rk[2], rk[3]), hi = bytes4(rk[4], rk[5], rk[6], rk[7]);
      ev = make_uint4(lo, hi, lo, hi);
    }
    const uint32_t glo = bytes4(g[0], g[1], g[2], g[3]), ghi = bytes4(g[4], g[5], g[6], g[7]);
    q[e * 16] = ev;
    q[(Tb::kT + e * Tb::kTStride) / 16] = make_uint4(glo, ghi, glo, ghi);
  }
  __syncthreads();
  for (int idx = tid; idx < 256 * 16; idx += nthreads) {
    const int k = idx & 15;
    if (k) q[idx] = q[idx - k];
  }
  constexpr int TC = CT / 2;  // 16-byte chunks per T row
  for (int idx = tid; idx < 256 * TC; idx += nthreads) {
    const int k = idx % TC;
    if (k) q[Tb::kT / 16 + idx] = q[Tb::kT / 16 + idx - k];
  }
}

// int8 arithmetic of one word from deposit-form lookups: perm(T[s], E[m])
// puts the 8 weights of presence byte m in position order (E[m] byte b =
// rank of bit b, or 0x0C for a zero weight; T[s] byte q = -1 or +1 for the
// q-th non-zero), and v_dot4 multiplies them with the position's 4 + 4
// activations (Eq. (2): w = p - 2n).
__device__ __forceinline__ int fast_math_i8(const LookI8& L, const uint32_t* x, int acc) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    acc = sdot4(__builtin_amdgcn_perm(L.tv[i].y, L.tv[i].x, L.sv[i].x), x[2 * i], acc);
    acc = sdot4(__builtin_amdgcn_perm(L.tv[i].y, L.tv[i].x, L.sv[i].y), x[2 * i + 1], acc);
  }
  return acc;
}

// Per-lane constants of the lookups: E copy offset; T base + copy offset.
struct FastLane {
  uint32_t ecp, tcp;
};

template <bool BF16, int CT>
__device__ __forceinline__ FastLane fast_lane(int lane) {
  using Tb = FastTables<BF16, CT>;
  FastLane f;
  f.ecp = static_cast<uint32_t>(lane & (Tb::kCE - 1)) * Tb::kEsz;
  f.tcp = Tb::kT + static_cast<uint32_t>(lane & (CT - 1)) * 8u;
  return f;
}

// Table lookups of one 32-weight word (presence word P, its compact signs S
// from bit 0).  Per presence byte m_i: E offset = perm(P, ecp) = m_i << 8 |
// copy; the byte's first sign is r_i = popcount of the earlier bytes (an LDS
// popcount table instead of v_bcnt measured slower: it adds a second
// dependent LDS round trip); the sign byte s_i = S >> r_i & 0xFF gives the T
// offset s_i * 8 CT | T base | copy (byte 0, r_0 = 0, with a 256-byte
// stride: one perm as well).
template <bool BF16, int CT>
__device__ __forceinline__ Look<BF16> fast_look(uint32_t P, uint32_t S, const FastTables<BF16, CT>& t,
                                                const FastLane& f) {
  using EE = typename std::conditional<BF16, uint4, uint2>::type;
  const uint8_t* b = t.bytes;
  Look<BF16> L;
  uint32_t r = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t eo = __builtin_amdgcn_perm(P, f.ecp, 0x0C0C0400u + (static_cast<uint32_t>(i) << 8));
    uint32_t to;
    if (i == 0 && CT == 32) {
      to = __builtin_amdgcn_perm(S, f.tcp, 0x0C020400u);
    } else {
      const uint32_t s = i == 0 ? (S & 0xFFu) : __builtin_amdgcn_ubfe(S, r, 8);
      to = (s << (CT == 32 ? 8 : CT == 16 ? 7 : 6)) | f.tcp;
    }
    if (i < 3) r = __builtin_popcount(__builtin_amdgcn_ubfe(P, 8 * i, 8)) + r;
    const EE ev = *reinterpret_cast<const EE*>(b + eo);
    const uint2 tv = *reinterpret_cast<const uint2*>(b + to);
    if constexpr (BF16) {
      L.sb[i] = ev;
      L.th[i] = tv;
    } else {
      L.sv[i] = ev;
      L.tv[i] = tv;
    }
  }
  return L;
}

}  // namespace bitcos_k
