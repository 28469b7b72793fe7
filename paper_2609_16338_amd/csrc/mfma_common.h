// Pieces shared by the kernels that multiply on the matrix cores: MFMA
// operand vector types and the deposit-form decode tables.
#pragma once

#include "bitcos_kernel.h"

namespace bitcos_k {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef int i32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));

// int8 weights in deposit form: exp[e] byte b = rank of bit b among the set
// bits of e if bit b is set, else 0x0C (v_perm_b32 writes 0); tsg[e] byte q =
// 0xFF if bit q of e is set, else 0x01.  perm(tsg[s], exp[m]) is then the 8
// weights of presence byte m with compact signs s, as int8.
struct DepTablesI8 {
  uint2 exp[256 * Cfg<false>::kCopies];
  uint2 tsg[256 * Cfg<false>::kCopies];
};

template <bool BF16>
struct MfmaTables {
  using type = DepTablesI8;
};
template <>
struct MfmaTables<true> {
  using type = Tables<true>;
};

__device__ __forceinline__ void build_mfma_tables(DepTablesI8& t, int tid, int nthreads) {
  constexpr int NC = Cfg<false>::kCopies;
  for (int idx = tid; idx < 256 * NC; idx += nthreads) {
    const int e = idx & 255;
    const int c = idx >> 8;
    uint32_t ex[8], g[8];
    uint32_t r = 0;
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const bool on = (e >> b) & 1;
      ex[b] = on ? r : 0x0Cu;
      r += on;
      g[b] = on ? 0xFFu : 0x01u;
    }
    t.exp[e * NC + c] = make_uint2(bytes4(ex[0], ex[1], ex[2], ex[3]), bytes4(ex[4], ex[5], ex[6], ex[7]));
    t.tsg[e * NC + c] = make_uint2(bytes4(g[0], g[1], g[2], g[3]), bytes4(g[4], g[5], g[6], g[7]));
  }
}
__device__ __forceinline__ void build_mfma_tables(Tables<true>& t, int tid, int n) { build_tables<true>(t, tid, n); }

__device__ __forceinline__ u32x4_t ld128(rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}
__device__ __forceinline__ u32x4_t ld128_s(rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}

}  // namespace bitcos_k
