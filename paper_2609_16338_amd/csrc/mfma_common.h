// Pieces shared by the kernels that multiply on the matrix cores: MFMA
// operand vector types, 16-byte buffer loads and cross-lane helpers.
#pragma once

#include "bitcos_kernel.h"

namespace bitcos_k {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef int i32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ u32x4_t ld128(rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}
__device__ __forceinline__ u32x4_t ld128_s(rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}

template <class T>
__device__ __forceinline__ T bits_as(uint32_t b) {
  return __builtin_bit_cast(T, b);
}
template <class T>
__device__ __forceinline__ uint32_t as_bits(T v) {
  return __builtin_bit_cast(uint32_t, v);
}
// A DPP quad permutation of v (CTRL: the quad_perm field).
template <int CTRL, class T>
__device__ __forceinline__ T qperm(T v) {
  return bits_as<T>(__builtin_amdgcn_update_dpp(0, as_bits(v), CTRL, 0xF, 0xF, false));
}

// A per-lane all-ones / all-zeros mask the compiler cannot see through.
// Conditions on cross-lane results are applied with these masks instead of
// selects: a select may be turned into a branch around the DPP or permlane
// move, which then runs with lanes switched off and reads them as zero.
__device__ __forceinline__ uint32_t lane_mask(bool on) {
  uint32_t m = on ? ~0u : 0u;
  asm volatile("" : "+v"(m));
  return m;
}

// The value of lane l ^ 16 and of lane l ^ 32: v_permlane16_swap exchanges
// the 16-lane rows of the pairs (0,1) and (2,3), v_permlane32_swap the wave's
// halves; with v in both operands the two results are v and the partner's
// value, so the partner's is their sum minus v (exact in modular arithmetic).
__device__ __forceinline__ uint32_t xor16(uint32_t v) {
  const auto p = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  return p[0] + p[1] - v;
}
__device__ __forceinline__ uint32_t xor32(uint32_t v) {
  const auto p = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return p[0] + p[1] - v;
}

// 4 x 4 transpose across the lanes l, l + 16, l + 32, l + 48: lane l + 16 a
// ends with v[b] = what lane l + 16 b held in v[a].  Two butterfly levels:
// v_permlane16_swap exchanges the odd 16-lane rows of its first operand with
// the even rows of its second (rows a and a ^ 1, components b and b ^ 1),
// v_permlane32_swap the upper half of its first operand with the lower half
// of its second (rows a and a ^ 2, components b and b ^ 2).
__device__ __forceinline__ void transpose_lanes16(uint32_t (&v)[4]) {
  const auto s01 = __builtin_amdgcn_permlane16_swap(v[0], v[1], false, false);
  const auto s23 = __builtin_amdgcn_permlane16_swap(v[2], v[3], false, false);
  v[0] = s01[0];
  v[1] = s01[1];
  v[2] = s23[0];
  v[3] = s23[1];
  const auto s02 = __builtin_amdgcn_permlane32_swap(v[0], v[2], false, false);
  const auto s13 = __builtin_amdgcn_permlane32_swap(v[1], v[3], false, false);
  v[0] = s02[0];
  v[2] = s02[1];
  v[1] = s13[0];
  v[3] = s13[1];
}

}  // namespace bitcos_k
