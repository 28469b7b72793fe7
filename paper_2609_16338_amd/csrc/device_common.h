// Device helpers shared by the three GEMV kernels: wave scans and segmented
// reductions over 64-wide wavefronts, byte packing, and the per-lane group
// bookkeeping of the scale epilogue.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bitcos_dev {

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Pointers into global memory.  Descriptor fields are generic pointers; using
// them through these types makes every access a global_* instruction (a flat
// access would also count against the LDS counter and serialise the
// prefetched loads with the table lookups).
typedef const __attribute__((address_space(1))) uint32_t* g_u32;
typedef const __attribute__((address_space(1))) uint16_t* g_u16;
typedef const __attribute__((address_space(1))) float* g_f32;
typedef __attribute__((address_space(1))) int* g_i32_out;
typedef __attribute__((address_space(1))) float* g_f32_out;

// Read-only for the whole kernel (descriptor tables, unit offsets): the
// constant address space lets these wave-uniform reads go through the scalar
// cache into SGPRs.
typedef const __attribute__((address_space(4))) uint32_t* c_u32;
__device__ __forceinline__ c_u32 cp_u32(const void* p) { return (c_u32)p; }

__device__ __forceinline__ g_u32 gp_u32(const void* p) { return (g_u32)p; }
__device__ __forceinline__ g_u16 gp_u16(const void* p) { return (g_u16)p; }
__device__ __forceinline__ g_f32 gp_f32(const void* p) { return (g_f32)p; }
__device__ __forceinline__ g_i32_out gp_i32_out(void* p) { return (g_i32_out)p; }
__device__ __forceinline__ g_f32_out gp_f32_out(void* p) { return (g_f32_out)p; }

// Buffer resources: a load through one checks its byte offset against the
// resource size and returns 0 past it, so lanes with nothing to read (a
// ragged last lane, rows past the end) pass kOOB and need no branch.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr uint32_t kOOB = 0x80000000u;  // past every section (sections are < 2 GiB)

__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), static_cast<short>(0),
                                           static_cast<int>(bytes), 0x00020000);
}
__device__ __forceinline__ uint32_t ld32(rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
}
__device__ __forceinline__ uint16_t ld16(rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0);
}

// One output element through a buffer resource (dropped past its range): a
// store, or with `add` an atomic add onto what y holds (fp32; int32 for raw
// sums).  A launch writes each element once, so the additions of launches
// that follow one another on a stream happen in that order and the result
// is deterministic.
__device__ __forceinline__ void put_y(uint32_t bits, rsrc_t r, uint32_t voff, uint32_t soff, bool add, bool raw) {
  if (!add)
    __builtin_amdgcn_raw_buffer_store_b32(bits, r, voff, soff, 0);
  else if (raw)
    __builtin_amdgcn_raw_ptr_buffer_atomic_add_i32(static_cast<int>(bits), r, voff, soff, 0);
  else
    __builtin_amdgcn_raw_ptr_buffer_atomic_fadd_f32(__builtin_bit_cast(float, bits), r, voff, soff, 0);
}

// Waits until every vector-memory access of the wave has completed: vmcnt 0,
// the LDS/scalar and export counts untouched (s_waitcnt immediate 0x0F70 on
// gfx9).  Issued through the builtin rather than inline asm so that the
// compiler's own wait insertion sees it: registers those accesses filled are
// then known to be ready, and no counted wait for them is placed after loads
// issued later (which would also wait for those later loads).  The empty asm
// keeps memory accesses (LDS reads of data staged by LDS-DMA) from moving
// above it.
__device__ __forceinline__ void wait_vmem_all() {
  __builtin_amdgcn_s_waitcnt(0x0F70);
  asm volatile("" ::: "memory");
}

constexpr int kWave = 64;
constexpr int kBlock = 256;  // 4 waves per workgroup

// Inclusive prefix sum over the 64 lanes of a wavefront (DPP row shifts inside
// each 16-lane row, then row broadcasts 15 and 31 across rows).
__device__ __forceinline__ int wave_incl_scan(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, false);  // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, false);  // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, false);  // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, false);  // row_shr:8
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xA, 0xF, false);  // row_bcast:15 -> rows 1, 3
  v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xC, 0xF, false);  // row_bcast:31 -> rows 2, 3
  return v;
}

__device__ __forceinline__ int lane63(int v) { return __builtin_amdgcn_readlane(v, 63); }

// Sum over aligned segments of SEG lanes with DPP moves (no LDS traffic).
// The sum is complete in the segment's last lane (j == SEG - 1); for
// SEG <= 16 every lane of the segment holds it.  The order of the additions
// is fixed, so float results are deterministic.
//   SEG 2, 4: quad_perm swaps (lane ^ 1, lane ^ 2);
//   SEG 8:    half-row mirror (lane i <-> 7 - i), then the two quad swaps;
//   SEG 16:   row rotations by 8, 4, 2, 1;
//   SEG 32:   row sums, then row 1 (3) adds lane 15 of row 0 (2);
//   SEG 64:   as 32, then row 3 adds lane 31.
template <int CTRL, int ROWS = 0xF>
__device__ __forceinline__ int dpp_i(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, ROWS, 0xF, false);
}

// Segments of a width that is not a power of two (SEG lanes from lane
// SEG * r) do not line up with DPP rows: lane j of a segment adds the value
// of the lane d below it, for d = 1, 2, 4, ... < SEG, where j >= d (lane moves
// through ds_bpermute, which touches no LDS memory).  After the last round
// lane j holds the sum of the segment's lanes max(0, j - 2^r + 1) .. j, so the
// last lane holds the whole segment's sum, as above.
template <int SEG, class T>
__device__ __forceinline__ T seg_sum_any(T v) {
  const int lane = static_cast<int>(__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u)));
  const int j = lane % SEG;
#pragma unroll
  for (int d = 1; d < SEG; d <<= 1) {
    const int o = __builtin_amdgcn_ds_bpermute(((lane - d) & 63) << 2, __builtin_bit_cast(int, v));
    v += j >= d ? __builtin_bit_cast(T, o) : T(0);
  }
  return v;
}

template <int SEG>
__device__ __forceinline__ int seg_sum(int v) {
  if constexpr (SEG & (SEG - 1)) {
    return seg_sum_any<SEG>(v);
  } else {
    static_assert(SEG == 2 || SEG == 4 || SEG == 8 || SEG == 16 || SEG == 32 || SEG == 64, "segment");
    if constexpr (SEG == 8) v += dpp_i<0x141>(v);  // row_half_mirror
    if constexpr (SEG <= 8) {
      v += dpp_i<0xB1>(v);                          // quad_perm [1,0,3,2]
      if constexpr (SEG >= 4) v += dpp_i<0x4E>(v);  // quad_perm [2,3,0,1]
    } else {
      v += dpp_i<0x128>(v);  // row_ror:8
      v += dpp_i<0x124>(v);  // row_ror:4
      v += dpp_i<0x122>(v);  // row_ror:2
      v += dpp_i<0x121>(v);  // row_ror:1
      if constexpr (SEG >= 32) v += dpp_i<0x142, 0xA>(v);  // row_bcast:15 into rows 1, 3
      if constexpr (SEG == 64) v += dpp_i<0x143, 0x8>(v);  // row_bcast:31 into row 3
    }
    return v;
  }
}

template <int CTRL, int ROWS = 0xF>
__device__ __forceinline__ float dpp_f(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, ROWS, 0xF, false));
}

template <int SEG>
__device__ __forceinline__ float seg_sum(float v) {
  if constexpr (SEG & (SEG - 1)) {
    return seg_sum_any<SEG>(v);
  } else {
    static_assert(SEG == 2 || SEG == 4 || SEG == 8 || SEG == 16 || SEG == 32 || SEG == 64, "segment");
    if constexpr (SEG == 8) v += dpp_f<0x141>(v);
    if constexpr (SEG <= 8) {
      v += dpp_f<0xB1>(v);
      if constexpr (SEG >= 4) v += dpp_f<0x4E>(v);
    } else {
      v += dpp_f<0x128>(v);
      v += dpp_f<0x124>(v);
      v += dpp_f<0x122>(v);
      v += dpp_f<0x121>(v);
      if constexpr (SEG >= 32) v += dpp_f<0x142, 0xA>(v);
      if constexpr (SEG == 64) v += dpp_f<0x143, 0x8>(v);
    }
    return v;
  }
}

__device__ __forceinline__ uint32_t bytes4(uint32_t b0, uint32_t b1, uint32_t b2, uint32_t b3) {
  return (b0 & 0xFF) | (b1 & 0xFF) << 8 | (b2 & 0xFF) << 16 | (b3 & 0xFF) << 24;
}

__device__ __forceinline__ float half_bits_to_float(uint16_t h) {
  return static_cast<float>(__builtin_bit_cast(_Float16, h));
}

__device__ __forceinline__ int sdot4(uint32_t a, uint32_t b, int c) {
  return __builtin_amdgcn_sdot4(static_cast<int>(a), static_cast<int>(b), c, false);
}

__device__ __forceinline__ float bdot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                         __builtin_bit_cast(bf16x2_t, b), c, false);
}

// Running sum at the last unit of every scale group a lane touches.
//
// A lane owns units [u0, u0 + PER) of a row (units of UPG per scale group);
// run[i] is the running accumulator after unit i, constant past the lane's
// last real unit.  With phase ph = u0 % UPG, group q of the lane ends at unit
// UPG*q + UPG - 1 - ph (clamped to PER - 1).  NQ = number of groups a lane can
// touch.  The phase is a run-time lane value; when PER is a multiple of UPG
// every lane starts on a group boundary and ph is 0.
template <int PER, int UPG>
struct GroupEnds {
  static constexpr bool kAligned = PER % UPG == 0;
  static constexpr int kNQ = kAligned ? PER / UPG : (PER + 2 * UPG - 2) / UPG;

  template <class T>
  __device__ __forceinline__ static T pick(const T (&run)[PER], int q, int ph) {
    if (kAligned) {
      const int e = UPG * q + UPG - 1;
      return run[e < PER ? e : PER - 1];
    }
    T r = T(0);
#pragma unroll
    for (int p = 0; p < UPG; ++p) {
      int e = UPG * q + UPG - 1 - p;
      if (e > PER - 1) e = PER - 1;
      if (e >= 0) r = (ph == p) ? run[e] : r;
    }
    return r;
  }
};

}  // namespace bitcos_dev
