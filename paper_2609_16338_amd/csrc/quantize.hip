// Per-group int8 quantisation of bf16 activations (Sec. II-C of "Breaking the
// 1.58-bit Barrier for Ternary LLMs": activations are quantised to int8 per
// group of 128 and the group scale is applied once per group).  The paper
// does not state the rule; this library uses the symmetric absmax one:
//   a = max|x| / 127 (fp32; a = 1 for an all-zero group),
//   q = clamp(round_half_even(x / a), -127, 127), divisions IEEE fp32.
// One wavefront per (row, group): each lane converts two bf16 values.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/bitcos.h"
#include "launch_common.h"

namespace {

__global__ void __launch_bounds__(256) quantize_kernel(const uint32_t* __restrict__ x, int32_t groups,
                                                       int64_t total, int8_t* __restrict__ q,
                                                       float* __restrict__ scale) {
  const int lane = threadIdx.x & 63;
  const int64_t gid = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (gid >= total) return;
  const uint32_t pair = x[gid * 64 + lane];
  const float v0 = __builtin_bit_cast(float, pair << 16);
  const float v1 = __builtin_bit_cast(float, pair & 0xFFFF0000u);
  float amax = fmaxf(fabsf(v0), fabsf(v1));
#pragma unroll
  for (int off = 32; off >= 1; off /= 2) amax = fmaxf(amax, __shfl_xor(amax, off, 64));
  const float a = amax == 0.0f ? 1.0f : __fdiv_rn(amax, 127.0f);
  const float q0 = fminf(fmaxf(rintf(__fdiv_rn(v0, a)), -127.0f), 127.0f);
  const float q1 = fminf(fmaxf(rintf(__fdiv_rn(v1, a)), -127.0f), 127.0f);
  const uint16_t packed = static_cast<uint16_t>(static_cast<uint8_t>(static_cast<int8_t>(q0))) |
                          static_cast<uint16_t>(static_cast<uint8_t>(static_cast<int8_t>(q1))) << 8;
  reinterpret_cast<uint16_t*>(q)[gid * 64 + lane] = packed;
  if (lane == 0) scale[gid] = a;
  (void)groups;
}

}  // namespace

extern "C" int bitcos_quantize_act(const void* x_bf16_dev, int32_t m, int32_t k, int8_t* q_dev,
                                   float* scale_dev, void* stream) {
  if (!x_bf16_dev || !q_dev || !scale_dev || m < 1 || k < 128 || k % 128) return BITCOS_E_ARG;
  const int64_t total = static_cast<int64_t>(m) * (k / 128);
  const int64_t blocks = (total + 3) / 4;
  if (blocks > 0x7FFFFFFF) return BITCOS_E_UNSUPPORTED;
  hipLaunchKernelGGL(quantize_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0,
                     static_cast<hipStream_t>(stream), static_cast<const uint32_t*>(x_bf16_dev),
                     k / 128, total, q_dev, scale_dev);
  return bitcos_launch_status();
}
