// Sum of the partial outputs of a split row: a GEMV whose rows are too long
// for one batch-1 tile is computed as column blocks, the first writing y and
// the others writing one slice each of a partial buffer (all in one launch),
// and this kernel adds the slices into y in block order.  Every element gets
// the same fp32 additions, in the same order, as the accumulating output
// modes would give it with one launch per block (Sec. II-C: the row sum over
// K taken block by block).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "../../include/bitcos.h"
#include "launch_common.h"

namespace {

constexpr int kPartialsThreads = 256;

// y[i] += parts[0][i] + ... + parts[nparts - 1][i], left to right; four
// consecutive elements per thread when the buffers are 16-byte aligned.
__global__ void __launch_bounds__(kPartialsThreads) add_partials_kernel(float* __restrict__ y,
                                                                        const float* __restrict__ parts,
                                                                        int32_t nparts, int64_t n, bool vec4) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kPartialsThreads;
  const int64_t t0 = static_cast<int64_t>(blockIdx.x) * kPartialsThreads + threadIdx.x;
  if (vec4) {
    const int64_t n4 = n / 4;
    for (int64_t i = t0; i < n4; i += stride) {
      float4 a = reinterpret_cast<const float4*>(y)[i];
      for (int32_t j = 0; j < nparts; ++j) {
        const float4 p = reinterpret_cast<const float4*>(parts + j * n)[i];
        a.x += p.x;
        a.y += p.y;
        a.z += p.z;
        a.w += p.w;
      }
      reinterpret_cast<float4*>(y)[i] = a;
    }
    for (int64_t i = 4 * n4 + t0; i < n; i += stride) {
      float a = y[i];
      for (int32_t j = 0; j < nparts; ++j) a += parts[j * n + i];
      y[i] = a;
    }
    return;
  }
  for (int64_t i = t0; i < n; i += stride) {
    float a = y[i];
    for (int32_t j = 0; j < nparts; ++j) a += parts[j * n + i];
    y[i] = a;
  }
}

}  // namespace

extern "C" int bitcos_add_partials(float* y_dev, const float* parts_dev, int32_t nparts, int64_t n,
                                   void* stream) {
  if (!y_dev || !parts_dev || nparts < 1 || n < 1) return BITCOS_E_ARG;
  const bool vec4 = (reinterpret_cast<uintptr_t>(y_dev) | reinterpret_cast<uintptr_t>(parts_dev)) % 16 == 0 &&
                    n % 4 == 0;
  const int64_t work = vec4 ? n / 4 : n;
  const int64_t blocks = std::min<int64_t>((work + kPartialsThreads - 1) / kPartialsThreads, 8192);
  hipLaunchKernelGGL(add_partials_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kPartialsThreads), 0,
                     static_cast<hipStream_t>(stream), y_dev, parts_dev, nparts, n, vec4);
  return bitcos_launch_status();
}
