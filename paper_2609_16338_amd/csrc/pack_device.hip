// Device-side BITCOS packer: the same blob bytes as bitcos_pack, computed on
// the GPU from a ternary matrix already in device memory (Sec. II-A: presence
// bitmap + sign vector compacted to the non-zeros, in row-major order).
//
//   plan:  one wave per row counts its non-zeros (and flags values outside
//          {-1, 0, 1}); one workgroup turns the counts into exclusive row
//          offsets; the total is read back to size the sign section.
//   pack:  the blob is zeroed; one wave per row walks the row's 32-weight
//          words 64 at a time, writes each presence word, compacts the word's
//          sign bits (negative weights among the present ones, in order) and
//          ORs them into the sign stream at the row offset plus a wavefront
//          prefix of the words' popcounts; then the unit offsets (row offsets
//          at unit boundaries) and the scales (validated) are written.
//
// Workspace layout (caller device memory, bitcos_plan_device_workspace bytes):
//   u32[0] value flag (weight outside {-1,0,1}, bad scale, or W changed
//          between plan and pack), u32[1] unused, u64 at byte 8: nnz,
//   u32[4 ..] row offsets, n + 1 entries.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "../../include/bitcos.h"
#include "device_common.h"
#include "launch_common.h"
#include "plan.h"

namespace {

using namespace bitcos_dev;

constexpr int kRowsPerBlock = 4;  // one wave per row
constexpr int kScanThreads = 1024;

struct WsHeader {
  uint32_t flag;
  uint32_t unused;
  uint64_t nnz;
};
static_assert(sizeof(WsHeader) == 16, "workspace header is 16 bytes");

__device__ __forceinline__ uint32_t* ws_rows(void* ws) {
  return reinterpret_cast<uint32_t*>(static_cast<uint8_t*>(ws) + sizeof(WsHeader));
}

// Presence and negative masks of 4 weights (one dword of int8) at bits
// [4 * part, 4 * part + 4); `bad` collects values outside {-1, 0, 1}.
__device__ __forceinline__ void classify4(uint32_t v, int part, uint32_t& pres, uint32_t& neg, uint32_t& bad) {
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const uint32_t byte = (v >> (8 * b)) & 0xFFu;
    pres |= uint32_t(byte != 0u) << (4 * part + b);
    neg |= uint32_t(byte == 0xFFu) << (4 * part + b);
    bad |= uint32_t(byte != 0u && byte != 1u && byte != 0xFFu);
  }
}

// Presence / negative words of the 32 weights starting at weight 32 * word of
// row `row` (zero past the end of the row or matrix).
__device__ __forceinline__ void word_masks(rsrc_t rw, int row, int k, int word, uint32_t& pres,
                                           uint32_t& neg, uint32_t& bad) {
  pres = 0;
  neg = 0;
  const bool in = word < k / 32;
  const uint32_t off = in ? (static_cast<uint32_t>(row) * static_cast<uint32_t>(k) + 32u * word) : kOOB;
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const uint4 q = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rw, off + 16u * c, 0, 0));
    classify4(q.x, 4 * c + 0, pres, neg, bad);
    classify4(q.y, 4 * c + 1, pres, neg, bad);
    classify4(q.z, 4 * c + 2, pres, neg, bad);
    classify4(q.w, 4 * c + 3, pres, neg, bad);
  }
}

__global__ void __launch_bounds__(kRowsPerBlock * kWave) count_rows_kernel(const int8_t* w, int n, int k, void* ws) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
  if (row >= n) return;  // whole wave
  const rsrc_t rw = make_rsrc(w, static_cast<uint32_t>(n) * static_cast<uint32_t>(k));
  uint32_t cnt = 0, bad = 0;
  for (int w0 = 0; w0 < k / 32; w0 += kWave) {
    uint32_t pres, neg;
    word_masks(rw, row, k, w0 + lane, pres, neg, bad);
    cnt += __builtin_popcount(pres);
  }
  const int tot = seg_sum<64>(static_cast<int>(cnt));
  if (lane == 63) ws_rows(ws)[row] = static_cast<uint32_t>(tot);
  if (bad) atomicOr(&static_cast<WsHeader*>(ws)->flag, 1u);
}

// Exclusive scan of the n row counts in place (row offsets), total into the
// header and row n.  One workgroup; each thread owns a contiguous slice.
__global__ void __launch_bounds__(kScanThreads) scan_rows_kernel(int n, void* ws) {
  __shared__ uint64_t part[kScanThreads];
  uint32_t* rows = ws_rows(ws);
  const int t = threadIdx.x;
  const int per = (n + kScanThreads - 1) / kScanThreads;
  const int lo = min(n, t * per), hi = min(n, lo + per);
  uint64_t s = 0;
  for (int i = lo; i < hi; ++i) s += rows[i];
  part[t] = s;
  __syncthreads();
  for (int d = 1; d < kScanThreads; d <<= 1) {  // inclusive Hillis-Steele scan
    const uint64_t v = t >= d ? part[t - d] : 0;
    __syncthreads();
    part[t] += v;
    __syncthreads();
  }
  uint64_t run = part[t] - s;  // exclusive prefix of this slice
  for (int i = lo; i < hi; ++i) {
    const uint32_t c = rows[i];
    rows[i] = static_cast<uint32_t>(run);
    run += c;
  }
  if (t == kScanThreads - 1) {
    const uint64_t total = part[t];
    static_cast<WsHeader*>(ws)->nnz = total;
    rows[n] = static_cast<uint32_t>(total);
  }
}

// Compact the sign bits of the present weights of one word, in order.
__device__ __forceinline__ uint32_t compact_signs(uint32_t pres, uint32_t neg) {
  uint32_t out = 0;
  int q = 0;
  while (pres) {
    const int b = __builtin_ctz(pres);
    out |= ((neg >> b) & 1u) << q;
    ++q;
    pres &= pres - 1u;
  }
  return out;
}

__global__ void __launch_bounds__(kRowsPerBlock * kWave)
    pack_rows_kernel(const int8_t* w, int n, int k, void* ws, uint32_t* bitmap, uint32_t* signs, uint64_t nnz) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
  if (row >= n) return;  // whole wave
  const uint32_t* rows = ws_rows(ws);
  const uint32_t start = rows[row], end = rows[row + 1];
  const rsrc_t rw = make_rsrc(w, static_cast<uint32_t>(n) * static_cast<uint32_t>(k));
  const int upr = k / 32;
  uint32_t carry = start, bad = 0;
  for (int w0 = 0; w0 < upr; w0 += kWave) {
    const int word = w0 + lane;
    uint32_t pres, neg;
    word_masks(rw, row, k, word, pres, neg, bad);
    const int pc = __builtin_popcount(pres);
    const int incl = wave_incl_scan(pc);
    const uint32_t pos = carry + static_cast<uint32_t>(incl - pc);
    carry += static_cast<uint32_t>(lane63(incl));
    if (word < upr) bitmap[static_cast<size_t>(row) * upr + word] = pres;
    // The planned row range bounds every write (W changed since the plan:
    // flagged, nothing written outside the row's range).
    if (pc > 0 && pos + static_cast<uint32_t>(pc) <= end && end <= nnz) {
      const uint32_t cs = compact_signs(pres, neg);
      const uint32_t d = pos >> 5, sh = pos & 31u;
      if (cs) {
        atomicOr(&signs[d], cs << sh);
        if (sh + static_cast<uint32_t>(pc) > 32u) atomicOr(&signs[d + 1], cs >> (32u - sh));
      }
    } else if (pc > 0) {
      bad = 1;
    }
  }
  if (lane == 63 && carry != end) bad = 1;
  if (bad) atomicOr(&static_cast<WsHeader*>(ws)->flag, 1u);
}

__global__ void offsets_kernel(const void* ws, int n, int unit_rows, int units, uint32_t* offsets) {
  const int u = blockIdx.x * blockDim.x + threadIdx.x;
  if (u > units) return;
  const uint32_t* rows = reinterpret_cast<const uint32_t*>(static_cast<const uint8_t*>(ws) + sizeof(WsHeader));
  offsets[u] = rows[min(static_cast<int64_t>(u) * unit_rows, static_cast<int64_t>(n))];
}

__global__ void scales_kernel(const uint16_t* src, int64_t count, uint16_t* dst, void* ws) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= count) return;
  const uint16_t h = src[i];
  dst[i] = h;
  if ((h & 0x8000u) || (h & 0x7C00u) == 0x7C00u) atomicOr(&static_cast<WsHeader*>(ws)->flag, 1u);
}

int check_shape(int32_t n, int32_t k, int32_t group, int32_t unit_rows) {
  if (n < 1 || k < 1 || unit_rows < 0) return BITCOS_E_ARG;
  if (group != 0 && group != 128) return BITCOS_E_ARG;
  if (k % (group == 128 ? 128 : 32)) return BITCOS_E_ARG;
  if (static_cast<int64_t>(n) * k >= (int64_t(1) << 31)) return BITCOS_E_UNSUPPORTED;  // buffer ranges
  return BITCOS_OK;
}

int sync_status(hipStream_t st) {
  if (hipGetLastError() != hipSuccess) return BITCOS_E_HIP;
  if (hipStreamSynchronize(st) != hipSuccess) return BITCOS_E_HIP;
  return BITCOS_OK;
}

// Workspace of bitcos_pack_device_noalloc for matrices of up to
// BITCOS_NOALLOC_MAX_ROWS rows: the header and n + 1 row offsets of the
// plan.  One copy per GPU the library runs on, held until the process ends.
constexpr size_t kNoallocBytes =
    (sizeof(WsHeader) + 4u * (static_cast<size_t>(BITCOS_NOALLOC_MAX_ROWS) + 1) + 15u) / 16u * 16u;
__device__ __align__(256) uint8_t scratch[kNoallocBytes];

constexpr int kMaxDevices = 64;

// Device address of this GPU's `scratch`, looked up once per device with
// that device current.  The host-side name of a __device__ array is not its
// device address; only this pointer may reach kernels and copies.
int noalloc_workspace(void** out) {
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return BITCOS_E_HIP;
  std::lock_guard<std::mutex> g(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return BITCOS_E_HIP;
    addr[dev] = p;
  }
  *out = addr[dev];
  return BITCOS_OK;
}

}  // namespace

extern "C" {

size_t bitcos_plan_device_workspace(int32_t n) {
  if (n < 1) return 0;
  return (sizeof(WsHeader) + 4u * (static_cast<size_t>(n) + 1) + 15u) / 16u * 16u;
}

int bitcos_plan_device(const int8_t* w_dev, int32_t n, int32_t k, int32_t group, int32_t unit_rows,
                       void* ws_dev, size_t ws_bytes, bitcos_layout* out, void* stream) {
  if (!w_dev || !ws_dev || !out) return BITCOS_E_ARG;
  int st = check_shape(n, k, group, unit_rows);
  if (st) return st;
  if (ws_bytes < bitcos_plan_device_workspace(n)) return BITCOS_E_SPACE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (hipMemsetAsync(ws_dev, 0, sizeof(WsHeader), s) != hipSuccess) return BITCOS_E_HIP;
  const unsigned blocks = static_cast<unsigned>((n + kRowsPerBlock - 1) / kRowsPerBlock);
  hipLaunchKernelGGL(count_rows_kernel, dim3(blocks), dim3(kRowsPerBlock * kWave), 0, s, w_dev, n, k, ws_dev);
  hipLaunchKernelGGL(scan_rows_kernel, dim3(1), dim3(kScanThreads), 0, s, n, ws_dev);
  WsHeader h;
  if (hipMemcpyAsync(&h, ws_dev, sizeof(h), hipMemcpyDeviceToHost, s) != hipSuccess) return BITCOS_E_HIP;
  st = sync_status(s);
  if (st) return st;
  if (h.flag) return BITCOS_E_VALUE;
  return bitcos::bitcos_layout_for(n, k, group, unit_rows, h.nnz, out);
}

int bitcos_pack_device(const int8_t* w_dev, const uint16_t* scales_dev, const bitcos_layout* L,
                       void* ws_dev, size_t ws_bytes, void* dst_dev, size_t cap, void* stream) {
  if (!w_dev || !scales_dev || !L || !ws_dev || !dst_dev) return BITCOS_E_ARG;
  if (L->version != BITCOS_LAYOUT_VERSION || L->format != BITCOS_FMT_BITCOS || L->unit_rows < 1)
    return BITCOS_E_ARG;
  int st = check_shape(L->n, L->k, L->group, L->unit_rows);
  if (st) return st;
  if (ws_bytes < bitcos_plan_device_workspace(L->n)) return BITCOS_E_SPACE;
  if (cap < L->total_bytes) return BITCOS_E_SPACE;
  bitcos_layout chk;  // the layout must be the one the plan gives for its nnz
  st = bitcos::bitcos_layout_for(L->n, L->k, L->group, L->unit_rows, L->nnz, &chk);
  if (st || chk.total_bytes != L->total_bytes || chk.sec_off[BITCOS_SEC_SCALES] != L->sec_off[BITCOS_SEC_SCALES])
    return BITCOS_E_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  uint8_t* blob = static_cast<uint8_t*>(dst_dev);
  if (hipMemsetAsync(blob, 0, L->total_bytes, s) != hipSuccess) return BITCOS_E_HIP;
  if (hipMemsetAsync(ws_dev, 0, sizeof(uint32_t), s) != hipSuccess) return BITCOS_E_HIP;  // value flag
  const int n = L->n, k = L->k;
  const unsigned blocks = static_cast<unsigned>((n + kRowsPerBlock - 1) / kRowsPerBlock);
  hipLaunchKernelGGL(pack_rows_kernel, dim3(blocks), dim3(kRowsPerBlock * kWave), 0, s, w_dev, n, k, ws_dev,
                     reinterpret_cast<uint32_t*>(blob + L->sec_off[BITCOS_SEC_BITMAP]),
                     reinterpret_cast<uint32_t*>(blob + L->sec_off[BITCOS_SEC_SIGNS]), L->nnz);
  const int units = (n + L->unit_rows - 1) / L->unit_rows;
  hipLaunchKernelGGL(offsets_kernel, dim3((units + 1 + 255) / 256), dim3(256), 0, s, ws_dev, n, L->unit_rows, units,
                     reinterpret_cast<uint32_t*>(blob + L->sec_off[BITCOS_SEC_OFFSETS]));
  const int64_t ns = L->group == 128 ? static_cast<int64_t>(n) * (k / 128) : 1;
  hipLaunchKernelGGL(scales_kernel, dim3(static_cast<unsigned>((ns + 255) / 256)), dim3(256), 0, s, scales_dev, ns,
                     reinterpret_cast<uint16_t*>(blob + L->sec_off[BITCOS_SEC_SCALES]), ws_dev);
  uint32_t flag = 0;
  if (hipMemcpyAsync(&flag, ws_dev, sizeof(flag), hipMemcpyDeviceToHost, s) != hipSuccess) return BITCOS_E_HIP;
  st = sync_status(s);
  if (st) return st;
  return flag ? BITCOS_E_VALUE : BITCOS_OK;
}

int bitcos_pack_device_noalloc(const int8_t* w_dev, const uint16_t* scales_dev, int32_t n, int32_t k,
                               int32_t group, int32_t unit_rows, bitcos_layout* out, void* dst_dev, size_t cap,
                               void* stream) {
  if (!w_dev || !scales_dev || !out || !dst_dev) return BITCOS_E_ARG;
  int st = check_shape(n, k, group, unit_rows);
  if (st) return st;
  if (n > BITCOS_NOALLOC_MAX_ROWS) return BITCOS_E_SPACE;  // more rows than the fixed workspace holds
  void* ws = nullptr;
  st = noalloc_workspace(&ws);
  if (st) return st;
  const size_t ws_bytes = bitcos_plan_device_workspace(n);
  st = bitcos_plan_device(w_dev, n, k, group, unit_rows, ws, ws_bytes, out, stream);
  if (st) return st;
  if (cap < out->total_bytes) return BITCOS_E_SPACE;  // *out tells the caller the size
  return bitcos_pack_device(w_dev, scales_dev, out, ws, ws_bytes, dst_dev, cap, stream);
}

}  // extern "C"
