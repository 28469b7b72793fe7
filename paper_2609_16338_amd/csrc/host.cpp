// Host half of libbitcos: status strings, validation, and the plan / pack /
// unpack functions of the three formats (BITCOS, five-trit, 2-bit).
//
// BITCOS (Sec. II-A of "Breaking the 1.58-bit Barrier for Ternary LLMs"):
// one presence bit per weight plus one sign bit per non-zero weight, both in
// row-major tensor order, least significant bit first.  The packer writes the
// two streams in one pass over W, the per-unit sign offsets from per-row
// counts, and the fp16 scales verbatim.
#include <cstdint>
#include <cstring>
#include <vector>

#include "../../include/bitcos.h"
#include "plan.h"

namespace {

constexpr uint64_t kAlign = 256;
constexpr uint64_t kSignPad = 16;
constexpr uint64_t kTrit5Pad = 16;
constexpr int kTrit5Block = 26;

uint64_t round_up(uint64_t v, uint64_t a) { return (v + a - 1) / a * a; }

// fp16 bit pattern is finite and non-negative (+0 allowed).
bool scale_ok(uint16_t h) { return (h & 0x8000u) == 0 && (h & 0x7C00u) != 0x7C00u; }

int64_t num_scales(int32_t n, int32_t k, int32_t group) {
  return group == 128 ? int64_t(n) * (k / 128) : 1;
}

// Lay out sections 0..3 with the given byte lengths (0 = absent) at 256-byte
// boundaries, in index order.
void place_sections(bitcos_layout* L, const uint64_t bytes[4]) {
  uint64_t pos = 0;
  for (int s = 0; s < 4; ++s) {
    L->sec_bytes[s] = bytes[s];
    if (bytes[s] == 0) {
      L->sec_off[s] = 0;
      continue;
    }
    pos = round_up(pos, kAlign);
    L->sec_off[s] = pos;
    pos += bytes[s];
  }
  L->total_bytes = round_up(pos, kAlign);
}

int check_common(const int8_t* w, int32_t n, int32_t k, int32_t group, int k_mult) {
  if (!w || n < 1 || k < 1) return BITCOS_E_ARG;
  if (group != 0 && group != 128) return BITCOS_E_ARG;
  if (k % k_mult) return BITCOS_E_ARG;
  return BITCOS_OK;
}

// Count non-zeros; E_VALUE if any weight lies outside {-1, 0, 1}.
int count_nnz(const int8_t* w, int64_t count, uint64_t* nnz) {
  uint64_t c = 0;
  int bad = 0;
  for (int64_t i = 0; i < count; ++i) {
    int v = w[i];
    bad |= (v < -1) | (v > 1);
    c += v != 0;
  }
  if (bad) return BITCOS_E_VALUE;
  *nnz = c;
  return BITCOS_OK;
}

int check_layout(const bitcos_layout* L, uint32_t fmt) {
  if (!L || L->version != BITCOS_LAYOUT_VERSION || L->format != fmt) return BITCOS_E_ARG;
  if (L->n < 1 || L->k < 1 || (L->group != 0 && L->group != 128)) return BITCOS_E_ARG;
  return BITCOS_OK;
}

int check_scales(const uint16_t* s, int64_t count) {
  if (!s) return BITCOS_E_ARG;
  for (int64_t i = 0; i < count; ++i)
    if (!scale_ok(s[i])) return BITCOS_E_VALUE;
  return BITCOS_OK;
}

}  // namespace

extern "C" {

const char* bitcos_strerror(int status) {
  switch (status) {
    case BITCOS_OK: return "ok";
    case BITCOS_E_ARG: return "invalid argument";
    case BITCOS_E_VALUE: return "invalid value (weight, scale or blob contents)";
    case BITCOS_E_SPACE: return "destination buffer too small";
    case BITCOS_E_HIP: return "HIP runtime or launch error";
    case BITCOS_E_UNSUPPORTED: return "no kernel for this shape, dtype or batch";
    default: return "unknown status";
  }
}

uint32_t bitcos_version(void) { return BITCOS_LAYOUT_VERSION; }

}  // extern "C"

// ---------------------------------------------------------------------------
// BITCOS
// ---------------------------------------------------------------------------

namespace bitcos {

int bitcos_layout_for(int32_t n, int32_t k, int32_t group, int32_t unit_rows, uint64_t nnz,
                      bitcos_layout* out) {
  if (nnz > 0xFFFFFFFFull) return BITCOS_E_UNSUPPORTED;  // 32-bit sign offsets
  if (unit_rows == 0) unit_rows = bitcos::bitcos_default_unit_rows(n, k);
  bitcos_layout L;
  std::memset(&L, 0, sizeof(L));
  L.version = BITCOS_LAYOUT_VERSION;
  L.format = BITCOS_FMT_BITCOS;
  L.n = n;
  L.k = k;
  L.group = group;
  L.unit_rows = unit_rows;
  L.nnz = nnz;
  const uint64_t nunits = (uint64_t(n) + unit_rows - 1) / unit_rows;
  const int64_t ns = num_scales(n, k, group);
  uint64_t bytes[4] = {
      uint64_t(n) * uint64_t(k) / 8,
      (nnz + 31) / 32 * 4 + kSignPad,
      (nunits + 1) * 4,
      uint64_t(ns) * 2,
  };
  place_sections(&L, bytes);
  L.payload_bits = uint64_t(n) * uint64_t(k) + nnz + 16ull * uint64_t(ns);
  *out = L;
  return BITCOS_OK;
}

}  // namespace bitcos

extern "C" {

int bitcos_plan(const int8_t* w, int32_t n, int32_t k, int32_t group, int32_t unit_rows,
                bitcos_layout* out) {
  if (!out) return BITCOS_E_ARG;
  int st = check_common(w, n, k, group, group == 128 ? 128 : 32);
  if (st) return st;
  if (unit_rows < 0) return BITCOS_E_ARG;
  uint64_t nnz = 0;
  st = count_nnz(w, int64_t(n) * k, &nnz);
  if (st) return st;
  return bitcos::bitcos_layout_for(n, k, group, unit_rows, nnz, out);
}

int bitcos_pack(const int8_t* w, const uint16_t* scales_f16, const bitcos_layout* L, void* dst,
                size_t cap) {
  int st = check_layout(L, BITCOS_FMT_BITCOS);
  if (st) return st;
  if (!w || !dst || L->unit_rows < 1) return BITCOS_E_ARG;
  const int32_t n = L->n, k = L->k;
  if (k % (L->group == 128 ? 128 : 32)) return BITCOS_E_ARG;
  if (cap < L->total_bytes) return BITCOS_E_SPACE;
  const int64_t ns = num_scales(n, k, L->group);
  st = check_scales(scales_f16, ns);
  if (st) return st;

  uint8_t* blob = static_cast<uint8_t*>(dst);
  std::memset(blob, 0, L->total_bytes);
  uint32_t* bitmap = reinterpret_cast<uint32_t*>(blob + L->sec_off[BITCOS_SEC_BITMAP]);
  uint32_t* signs = reinterpret_cast<uint32_t*>(blob + L->sec_off[BITCOS_SEC_SIGNS]);
  uint32_t* offs = reinterpret_cast<uint32_t*>(blob + L->sec_off[BITCOS_SEC_OFFSETS]);

  // One pass: build each 32-weight presence word and append the signs of its
  // non-zeros to the sign stream at the running bit position.
  const uint64_t words = uint64_t(n) * uint64_t(k) / 32;
  const uint64_t sign_words = (L->nnz + 31) / 32;
  uint64_t bitpos = 0;
  const int32_t words_per_row = k / 32;
  const uint64_t nunits = (uint64_t(n) + L->unit_rows - 1) / L->unit_rows;
  for (uint64_t wi = 0; wi < words; ++wi) {
    if (wi % words_per_row == 0) {
      uint64_t row = wi / words_per_row;
      if (row % L->unit_rows == 0) {
        if (bitpos > 0xFFFFFFFFull) return BITCOS_E_VALUE;
        offs[row / L->unit_rows] = uint32_t(bitpos);
      }
    }
    const int8_t* src = w + wi * 32;
    uint32_t pres = 0, neg = 0;
    int cnt = 0;
    for (int b = 0; b < 32; ++b) {
      int v = src[b];
      if (v < -1 || v > 1) return BITCOS_E_VALUE;
      if (v != 0) {
        pres |= 1u << b;
        neg |= uint32_t(v < 0) << cnt;
        ++cnt;
      }
    }
    bitmap[wi] = pres;
    if (cnt) {
      if (bitpos + cnt > L->nnz) return BITCOS_E_VALUE;  // W differs from the planned one
      const uint64_t word = bitpos >> 5;
      const uint32_t sh = uint32_t(bitpos & 31);
      signs[word] |= neg << sh;
      if (sh && sh + cnt > 32) signs[word + 1] |= neg >> (32 - sh);
      bitpos += cnt;
    }
  }
  if (bitpos != L->nnz) return BITCOS_E_VALUE;
  (void)sign_words;
  offs[nunits] = uint32_t(bitpos);
  std::memcpy(blob + L->sec_off[BITCOS_SEC_SCALES], scales_f16, size_t(ns) * 2);
  return BITCOS_OK;
}

int bitcos_unpack(const bitcos_layout* L, const void* blob_v, size_t blob_bytes, int8_t* w_out,
                  uint16_t* scales_out) {
  int st = check_layout(L, BITCOS_FMT_BITCOS);
  if (st) return st;
  if (!blob_v || !w_out || !scales_out || L->unit_rows < 1) return BITCOS_E_ARG;
  if (blob_bytes < L->total_bytes) return BITCOS_E_SPACE;
  const uint8_t* blob = static_cast<const uint8_t*>(blob_v);
  const int32_t n = L->n, k = L->k;
  const uint32_t* bitmap = reinterpret_cast<const uint32_t*>(blob + L->sec_off[BITCOS_SEC_BITMAP]);
  const uint32_t* signs = reinterpret_cast<const uint32_t*>(blob + L->sec_off[BITCOS_SEC_SIGNS]);
  const uint32_t* offs = reinterpret_cast<const uint32_t*>(blob + L->sec_off[BITCOS_SEC_OFFSETS]);
  const uint64_t words = uint64_t(n) * uint64_t(k) / 32;
  const int32_t words_per_row = k / 32;
  uint64_t bitpos = 0;
  for (uint64_t wi = 0; wi < words; ++wi) {
    if (wi % words_per_row == 0) {
      uint64_t row = wi / words_per_row;
      if (row % L->unit_rows == 0 && offs[row / L->unit_rows] != bitpos) return BITCOS_E_VALUE;
    }
    uint32_t pres = bitmap[wi];
    int8_t* d = w_out + wi * 32;
    for (int b = 0; b < 32; ++b) {
      if (pres >> b & 1u) {
        if (bitpos >= L->nnz) return BITCOS_E_VALUE;
        uint32_t s = signs[bitpos >> 5] >> (bitpos & 31) & 1u;
        d[b] = s ? int8_t(-1) : int8_t(1);
        ++bitpos;
      } else {
        d[b] = 0;
      }
    }
  }
  const uint64_t nunits = (uint64_t(n) + L->unit_rows - 1) / L->unit_rows;
  if (bitpos != L->nnz || offs[nunits] != bitpos) return BITCOS_E_VALUE;
  std::memcpy(scales_out, blob + L->sec_off[BITCOS_SEC_SCALES],
              size_t(num_scales(n, k, L->group)) * 2);
  return BITCOS_OK;
}

// ---------------------------------------------------------------------------
// Five-trit baseline: 26 bytes per 128-weight block
// ---------------------------------------------------------------------------

static int fixed_rate_plan(const int8_t* w, int32_t n, int32_t k, int32_t group, uint32_t fmt,
                           bitcos_layout* out) {
  if (!out) return BITCOS_E_ARG;
  int st = check_common(w, n, k, group, 128);
  if (st) return st;
  uint64_t nnz = 0;
  st = count_nnz(w, int64_t(n) * k, &nnz);
  if (st) return st;
  bitcos_layout L;
  std::memset(&L, 0, sizeof(L));
  L.version = BITCOS_LAYOUT_VERSION;
  L.format = fmt;
  L.n = n;
  L.k = k;
  L.group = group;
  L.unit_rows = 0;
  L.nnz = nnz;
  const int64_t ns = num_scales(n, k, group);
  const uint64_t blocks = uint64_t(n) * (k / 128);
  uint64_t code_bytes = fmt == BITCOS_FMT_TRIT5 ? blocks * kTrit5Block + kTrit5Pad : blocks * 32;
  uint64_t bytes[4] = {code_bytes, 0, 0, uint64_t(ns) * 2};
  place_sections(&L, bytes);
  uint64_t sym = fmt == BITCOS_FMT_TRIT5 ? blocks * kTrit5Block * 8 : 2ull * n * uint64_t(k);
  L.payload_bits = sym + 16ull * uint64_t(ns);
  *out = L;
  return BITCOS_OK;
}

int trit5_plan(const int8_t* w, int32_t n, int32_t k, int32_t group, bitcos_layout* out) {
  return fixed_rate_plan(w, n, k, group, BITCOS_FMT_TRIT5, out);
}

int bit2_plan(const int8_t* w, int32_t n, int32_t k, int32_t group, bitcos_layout* out) {
  return fixed_rate_plan(w, n, k, group, BITCOS_FMT_BIT2, out);
}

static int fixed_rate_prologue(const bitcos_layout* L, uint32_t fmt, const int8_t* w,
                               const uint16_t* scales, void* dst, size_t cap) {
  int st = check_layout(L, fmt);
  if (st) return st;
  if (!w || !dst || L->k % 128) return BITCOS_E_ARG;
  if (cap < L->total_bytes) return BITCOS_E_SPACE;
  return check_scales(scales, num_scales(L->n, L->k, L->group));
}

int trit5_pack(const int8_t* w, const uint16_t* scales_f16, const bitcos_layout* L, void* dst,
               size_t cap) {
  int st = fixed_rate_prologue(L, BITCOS_FMT_TRIT5, w, scales_f16, dst, cap);
  if (st) return st;
  uint8_t* blob = static_cast<uint8_t*>(dst);
  std::memset(blob, 0, L->total_bytes);
  uint8_t* codes = blob + L->sec_off[BITCOS_SEC_CODES];
  const uint64_t blocks = uint64_t(L->n) * (L->k / 128);
  for (uint64_t b = 0; b < blocks; ++b) {
    const int8_t* src = w + b * 128;
    uint8_t* out = codes + b * kTrit5Block;
    for (int j = 0; j < kTrit5Block; ++j) {
      int val = 0, pow3 = 1;
      for (int t = 0; t < 5; ++t, pow3 *= 3) {
        int idx = 5 * j + t;
        int digit = 1;  // weight 0 for positions past the block
        if (idx < 128) {
          int v = src[idx];
          if (v < -1 || v > 1) return BITCOS_E_VALUE;
          digit = v + 1;
        }
        val += digit * pow3;
      }
      out[j] = uint8_t(val);
    }
  }
  std::memcpy(blob + L->sec_off[BITCOS_SEC_SCALES], scales_f16,
              size_t(num_scales(L->n, L->k, L->group)) * 2);
  return BITCOS_OK;
}

int trit5_unpack(const bitcos_layout* L, const void* blob_v, size_t blob_bytes, int8_t* w_out,
                 uint16_t* scales_out) {
  int st = check_layout(L, BITCOS_FMT_TRIT5);
  if (st) return st;
  if (!blob_v || !w_out || !scales_out || L->k % 128) return BITCOS_E_ARG;
  if (blob_bytes < L->total_bytes) return BITCOS_E_SPACE;
  const uint8_t* blob = static_cast<const uint8_t*>(blob_v);
  const uint8_t* codes = blob + L->sec_off[BITCOS_SEC_CODES];
  const uint64_t blocks = uint64_t(L->n) * (L->k / 128);
  for (uint64_t b = 0; b < blocks; ++b) {
    int8_t* out = w_out + b * 128;
    for (int j = 0; j < kTrit5Block; ++j) {
      int val = codes[b * kTrit5Block + j];
      if (val > 242) return BITCOS_E_VALUE;
      for (int t = 0; t < 5; ++t) {
        int digit = val % 3;
        val /= 3;
        int idx = 5 * j + t;
        if (idx < 128)
          out[idx] = int8_t(digit - 1);
        else if (digit != 1)
          return BITCOS_E_VALUE;
      }
    }
  }
  std::memcpy(scales_out, blob + L->sec_off[BITCOS_SEC_SCALES],
              size_t(num_scales(L->n, L->k, L->group)) * 2);
  return BITCOS_OK;
}

// ---------------------------------------------------------------------------
// 2-bit baseline: code w + 1, 16 weights per u32
// ---------------------------------------------------------------------------

int bit2_pack(const int8_t* w, const uint16_t* scales_f16, const bitcos_layout* L, void* dst,
              size_t cap) {
  int st = fixed_rate_prologue(L, BITCOS_FMT_BIT2, w, scales_f16, dst, cap);
  if (st) return st;
  uint8_t* blob = static_cast<uint8_t*>(dst);
  std::memset(blob, 0, L->total_bytes);
  uint32_t* codes = reinterpret_cast<uint32_t*>(blob + L->sec_off[BITCOS_SEC_CODES]);
  const uint64_t words = uint64_t(L->n) * uint64_t(L->k) / 16;
  for (uint64_t i = 0; i < words; ++i) {
    const int8_t* src = w + i * 16;
    uint32_t word = 0;
    for (int t = 0; t < 4; ++t)
      for (int b = 0; b < 4; ++b) {
        int v = src[4 * t + b];
        if (v < -1 || v > 1) return BITCOS_E_VALUE;
        word |= uint32_t(v + 1) << (8 * b + 2 * t);
      }
    codes[i] = word;
  }
  std::memcpy(blob + L->sec_off[BITCOS_SEC_SCALES], scales_f16,
              size_t(num_scales(L->n, L->k, L->group)) * 2);
  return BITCOS_OK;
}

int bit2_unpack(const bitcos_layout* L, const void* blob_v, size_t blob_bytes, int8_t* w_out,
                uint16_t* scales_out) {
  int st = check_layout(L, BITCOS_FMT_BIT2);
  if (st) return st;
  if (!blob_v || !w_out || !scales_out || L->k % 128) return BITCOS_E_ARG;
  if (blob_bytes < L->total_bytes) return BITCOS_E_SPACE;
  const uint8_t* blob = static_cast<const uint8_t*>(blob_v);
  const uint32_t* codes = reinterpret_cast<const uint32_t*>(blob + L->sec_off[BITCOS_SEC_CODES]);
  const uint64_t words = uint64_t(L->n) * uint64_t(L->k) / 16;
  for (uint64_t i = 0; i < words; ++i) {
    uint32_t word = codes[i];
    for (int t = 0; t < 4; ++t)
      for (int b = 0; b < 4; ++b) {
        uint32_t c = word >> (8 * b + 2 * t) & 3u;
        if (c == 3) return BITCOS_E_VALUE;
        w_out[i * 16 + 4 * t + b] = int8_t(int(c) - 1);
      }
  }
  std::memcpy(scales_out, blob + L->sec_off[BITCOS_SEC_SCALES],
              size_t(num_scales(L->n, L->k, L->group)) * 2);
  return BITCOS_OK;
}

}  // extern "C"
