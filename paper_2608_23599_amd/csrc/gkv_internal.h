// Internal helpers shared by the host and device code of libgkv (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gkv.h"

#define GKV_HD __host__ __device__ __forceinline__

namespace gkv {

constexpr int D = 128;
constexpr int P = 64;
constexpr int KC = 4;
constexpr int kExactBytes = P * D * 2;  // 16384
constexpr int kSZBytes = 2 * D * 2;     // scale + zero, 512
constexpr int kCentBytes = KC * D * 2 + P * 2 / 8;  // 1040
constexpr int kMeanBytes = D * 2;                   // 256

GKV_HD int64_t block_bytes(int level) {
  switch (level) {
    case GKV_EXACT: return kExactBytes;
    case GKV_INT8: return kSZBytes + P * D;
    case GKV_INT4: return kSZBytes + P * D / 2;
    case GKV_INT2: return kSZBytes + P * D / 4;
    case GKV_CENTROID: return kCentBytes;
    case GKV_MEAN: return kMeanBytes;
    default: return 0;
  }
}

GKV_HD bool is_int_level(int level) { return level == GKV_INT8 || level == GKV_INT4 || level == GKV_INT2; }

// Ladder order: larger = more precise.
GKV_HD int level_rank(int level) {
  switch (level) {
    case GKV_MEAN: return 0;
    case GKV_CENTROID: return 1;
    case GKV_INT2: return 2;
    case GKV_INT4: return 3;
    case GKV_INT8: return 4;
    case GKV_EXACT: return 5;
    default: return -1;
  }
}

// ---------------------------------------------------------------- record layout
// Element n (0..31) of lane l's chunk -> (token, channel) inside the 64x128 block,
// for page `pg`.  See the layout description in gkv.h.
GKV_HD void chunk_coord(int tensor, int pg, int lane, int n, int &tok, int &ch) {
  const int kg = lane >> 4, m = lane & 15;
  if (tensor == GKV_KEYS) {
    tok = 16 * pg + m;
    ch = 32 * (n >> 3) + 8 * kg + (n & 7);
  } else {
    tok = 16 * pg + 4 * kg + (n & 3);
    ch = 16 * (n >> 2) + m;
  }
}

// Channel held by scale/zero entry e (lane order).
GKV_HD int sz_channel(int tensor, int e) {
  const int kg = e >> 5, n = e & 31;
  return tensor == GKV_KEYS ? 32 * (n >> 3) + 8 * kg + (n & 7) : 16 * (n >> 2) + 4 * kg + (n & 3);
}

// Bit position of code x_n inside its 32-bit word, and the word index.
GKV_HD int code_word(int bits, int n) { return n / (32 / bits); }
GKV_HD int code_pos(int bits, int n) {
  if (bits == 8) return 8 * (n & 3);
  if (bits == 4) {
    const int t[8] = {4, 20, 12, 28, 0, 16, 8, 24};
    return t[n & 7];
  }
  const int t[16] = {8, 24, 14, 30, 6, 22, 12, 28, 4, 20, 10, 26, 0, 16, 2, 18};
  return t[n & 15];
}

// Value-centroid storage index of (centroid k, channel d).
GKV_HD int vcent_index(int k, int d) { return ((d & 15) * 8 + (d >> 4)) * KC + k; }

// Page-box storage index (pair base, in uint16 units) of (page p, channel d) for one (b,h).
GKV_HD int64_t box_index(int64_t p, int d) { return (((p >> 6) * D + d) * 64 + (p & 63)) * 2; }

// ---------------------------------------------------------------- fp16 rounding
// fp64 -> fp16 bit pattern with a single round-to-nearest-even, written from the
// IEEE 754 encodings (the hardware has no direct fp64 -> fp16 conversion, and going
// through fp32 would round twice).
GKV_HD uint16_t f64_to_f16(double x) {
  uint64_t u;
  __builtin_memcpy(&u, &x, 8);
  const uint16_t sign = (uint16_t)((u >> 48) & 0x8000u);
  const int ex = (int)((u >> 52) & 0x7FF);
  const uint64_t man = u & 0xFFFFFFFFFFFFFull;
  if (ex == 0x7FF) return (uint16_t)(sign | 0x7C00u | (man ? 0x200u : 0u));
  if (ex == 0) return sign;  // fp64 zero or subnormal: far below half the fp16 subnormal unit
  const int e = ex - 1023;
  if (e > 15) return (uint16_t)(sign | 0x7C00u);
  if (e >= -14) {
    uint32_t hm = (uint32_t)(man >> 42);
    const uint64_t rem = man & ((1ull << 42) - 1);
    const uint64_t half = 1ull << 41;
    if (rem > half || (rem == half && (hm & 1u))) hm++;
    uint32_t he = (uint32_t)(e + 15);
    if (hm == 0x400u) {
      hm = 0;
      he++;
    }
    if (he >= 31u) return (uint16_t)(sign | 0x7C00u);
    return (uint16_t)(sign | (he << 10) | hm);
  }
  // fp16 subnormal range: result = round(value / 2^-24)
  const int s = 28 - e;  // >= 43
  if (s >= 64) return sign;
  const uint64_t mf = (1ull << 52) | man;
  uint64_t q = mf >> s;
  const uint64_t rem = mf & ((1ull << s) - 1);
  const uint64_t half = 1ull << (s - 1);
  if (rem > half || (rem == half && (q & 1ull))) q++;
  return (uint16_t)(sign | (uint16_t)q);
}

GKV_HD uint16_t canon_zero(uint16_t h) { return h == 0x8000u ? (uint16_t)0 : h; }

GKV_HD double f16_to_f64(uint16_t h) {
  // exact widening, written out so the host and device agree bit for bit
  const uint32_t sign = h >> 15, ex = (h >> 10) & 0x1F, man = h & 0x3FF;
  double v;
  if (ex == 0) {
    v = (double)man * 0x1p-24;
  } else if (ex == 31) {
    v = man ? __builtin_nan("") : __builtin_inf();
  } else {
    v = (double)(man | 0x400) * __builtin_ldexp(1.0, (int)ex - 25);
  }
  return sign ? -v : v;
}

}  // namespace gkv

// Host-side validation shared by the call wrappers (host.cpp).
gkv_status gkv_validate_cache(const gkv_cache *c);

// Writes seq_len[b] = v on the device, ordered on `stream` (encode.hip).
gkv_status gkv_launch_set_len(int64_t *seq_len, int b, int64_t v, hipStream_t stream);

// Tokens of sequence b (-1: retired), from the host mirror.
inline int64_t seq_tokens(const gkv_cache *c, int b) { return c->seq_len_host ? c->seq_len_host[b] : c->T; }

// Compute units of the current device (cached per device; attn.hip).
int gkv_device_cus();

// Sets c->version to a new process-wide unique stamp (host.cpp); every call that
// changes the block tables, T or nres calls it on success.
void gkv_stamp(gkv_cache *c);
void gkv_append_commit(gkv_cache *c, bool any_open);
constexpr int GKV_APPEND_LAYERS = 16;  // layers of one multi-layer append launch
gkv_status gkv_launch_append_layers(gkv_cache *const *caches, int L, const uint16_t *k_new, const uint16_t *v_new,
                                    hipStream_t stream);
