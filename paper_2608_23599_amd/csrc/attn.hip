// Fused dequant + online-softmax GQA decode attention over a graded cache
// (sections 3.1, 3.5 and 3.7), and the split-context reduction.
//
// Work split: grid (nsplit, Hkv, B) x 4 wavefronts.  Each wavefront owns a
// contiguous, byte-balanced range of "visits" (a block plus the 16-token tiles of
// it that are read) of one (b, KV head) and keeps an online-softmax state for
// the up-to-16 query heads of the group in MFMA accumulator layout.  The four
// wavefronts of a workgroup are merged in LDS into one partial (m, l, o) per
// head; the last workgroup of a (b, KV head) to finish merges its partials.
//
// Per 16-token tile the wavefront issues
//   S[token][head] = sum_d A[token][d] * B[d][head]       (4 x MFMA 16x16x32 f16)
// with A = the tile's key codes (every lane loads exactly its operand chunk; the
// packed record layout is built for it) and B = the group's queries, so one key
// tile feeds every query head of the group, and
//   O[d][head] += sum_t V[d][t] * P[t][head]              (8 x MFMA 16x16x16 f16)
// with P taken straight from the S accumulators.
//
// Integer codes enter the MFMA as fp16 (offset + code): the code bits are OR-ed
// into the mantissa of a fixed exponent (one v_and_or per two codes), which is
// exact.  For keys the per-channel scale is folded into the query as two fp16
// terms (q' = hi + lo of q * s) and the zero point and the offsets into one
// per-block constant computed by MFMA:  S = sum_d (off_d + c_d) q'_d
// + sum_d z_d q_d - sum_d off_d q'_d.  For values the per-channel scale and zero are applied
// once per block: O += s_d * (acc - off * sum_t p_t) + z_d * sum_t p_t.
#include <hip/hip_runtime.h>

#include "gkv_internal.h"

using namespace gkv;

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half4 __attribute__((ext_vector_type(4)));
typedef float f4 __attribute__((ext_vector_type(4)));

namespace {

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr float kNegInf = -__builtin_inff();
constexpr float kRescale = 8.0f;  // lazy rescale threshold (log2 units): p <= 2^8 in fp16

union U8 {
  half8 h;
  uint32_t u[4];
  uint4 v;
};
union U4 {
  half4 h;
  uint32_t u[2];
};

__device__ __forceinline__ f4 mfma32(half8 a, half8 b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f4 mfma16(half4 a, half4 b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x16f16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ uint32_t andor(uint32_t x, uint32_t m, uint32_t c) { return (x & m) | c; }
__device__ __forceinline__ uint32_t perm(uint32_t hi, uint32_t lo, uint32_t sel) {
  return __builtin_amdgcn_perm(hi, lo, sel);
}

// ---------------------------------------------------------------- code unpacking
// fp16 magic exponents: code bits at mantissa [p, p+b) of exponent e give 2^(10-p) + c.
constexpr uint32_t M1024 = 0x64646464u;  // byte-wise exponent for perm (1024 + byte)
constexpr uint32_t E64 = 0x54005400u, E16 = 0x4C004C00u, E4 = 0x44004400u;

template <int BITS>
struct Unpack;

template <>
struct Unpack<8> {
  static constexpr int kWords = 8;
  __device__ static uint32_t pair(const uint32_t *w, int q) {  // pair q (0..15) = codes 2q, 2q+1
    return perm(M1024, w[q >> 1], (q & 1) ? 0x04030402u : 0x04010400u);
  }
};
template <>
struct Unpack<4> {
  static constexpr int kWords = 4;
  __device__ static uint32_t pair(const uint32_t *w, int q) {
    const uint32_t x = w[q >> 2];
    switch (q & 3) {
      case 0: return andor(x, 0x00F000F0u, E64);
      case 1: return andor(x >> 8, 0x00F000F0u, E64);
      case 2: return andor(x << 6, 0x03C003C0u, E16);
      default: return andor(x >> 2, 0x03C003C0u, E16);
    }
  }
};
template <>
struct Unpack<2> {
  static constexpr int kWords = 2;
  __device__ static uint32_t pair(const uint32_t *w, int q) {
    const uint32_t x = w[q >> 3];
    switch (q & 7) {
      case 0: return andor(x, 0x03000300u, E4);
      case 1: return andor(x >> 6, 0x03000300u, E4);
      case 2: return andor(x, 0x00C000C0u, E16);
      case 3: return andor(x >> 6, 0x00C000C0u, E16);
      case 4: return andor(x, 0x00300030u, E64);
      case 5: return andor(x >> 6, 0x00300030u, E64);
      case 6: return andor(x << 8, 0x03000300u, E4);
      default: return andor(x << 6, 0x03000300u, E4);
    }
  }
};

// Offset (as fp16 pair, negated) of code pair q.
template <int BITS>
__device__ __forceinline__ uint32_t neg_off_pair(int q) {
  if (BITS == 8) return 0xE400E400u;  // -1024
  if (BITS == 4) return (q & 3) < 2 ? 0xD400D400u : 0xCC00CC00u;  // -64 / -16
  const int r = q & 7;
  return (r < 2 || r >= 6) ? 0xC400C400u : (r < 4 ? 0xCC00CC00u : 0xD400D400u);  // -4 / -16 / -64
}
// Value offset of the codes of value MFMA j (uniform per j by construction).
template <int BITS>
__device__ __forceinline__ float v_off(int j) {
  if (BITS == 8) return 1024.f;
  if (BITS == 4) return (j & 1) ? 16.f : 64.f;
  const int r = j & 3;
  return r == 1 ? 16.f : (r == 2 ? 64.f : 4.f);
}

// ---------------------------------------------------------------- parameters
struct AttnParams {
  const uint16_t *q;
  const int8_t *level;
  const int64_t *koff, *voff;
  const uint8_t *arena;
  const uint64_t *res_mask;
  const uint8_t *res_rows;
  const int32_t *pages;
  float *part;
  uint32_t *arrive;  // per (b, KV head) arrival counters; zero between calls
  float *out;
  int64_t T;
  int nblk_cap, Hkv, G, nres, nrb_cap, topk, page, nsplit;
  float sl2;  // log2(e) / sqrt(D)
};

struct State {
  f4 O[8];
  float m, l;
};

__device__ __forceinline__ float wave_max16(float x) {  // max over the 4 lanes of a head (kg)
  x = fmaxf(x, __shfl_xor(x, 16));
  x = fmaxf(x, __shfl_xor(x, 32));
  return x;
}

// Masks S to the valid tokens, updates the running max (lazily), and returns
// P (fp16 pairs) in the B-operand layout of the value MFMA.
__device__ __forceinline__ void softmax_tiles(const AttnParams &p, State &st, f4 *S, uint32_t (*Pw)[2],
                                              int tiles, uint64_t valid, int kg) {
  float bm = kNegInf;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    if (!(tiles & (1 << t))) continue;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int tok = 16 * t + 4 * kg + r;
      if ((valid >> tok) & 1ull) bm = fmaxf(bm, S[t][r]);
    }
  }
  bm = wave_max16(bm) * p.sl2;
  const bool need = bm > st.m + kRescale;
  if (__any(need)) {
    const float mn = need ? bm : st.m;
    const float alpha = need ? exp2f(st.m - mn) : 1.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j) st.O[j] *= alpha;
    st.l *= alpha;
    st.m = mn;
  }
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    if (!(tiles & (1 << t))) continue;
    float pv[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int tok = 16 * t + 4 * kg + r;
      pv[r] = ((valid >> tok) & 1ull) ? exp2f(fmaf(S[t][r], p.sl2, -st.m)) : 0.0f;
    }
    U4 u;
    u.h = half4{(_Float16)pv[0], (_Float16)pv[1], (_Float16)pv[2], (_Float16)pv[3]};
    Pw[t][0] = u.u[0];
    Pw[t][1] = u.u[1];
  }
}

__device__ __forceinline__ half4 as_h4(const uint32_t *w) {
  U4 u;
  u.u[0] = w[0];
  u.u[1] = w[1];
  return u.h;
}

// ---------------------------------------------------------------- exact blocks
__device__ void visit_exact(const AttnParams &p, State &st, const half8 *qB, const uint8_t *kp,
                            const uint8_t *vp, int tiles, uint64_t valid, int lane) {
  const int kg = lane >> 4;
  f4 S[4];
  uint32_t Pw[4][2];
  const half4 ones = half4{(_Float16)1, (_Float16)1, (_Float16)1, (_Float16)1};
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    if (!(tiles & (1 << t))) continue;
    const uint4 *kc = (const uint4 *)(kp + (size_t)(t * 64 + lane) * 64);
    U8 a[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) a[i].v = kc[i];
    f4 acc = {0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < 4; ++i) acc = mfma32(a[i].h, qB[i], acc);
    S[t] = acc;
  }
  softmax_tiles(p, st, S, Pw, tiles, valid, kg);
  f4 pb = {0, 0, 0, 0};
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    if (!(tiles & (1 << t))) continue;
    const half4 P4 = as_h4(Pw[t]);
    pb = mfma16(ones, P4, pb);
    const uint4 *vc = (const uint4 *)(vp + (size_t)(t * 64 + lane) * 64);
    U8 a[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) a[i].v = vc[i];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      U4 v;
      v.u[0] = a[j >> 1].u[2 * (j & 1)];
      v.u[1] = a[j >> 1].u[2 * (j & 1) + 1];
      st.O[j] = mfma16(v.h, P4, st.O[j]);
    }
  }
  st.l += pb[0];
}

// ---------------------------------------------------------------- scalar-code blocks
template <int BITS>
__device__ void visit_int(const AttnParams &p, State &st, const half8 *qB, const uint8_t *kp,
                          const uint8_t *vp, int tiles, uint64_t valid, int lane) {
  constexpr int NW = Unpack<BITS>::kWords;
  const int kg = lane >> 4;
  // key scale / zero for this lane's channels (lane order, 32 entries per kg)
  U8 sK[4], zK[4];
  {
    const uint4 *s4 = (const uint4 *)(kp + kg * 64);
    const uint4 *z4 = (const uint4 *)(kp + 256 + kg * 64);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      sK[i].v = s4[i];
      zK[i].v = z4[i];
    }
  }
  // key codes of the tiles read
  uint32_t kw[4][NW];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    if (!(tiles & (1 << t))) continue;
    const uint32_t *src = (const uint32_t *)(kp + kSZBytes + (size_t)(t * 64 + lane) * (4 * BITS));
    if (NW >= 4) {
#pragma unroll
      for (int q = 0; q < NW; q += 4) {
        const uint4 v = *(const uint4 *)(src + q);
        kw[t][q] = v.x;
        kw[t][q + 1] = v.y;
        kw[t][q + 2] = v.z;
        kw[t][q + 3] = v.w;
      }
    } else {
      const uint2 v = *(const uint2 *)src;
      kw[t][0] = v.x;
      kw[t][1] = v.y;
    }
  }
  // q * s split into two fp16 terms, q' = hi + lo: hi = fp16(q * s) and
  // lo = fp16(q * s - hi) (q * s and q * s - hi are exact in fp32), so the folded
  // scale keeps ~22 bits; then the per-block constant sum z q - sum off q'.
  half8 qh[4], ql[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    qh[i] = qB[i] * sK[i].h;
#pragma unroll
    for (int e = 0; e < 8; ++e)
      ql[i][e] = (_Float16)__builtin_fmaf((float)qB[i][e], (float)sK[i].h[e], -(float)qh[i][e]);
  }
  f4 c0 = {0, 0, 0, 0};
#pragma unroll
  for (int i = 0; i < 4; ++i) c0 = mfma32(zK[i].h, qB[i], c0);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    U8 o;
#pragma unroll
    for (int e = 0; e < 4; ++e) o.u[e] = neg_off_pair<BITS>(4 * i + e);
    c0 = mfma32(o.h, qh[i], c0);
    c0 = mfma32(o.h, ql[i], c0);
  }
  f4 S[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    if (!(tiles & (1 << t))) continue;
    f4 acc = c0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      U8 a;
#pragma unroll
      for (int e = 0; e < 4; ++e) a.u[e] = Unpack<BITS>::pair(kw[t], 4 * i + e);
      acc = mfma32(a.h, qh[i], acc);
      acc = mfma32(a.h, ql[i], acc);
    }
    S[t] = acc;
  }
  uint32_t Pw[4][2];
  softmax_tiles(p, st, S, Pw, tiles, valid, kg);
  // values
  U8 sV[4], zV[4];
  {
    const uint4 *s4 = (const uint4 *)(vp + kg * 64);
    const uint4 *z4 = (const uint4 *)(vp + 256 + kg * 64);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      sV[i].v = s4[i];
      zV[i].v = z4[i];
    }
  }
  const half4 ones = half4{(_Float16)1, (_Float16)1, (_Float16)1, (_Float16)1};
  f4 pb = {0, 0, 0, 0};
  f4 acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) acc[j] = f4{0, 0, 0, 0};
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    if (!(tiles & (1 << t))) continue;
    uint32_t vw[NW];
    const uint32_t *src = (const uint32_t *)(vp + kSZBytes + (size_t)(t * 64 + lane) * (4 * BITS));
    if (NW >= 4) {
#pragma unroll
      for (int q = 0; q < NW; q += 4) {
        const uint4 v = *(const uint4 *)(src + q);
        vw[q] = v.x;
        vw[q + 1] = v.y;
        vw[q + 2] = v.z;
        vw[q + 3] = v.w;
      }
    } else {
      const uint2 v = *(const uint2 *)src;
      vw[0] = v.x;
      vw[1] = v.y;
    }
    const half4 P4 = as_h4(Pw[t]);
    pb = mfma16(ones, P4, pb);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      U4 a;
      a.u[0] = Unpack<BITS>::pair(vw, 2 * j);
      a.u[1] = Unpack<BITS>::pair(vw, 2 * j + 1);
      acc[j] = mfma16(a.h, P4, acc[j]);
    }
  }
  // epilogue: O[d][h] += s_d * (acc - off * sum p) + z_d * sum p, d = 16j + 4kg + r
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const float off = v_off<BITS>(j);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int n = 4 * j + r;
      const float s = (float)sV[n >> 3].h[n & 7];
      const float z = (float)zV[n >> 3].h[n & 7];
      const float x = fmaf(-off, pb[r], acc[j][r]);
      st.O[j][r] = fmaf(s, x, fmaf(z, pb[r], st.O[j][r]));
    }
  }
  st.l += pb[0];
}

// ---------------------------------------------------------------- centroid blocks
__device__ void visit_centroid(const AttnParams &p, State &st, const half8 *qB, const uint8_t *kp,
                               const uint8_t *vp, uint64_t valid, int lane) {
  const int kg = lane >> 4, m16 = lane & 15;
  // logits of the 4 key centroids: rows 4kg + r of A hold centroid r
  f4 sc = {0, 0, 0, 0};
  {
    const uint16_t *cen = (const uint16_t *)kp + (m16 & 3) * D + 8 * kg;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      U8 a;
      a.v = *(const uint4 *)(cen + 32 * i);
      sc = mfma32(a.h, qB[i], sc);
    }
  }
  // joint (key id, value id) counts over the valid tokens
  const uint32_t *kid = (const uint32_t *)(kp + KC * D * 2);
  const uint32_t *vid = (const uint32_t *)(vp + KC * D * 2);
  const int tk = lane;
  const uint32_t ki = (kid[tk >> 4] >> (2 * (tk & 15))) & 3u;
  const uint32_t vi = (vid[tk >> 4] >> (2 * (tk & 15))) & 3u;
  const bool on = (valid >> tk) & 1ull;
  float cnt[4][4];
  float used[4];
#pragma unroll
  for (int a = 0; a < 4; ++a) {
    float tot = 0.f;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      cnt[a][v] = (float)__popcll(__ballot(on && ki == (uint32_t)a && vi == (uint32_t)v));
      tot += cnt[a][v];
    }
    used[a] = tot;
  }
  float bm = kNegInf;
#pragma unroll
  for (int a = 0; a < 4; ++a)
    if (used[a] > 0.f) bm = fmaxf(bm, sc[a]);
  bm *= p.sl2;
  const bool need = bm > st.m + kRescale;
  if (__any(need)) {
    const float mn = need ? bm : st.m;
    const float alpha = need ? exp2f(st.m - mn) : 1.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j) st.O[j] *= alpha;
    st.l *= alpha;
    st.m = mn;
  }
  float pk[4];
#pragma unroll
  for (int a = 0; a < 4; ++a) pk[a] = used[a] > 0.f ? exp2f(fmaf(sc[a], p.sl2, -st.m)) : 0.f;
  _Float16 wh[4];
  float lsum = 0.f;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    float w = 0.f;
#pragma unroll
    for (int a = 0; a < 4; ++a) w = fmaf(cnt[a][v], pk[a], w);
    wh[v] = (_Float16)w;
    lsum += (float)wh[v];
  }
  // O[d][h] += sum_v W[v][h] * vc[v][d]: rows k = 4kg + r, only kg == 0 carries data
  const half4 zero4 = half4{(_Float16)0, (_Float16)0, (_Float16)0, (_Float16)0};
  const half4 B = kg == 0 ? half4{wh[0], wh[1], wh[2], wh[3]} : zero4;
  U8 vc[4];
  {
    const uint4 *src = (const uint4 *)((const uint16_t *)vp + m16 * 8 * KC);
#pragma unroll
    for (int i = 0; i < 4; ++i) vc[i].v = kg == 0 ? src[i] : make_uint4(0, 0, 0, 0);
  }
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    U4 a;
    a.u[0] = vc[j >> 1].u[2 * (j & 1)];
    a.u[1] = vc[j >> 1].u[2 * (j & 1) + 1];
    st.O[j] = mfma16(a.h, B, st.O[j]);
  }
  st.l += lsum;
}

__device__ __forceinline__ uint32_t visit_cost(int level) {  // 16-byte units of K + V
  return (uint32_t)(2 * block_bytes(level) / 16);
}

__device__ void do_visit(const AttnParams &p, State &st, const half8 *qB, int lv, const uint8_t *kp,
                         const uint8_t *vp, int tiles, uint64_t valid, int lane) {
  switch (lv) {
    case GKV_EXACT: visit_exact(p, st, qB, kp, vp, tiles, valid, lane); break;
    case GKV_INT8: visit_int<8>(p, st, qB, kp, vp, tiles, valid, lane); break;
    case GKV_INT4: visit_int<4>(p, st, qB, kp, vp, tiles, valid, lane); break;
    case GKV_INT2: visit_int<2>(p, st, qB, kp, vp, tiles, valid, lane); break;
    default: visit_centroid(p, st, qB, kp, vp, valid, lane); break;
  }
}

__device__ __forceinline__ uint64_t tile_bits(int tiles) {
  uint64_t m = 0;
  for (int t = 0; t < 4; ++t)
    if (tiles & (1 << t)) m |= 0xFFFFull << (16 * t);
  return m;
}

__device__ __forceinline__ int tiles_of(uint64_t valid) {
  int t = 0;
  for (int i = 0; i < 4; ++i)
    if ((valid >> (16 * i)) & 0xFFFFull) t |= 1 << i;
  return t;
}

__global__ void __launch_bounds__(kThreads) attn_kernel(AttnParams p) {
  const int sidx = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int kg = lane >> 4, m16 = lane & 15;
  const int64_t u = (int64_t)b * p.Hkv + h;
  const int W = p.nsplit * kWaves, w = sidx * kWaves + wave;
  const int64_t nblk = (p.T + P - 1) / P;

  half8 qB[4];
  {
    const bool hv = m16 < p.G;
    const uint16_t *qrow = p.q + (u * p.G + (hv ? m16 : 0)) * D + 8 * kg;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      U8 t;
      t.v = hv ? *(const uint4 *)(qrow + 32 * i) : make_uint4(0, 0, 0, 0);
      qB[i] = t.h;
    }
  }
  State st;
#pragma unroll
  for (int j = 0; j < 8; ++j) st.O[j] = f4{0, 0, 0, 0};
  st.m = kNegInf;
  st.l = 0.f;

  const int8_t *lvl = p.level + u * p.nblk_cap;
  const int64_t *ko = p.koff + u * p.nblk_cap;
  const int64_t *vo = p.voff + u * p.nblk_cap;

  if (p.pages == nullptr) {
    // ---------------- dense read: blocks 0..nblk-1, then residual pseudo-blocks
    const int nrb = (p.nres + P - 1) / P;
    const int64_t nvis = nblk + nrb;
    uint64_t total = 0;
    for (int64_t base = 0; base < nvis; base += 64) {
      const int64_t v = base + lane;
      uint32_t c = 0;
      if (v < nvis) c = v < nblk ? visit_cost(lvl[v]) : visit_cost(GKV_EXACT);
      for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o);
      total += c;
    }
    // visit v belongs to wavefront floor(W * (prefix + cost/2) / total)
    int64_t v0 = nvis, v1 = nvis;
    uint64_t run = 0;
    for (int64_t base = 0; base < nvis; base += 64) {
      const int64_t v = base + lane;
      uint32_t c = 0;
      if (v < nvis) c = v < nblk ? visit_cost(lvl[v]) : visit_cost(GKV_EXACT);
      uint32_t incl = c;
      for (int o = 1; o < 64; o <<= 1) {
        const uint32_t y = __shfl_up(incl, o);
        if (lane >= o) incl += y;
      }
      const uint64_t excl = run + incl - c;
      const int64_t own = v < nvis ? (int64_t)(((uint64_t)W * (2 * excl + c)) / (2 * total)) : (int64_t)W;
      const uint64_t ge0 = __ballot(own >= w), ge1 = __ballot(own >= w + 1);
      if (ge0 && v0 == nvis) v0 = base + __ffsll((long long)ge0) - 1;
      if (ge1) {
        v1 = base + __ffsll((long long)ge1) - 1;
        break;
      }
      run += __shfl(incl, 63);
    }
    for (int64_t v = v0; v < v1; ++v) {
      int lv;
      const uint8_t *kp, *vp;
      uint64_t valid;
      if (v < nblk) {
        lv = lvl[v];
        kp = p.arena + ko[v];
        vp = p.arena + vo[v];
        const int64_t left = p.T - v * P;
        valid = left >= P ? ~0ull : ((1ull << left) - 1);
        if (p.nres) valid &= ~p.res_mask[u * p.nblk_cap + v];
      } else {
        const int64_t rb = v - nblk;
        lv = GKV_EXACT;
        kp = p.res_rows + (u * p.nrb_cap + rb) * (2 * kExactBytes);
        vp = kp + kExactBytes;
        const int64_t left = p.nres - rb * P;
        valid = left >= P ? ~0ull : ((1ull << left) - 1);
      }
      const int tiles = tiles_of(valid);
      if (tiles) do_visit(p, st, qB, lv, kp, vp, tiles, valid, lane);
    }
  } else {
    // ---------------- Compressed-Quest read: selected pages (ascending) + current page
    const int32_t *pg = p.pages + u * p.topk;
    const int64_t cur = (p.T - 1) / 16;
    int cnt = 0;  // leading entries that are valid ranked pages
    for (int base = 0; base < p.topk; base += 64) {
      const int i = base + lane;
      const bool bad = i < p.topk && (pg[i] < 0 || pg[i] >= cur);
      const uint64_t bb = __ballot(bad);
      if (bb) {
        cnt = base + __ffsll((long long)bb) - 1;
        break;
      }
      cnt = base + 64 < p.topk ? base + 64 : p.topk;
    }
    const int n = cnt + 1;
    const int e0 = (int)(((int64_t)n * w) / W), e1 = (int)(((int64_t)n * (w + 1)) / W);
    int64_t cblk = -1;
    int tiles = 0;
    for (int e = e0; e <= e1; ++e) {
      int64_t page = -1;
      if (e < e1) page = e < cnt ? pg[e] : cur;
      const int64_t blk = page >= 0 ? page >> 2 : -1;
      if (blk != cblk && cblk >= 0) {
        const int64_t left = p.T - cblk * P;
        uint64_t valid = tile_bits(tiles);
        if (left < P) valid &= (1ull << left) - 1;
        do_visit(p, st, qB, lvl[cblk], p.arena + ko[cblk], p.arena + vo[cblk], tiles_of(valid), valid, lane);
        tiles = 0;
      }
      cblk = blk;
      if (page >= 0) tiles |= 1 << (page & 3);
    }
  }

  // ---------------- merge the four wavefronts and write one partial per head
  __shared__ float so[kWaves][16][D + 1];
  __shared__ float sm[kWaves][16], sl[kWaves][16];
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int r = 0; r < 4; ++r) so[wave][m16][16 * j + 4 * kg + r] = st.O[j][r];
  if (kg == 0) {
    sm[wave][m16] = st.m;
    sl[wave][m16] = st.l;
  }
  __syncthreads();
  float *out = p.part + (u * p.nsplit + sidx) * (int64_t)p.G * (D + 2);
  for (int i = threadIdx.x; i < p.G * D; i += kThreads) {
    const int g = i >> 7, d = i & 127;
    float M = kNegInf;
#pragma unroll
    for (int q = 0; q < kWaves; ++q) M = fmaxf(M, sm[q][g]);
    float L = 0.f, o = 0.f;
    if (M > kNegInf) {
#pragma unroll
      for (int q = 0; q < kWaves; ++q) {
        const float a = exp2f(sm[q][g] - M);
        L = fmaf(sl[q][g], a, L);
        o = fmaf(so[q][g][d], a, o);
      }
    }
    out[g * (D + 2) + 2 + d] = o;
    if (d == 0) {
      out[g * (D + 2)] = M;
      out[g * (D + 2) + 1] = L;
    }
  }
  // ---------------- the last workgroup of this (b, KV head) merges all partials
  __shared__ int last;
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) last = atomicAdd(p.arrive + u, 1u) == (uint32_t)(p.nsplit - 1);
  __syncthreads();
  if (!last) return;
  __threadfence();
  const float *base = p.part + u * p.nsplit * (int64_t)p.G * (D + 2);
  const int64_t stride = (int64_t)p.G * (D + 2);
  for (int i = threadIdx.x; i < p.G * D; i += kThreads) {
    const int g = i >> 7, d = i & 127;
    const float *pg = base + g * (D + 2);
    float M = kNegInf;
    for (int s = 0; s < p.nsplit; ++s) M = fmaxf(M, __builtin_nontemporal_load(pg + s * stride));
    float L = 0.f, o = 0.f;
    for (int s = 0; s < p.nsplit; ++s) {
      const float ms = __builtin_nontemporal_load(pg + s * stride);
      if (ms == kNegInf) continue;
      const float a = exp2f(ms - M);
      L = fmaf(__builtin_nontemporal_load(pg + s * stride + 1), a, L);
      o = fmaf(__builtin_nontemporal_load(pg + s * stride + 2 + d), a, o);
    }
    p.out[(u * p.G + g) * D + d] = o / L;
  }
  if (threadIdx.x == 0) p.arrive[u] = 0;  // leave the counter ready for the next call
}

}  // namespace

// ---------------------------------------------------------------- C ABI
static int attn_nsplit(const gkv_cache *c, int32_t topk) {
  const int64_t units = (int64_t)c->B * c->Hkv;
  const int64_t nblk = (c->T + P - 1) / P;
  int64_t waves;
  if (topk > 0) {
    waves = (topk + 1 + 3) / 4;
  } else {
    const int64_t nvis = nblk + (c->nres_cap + P - 1) / P;
    waves = 2048 / units;
    if (waves > nvis) waves = nvis;
  }
  if (waves < 1) waves = 1;
  if (waves > 4096) waves = 4096;
  return (int)((waves + kWaves - 1) / kWaves);
}

static int64_t attn_part_bytes(const gkv_cache *c, int32_t topk) {
  const int G = c->Hq / c->Hkv;
  return ((int64_t)c->B * c->Hkv * attn_nsplit(c, topk) * G * (D + 2) * 4 + 255) & ~(int64_t)255;
}

int64_t gkv_attn_workspace(const gkv_cache *c, int32_t topk) {
  return attn_part_bytes(c, topk) + (int64_t)c->B * c->Hkv * 4;
}

extern "C" gkv_status gkv_graded_decode_attn(const uint16_t *q, const gkv_cache *c, const int32_t *pages,
                                             int32_t topk, float *out, void *ws, int64_t ws_bytes, void *stream) {
  gkv_status st = gkv_validate_cache(c);
  if (st) return st;
  if (!q || !out || !ws) return GKV_E_ARG;
  if (c->T <= 0) return GKV_E_SHAPE;
  if (pages) {
    if (topk <= 0) return GKV_E_ARG;
    if (c->page != 16) return GKV_E_UNSUPPORTED;
    if (c->nres) return GKV_E_UNSUPPORTED;
  } else {
    topk = 0;
  }
  const int64_t need = gkv_attn_workspace(c, topk);
  if (ws_bytes < need) return GKV_E_WORKSPACE;
  AttnParams p;
  p.q = q;
  p.level = c->level;
  p.koff = c->koff;
  p.voff = c->voff;
  p.arena = c->arena;
  p.res_mask = c->res_mask;
  p.res_rows = c->res_rows;
  p.pages = pages;
  p.part = (float *)ws;
  p.arrive = (uint32_t *)((uint8_t *)ws + attn_part_bytes(c, topk));
  p.out = out;
  p.T = c->T;
  p.nblk_cap = c->nblk_cap;
  p.Hkv = c->Hkv;
  p.G = c->Hq / c->Hkv;
  p.nres = c->nres;
  p.nrb_cap = (c->nres_cap + P - 1) / P;
  p.topk = topk;
  p.page = 16;
  p.nsplit = attn_nsplit(c, topk);
  p.sl2 = 1.4426950408889634f / sqrtf((float)D);
  hipLaunchKernelGGL(attn_kernel, dim3(p.nsplit, c->Hkv, c->B), dim3(kThreads), 0, (hipStream_t)stream, p);
  return hipGetLastError() == hipSuccess ? GKV_OK : GKV_E_HIP;
}
