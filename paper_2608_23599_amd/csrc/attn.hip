// Fused dequant + online-softmax GQA decode attention over a graded cache
// (sections 3.1, 3.5 and 3.7), and the split-context reduction.
//
// Three kernels per call.  The plan kernel (one workgroup per (b, KV head)) writes a
// 32-byte descriptor per "visit" (a block and the tokens of it that are read: all
// valid tokens of a dense read minus the residual rows, or the selected pages of a
// Compressed-Quest read) and splits the visits over the wavefronts by a cost that
// counts bytes and pipeline items.  The attention kernel runs grid (nsplit, Hkv, B)
// x 4 wavefronts; each wavefront keeps an online-softmax state for the up-to-16
// query heads of the group in MFMA accumulator layout; the four wavefronts of a
// workgroup are merged in LDS into one partial (m, l, o) per head, and a merge
// kernel combines the partials of each (b, KV head).
//
// Memory pipeline: a visit is a sequence of "items" (an int block's key
// scale/zero, a 16-token K+V tile, a centroid block).  A producer cursor walks the
// wavefront's visits and copies items ahead into a private LDS ring with
// asynchronous global -> LDS loads (global_load_lds_dwordx4: every lane moves 16 B,
// so one instruction moves 1 KB); the visit descriptors arrive the same way, one
// 1 KB chunk (32 visits) ahead.  Issued items go through a small LDS queue to the
// consumer, which waits on the load counter for its item and computes from LDS.
// The copies are issued from inline assembly so that the compiler does not add a
// full load-counter wait in front of every LDS read; the waits are explicit, and
// no other vector-memory instruction runs inside the loop (the load counter
// retires in order, so any would wait for every copy in flight).
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

// the asynchronous copies set M0 themselves (see dma16)
#pragma clang diagnostic ignored "-Winline-asm"

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
// max(a, b) for non-NaN operands as one v_max_f32: fmaxf adds NaN-quieting copies of
// its operands.
__device__ __forceinline__ float vmax(float a, float b) {
  float r;
  asm("v_max_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
__device__ __forceinline__ uint32_t perm(uint32_t hi, uint32_t lo, uint32_t sel) {
  return __builtin_amdgcn_perm(hi, lo, sel);
}

// ---------------------------------------------------------------- code unpacking
// fp16 magic exponents: code bits at mantissa [p, p+b) of exponent e give 2^(10-p) + c.
constexpr uint32_t M1024 = 0x64646464u;  // byte-wise exponent for perm (1024 + byte)
constexpr uint32_t E64 = 0x54005400u, E16 = 0x4C004C00u, E4 = 0x44004400u;

// The fp16 exponent words sit in registers (see Mag) so that each pair is one
// v_and_or_b32: that instruction cannot take two literal constants.
struct Mag {
  uint32_t e64, e16, e4;
};

template <int BITS>
struct Unpack;

template <>
struct Unpack<8> {
  static constexpr int kWords = 8;
  __device__ static uint32_t pair(const uint32_t *w, int q, const Mag &) {  // codes 2q, 2q+1
    return perm(M1024, w[q >> 1], (q & 1) ? 0x04030402u : 0x04010400u);
  }
};
template <>
struct Unpack<4> {
  static constexpr int kWords = 4;
  __device__ static uint32_t pair(const uint32_t *w, int q, const Mag &mg) {
    const uint32_t x = w[q >> 2];
    switch (q & 3) {
      case 0: return andor(x, 0x00F000F0u, mg.e64);
      case 1: return andor(x >> 8, 0x00F000F0u, mg.e64);
      case 2: return andor(x << 6, 0x03C003C0u, mg.e16);
      default: return andor(x >> 2, 0x03C003C0u, mg.e16);
    }
  }
};
template <>
struct Unpack<2> {
  static constexpr int kWords = 2;
  __device__ static uint32_t pair(const uint32_t *w, int q, const Mag &mg) {
    const uint32_t x = w[q >> 3];
    switch (q & 7) {
      case 0: return andor(x, 0x03000300u, mg.e4);
      case 1: return andor(x >> 6, 0x03000300u, mg.e4);
      case 2: return andor(x, 0x00C000C0u, mg.e16);
      case 3: return andor(x >> 6, 0x00C000C0u, mg.e16);
      case 4: return andor(x, 0x00300030u, mg.e64);
      case 5: return andor(x >> 6, 0x00300030u, mg.e64);
      case 6: return andor(x << 8, 0x03000300u, mg.e4);
      default: return andor(x << 6, 0x03000300u, mg.e4);
    }
  }
};

// A register holding a constant that the compiler must not hoist out of the item
// loop (hoisted constants of every level's path would stay live together).
__device__ __forceinline__ uint32_t opaque(uint32_t c) {
  uint32_t r;
  asm volatile("v_mov_b32 %0, %1" : "=v"(r) : "s"(c));
  return r;
}

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
  uint8_t *visits;  // visit descriptors (plan kernel scratch), vcap per (b, KV head)
  uint8_t *plan;    // item descriptors, icap per (b, KV head)
  int32_t *split;   // first item of each wavefront, W + 1 per (b, KV head)
  float *part;
  int64_t T;
  int nblk_cap, Hkv, G, nres, nrb_cap, topk, nsplit;
  int64_t vcap, icap;
  float sl2;  // log2(e) / sqrt(D)
};

constexpr int kRing = 16384;    // staging ring per wavefront (bytes, a power of two)
constexpr int kDescBytes = 2048;  // item-descriptor ring: two 1 KB chunks
constexpr int kWaveLds = kRing + kDescBytes;  // LDS per wavefront
constexpr int kMaxWaves = 1024;   // wavefronts per (b, KV head)


// ---------------------------------------------------------------- async copies
// lds_wave_base is wave-uniform (it goes to M0; lane l writes 16 bytes at +16 l); the
// readfirstlane folds away when the compiler already holds it in a scalar register.
__device__ __forceinline__ void dma16(const void *g, uint32_t lds_wave_base) {
  const uint32_t m0v = __builtin_amdgcn_readfirstlane(lds_wave_base);
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(m0v) : "memory", "m0");
}
template <int N>
__device__ __forceinline__ void vm_wait() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
// Wait until at most n of this wavefront's loads are outstanding (rounded down to
// an immediate; waiting for more than needed is always safe).
__device__ __forceinline__ void wait_loads(uint32_t n) {
  if (n >= 24) vm_wait<24>();
  else if (n >= 16) vm_wait<16>();
  else if (n >= 12) vm_wait<12>();
  else if (n >= 8) vm_wait<8>();
  else if (n >= 6) vm_wait<6>();
  else if (n >= 4) vm_wait<4>();
  else if (n >= 3) vm_wait<3>();
  else if (n >= 2) vm_wait<2>();
  else if (n >= 1) vm_wait<1>();
  else vm_wait<0>();
}

// ---------------------------------------------------------------- wave-uniform values
// The walkers' state is the same in every lane; readfirstlane keeps it in scalar
// registers (the compiler cannot prove uniformity of values loaded from memory).
__device__ __forceinline__ int32_t uni(int32_t x) { return __builtin_amdgcn_readfirstlane(x); }
__device__ __forceinline__ int64_t uni64(int64_t x) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)x >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// ---------------------------------------------------------------- item sequence
// An item is one unit of the pipeline: a contiguous span of the ring filled by up
// to four copy segments, and one step of the consumer.
//   exact tile:   [K tile 4 KB][V tile 4 KB]
//   int group:    [K scale/zero if first][K codes of n tiles][V codes of n tiles]
//                 [V scale/zero if last]   (n consecutive read tiles of one block)
//   centroid:     [K record][V record]
// The plan kernel expands every visit into its items and writes one 32-byte
// descriptor per item; the attention kernel only follows the list.
enum ItemKind { kExactTile = 0, kIntGroup = 1, kCentroid = 2 };

// Item descriptor.  meta: kind (2 bits) | level (5) | first (1) | last (1) | tile
// mask (4) | tile count (3) | exact tile's valid-token bits (16).  geo: size in
// 16-byte units (10 bits) | load instructions (6) | 16-byte units per code segment (10).
struct ItemDesc {
  uint64_t kp, vp;  // K and V record addresses
  uint64_t valid;   // tokens of the block that are read
  uint32_t meta, geo;
};
static_assert(sizeof(ItemDesc) == 32, "descriptor size");
constexpr int kDescChunk = 1024 / sizeof(ItemDesc);  // descriptors per copy (one 1 KB copy)
constexpr uint32_t kMaxAhead = kDescChunk / 2;          // producer lead over the consumer, in items

struct Item {  // the consumer's view of an item
  uint32_t lin, end;  // linear ring positions of the item and after it
  uint32_t meta;
  __device__ int kind() const { return meta & 3u; }
  __device__ int lv() const { return (meta >> 2) & 31u; }
  __device__ bool first() const { return (meta >> 7) & 1u; }
  __device__ bool last() const { return (meta >> 8) & 1u; }
  __device__ uint32_t tiles() const { return (meta >> 9) & 15u; }
  __device__ int ntiles() const { return (meta >> 13) & 7u; }
  __device__ uint32_t tvalid() const { return meta >> 16; }
};

__device__ __forceinline__ uint32_t geo_size(uint32_t g) { return (g & 1023u) * 16u; }
__device__ __forceinline__ uint32_t geo_ninstr(uint32_t g) { return (g >> 10) & 63u; }
__device__ __forceinline__ uint32_t geo_units(uint32_t g) { return g >> 16; }

// Consecutive read tiles per int item: about 4 KB of codes (K + V).
__device__ __forceinline__ int group_tiles(int lv) { return lv == 2 ? 4 : (lv == 4 ? 2 : 1); }

// Copy `units` 16-byte units from `src` to LDS address `dst` (1 KB per instruction;
// only a last partial instruction is lane-predicated).
__device__ __forceinline__ void copy_segment(const uint8_t *src, uint32_t units, uint32_t dst, int lane) {
  const uint8_t *s = src + 16 * lane;
  const uint32_t full = units >> 6;
#pragma unroll 1
  for (uint32_t i = 0; i < full; ++i) dma16(s + 1024 * i, dst + 1024 * i);
  if (units & 63u) {
    if ((uint32_t)lane < (units & 63u)) dma16(s + 1024 * full, dst + 1024 * full);
  }
}

// ---------------------------------------------------------------- pipeline
// One wavefront's pipeline over its item list.  The producer copies items ahead
// into the LDS ring; the consumer pops them in order.  Both read the item
// descriptors from a two-slot LDS ring of 32-descriptor chunks, and both derive
// the same sequence of ring positions and load counts from the descriptors, so
// nothing else passes between them.  The producer copies chunk c + 1 just before
// item 32c + 16 and stays at most kMaxAhead items ahead of the consumer, so the
// slot it overwrites (chunk c - 1) is no longer read.
struct Pipe {
  const uint8_t *ring;   // staging ring (LDS)
  const uint8_t *dring;  // descriptor ring (LDS, 2 x 1 KB)
  const uint8_t *dsrc;   // this wavefront's descriptors (global)
  uint32_t ring_base, dlds;  // LDS addresses of the two rings (wave-uniform)
  uint32_t nitems;
  uint32_t issued;  // load instructions issued
  // producer
  uint32_t pk, plin, pchunk;  // next item, its ring position, load count through the last chunk copy
  bool pend;                  // descriptor of item pk already read
  uint64_t pkp, pvp;
  uint32_t pmeta, pgeo;
  // consumer
  uint32_t ck, clin, ccnt, hold;
  int lane;

  __device__ __forceinline__ void fetch_chunk(uint32_t c) {
    dma16(dsrc + (size_t)c * 1024 + 16 * lane, dlds + (c & 1) * 1024);
    pchunk = ++issued;
  }
  __device__ __forceinline__ const uint8_t *desc(uint32_t k) const {
    return dring + ((k / kDescChunk) & 1) * 1024 + (k % kDescChunk) * sizeof(ItemDesc);
  }
  __device__ __forceinline__ bool chunk_copy_before(uint32_t k) const {  // a chunk copy precedes item k
    return k % kDescChunk == kDescChunk / 2 && (k / kDescChunk + 1) * kDescChunk < nitems;
  }
  __device__ __forceinline__ static uint32_t place(uint32_t lin, uint32_t size) {  // no wrap inside an item
    const uint32_t off = lin & (kRing - 1);
    return off + size > kRing ? lin + (kRing - off) : lin;
  }

  __device__ __forceinline__ void pump() {
    while (pk < nitems && pk - ck < kMaxAhead) {
      if (!pend) {
        if (pk % kDescChunk == 0) wait_loads(issued - pchunk);  // chunk pk / 32 has landed
        const uint8_t *e = desc(pk);
        const uint4 d0 = *(const uint4 *)e, d1 = *(const uint4 *)(e + 16);
        pkp = (uint64_t)uni64((int64_t)(((uint64_t)d0.y << 32) | d0.x));
        pvp = (uint64_t)uni64((int64_t)(((uint64_t)d0.w << 32) | d0.z));
        pmeta = uni((int32_t)d1.z);
        pgeo = uni((int32_t)d1.w);
        pend = true;
      }
      const uint32_t size = geo_size(pgeo), lin = place(plin, size);
      if (lin + size - hold > (uint32_t)kRing) break;  // ring full
      if (chunk_copy_before(pk)) fetch_chunk(pk / kDescChunk + 1);
      // the copy segments of the item
      const uint8_t *kp = (const uint8_t *)(uintptr_t)pkp, *vp = (const uint8_t *)(uintptr_t)pvp;
      const int kind = pmeta & 3u, lv = (pmeta >> 2) & 31u;
      const uint32_t t0 = __builtin_ctz((pmeta >> 9) & 15u), un = geo_units(pgeo);
      const uint32_t koff = kind == kIntGroup ? kSZBytes + t0 * 256 * lv : (kind == kExactTile ? t0 * 4096 : 0);
      uint32_t dst = ring_base + (lin & (kRing - 1));
      if (kind == kIntGroup && ((pmeta >> 7) & 1u)) {
        copy_segment(kp, kSZBytes / 16, dst, lane);
        dst += kSZBytes;
      }
      copy_segment(kp + koff, un, dst, lane);
      dst += 16 * un;
      copy_segment(vp + koff, un, dst, lane);
      dst += 16 * un;
      if (kind == kIntGroup && ((pmeta >> 8) & 1u)) copy_segment(vp, kSZBytes / 16, dst, lane);
      issued += geo_ninstr(pgeo);
      plin = lin + size;
      ++pk;
      pend = false;
    }
  }
  // Pop the next item (false when the list is exhausted), wait for its copies.
  __device__ __forceinline__ bool pop(Item &it, uint64_t &valid, const uint8_t *&ip) {
    pump();
    if (ck == nitems) return false;
    const uint8_t *e = desc(ck);
    const uint4 d1 = *(const uint4 *)(e + 16);
    valid = (uint64_t)uni64((int64_t)(((uint64_t)d1.y << 32) | d1.x));
    it.meta = uni((int32_t)d1.z);
    const uint32_t geo = uni((int32_t)d1.w), size = geo_size(geo);
    it.lin = place(clin, size);
    it.end = it.lin + size;
    clin = it.end;
    if (chunk_copy_before(ck)) ++ccnt;
    ccnt += geo_ninstr(geo);
    ++ck;
    wait_loads(issued - ccnt);
    ip = ring + (it.lin & (kRing - 1));
    return true;
  }
  __device__ __forceinline__ void release(const Item &it) { hold = it.end; }
};

// ---------------------------------------------------------------- per-wave state
struct State {
  f4 O[8];
  float m, l;
};

// Maximum over the 4 lanes of a head (lanes m16 + 16 kg): the row-swap permutes
// pair lane l with l ^ 32 and l ^ 16.
__device__ __forceinline__ float wave_max16(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = vmax(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return vmax(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

__device__ __forceinline__ half4 as_h4(uint32_t a, uint32_t b) {
  U4 u;
  u.u[0] = a;
  u.u[1] = b;
  return u.h;
}

// Lazy online-softmax rescale: when the block maximum exceeds the running maximum
// by more than kRescale, move the maximum and rescale the accumulators.
__device__ __forceinline__ float rescale_factor(State &st, float bm) {
  const bool need = bm > st.m + kRescale;
  float alpha = 1.0f;
  if (__any(need)) {
    const float mn = need ? bm : st.m;
    alpha = need ? __builtin_amdgcn_exp2f(st.m - mn) : 1.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j) st.O[j] *= alpha;
    st.l *= alpha;
    st.m = mn;
  }
  return alpha;
}

// Probabilities of one tile (this lane's 4 token rows of its head) against the
// running maximum.  Only when some logit lies more than kRescale above it (always on
// the first tile, with m = -inf) does the wavefront take the tile maximum over the
// head's lanes and rescale.  Returns true when it rescaled (alpha holds the factor).
__device__ __forceinline__ bool tile_softmax(const AttnParams &p, State &st, f4 S, bool full, uint32_t mine,
                                             half4 &P4, float &alpha) {
  float x[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    x[r] = fmaf(S[r], p.sl2, -st.m);
    if (!full && !(mine & (1u << r))) x[r] = kNegInf;
  }
  const bool big = vmax(vmax(x[0], x[1]), vmax(x[2], x[3])) > kRescale;
  const bool resc = __any(big);
  alpha = 1.0f;
  if (resc) {
    float bm = kNegInf;
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (full || (mine & (1u << r))) bm = vmax(bm, S[r]);
    alpha = rescale_factor(st, wave_max16(bm) * p.sl2);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      x[r] = fmaf(S[r], p.sl2, -st.m);
      if (!full && !(mine & (1u << r))) x[r] = kNegInf;
    }
  }
  P4 = half4{(_Float16)__builtin_amdgcn_exp2f(x[0]), (_Float16)__builtin_amdgcn_exp2f(x[1]),
             (_Float16)__builtin_amdgcn_exp2f(x[2]), (_Float16)__builtin_amdgcn_exp2f(x[3])};
  return resc;
}

__device__ __forceinline__ uint4 lds16(const uint8_t *a) { return *(const uint4 *)a; }

// The group's queries live in LDS, one 272-byte row per head (padded against bank
// conflicts); lane (head m, kg) reads its B-operand chunk of MFMA i.
constexpr int kQRow = 272;
// With PACK (group of at most 8 heads) MFMA columns 8..15 repeat heads 0..7, so
// that an int block can carry the high and low query terms in one MFMA.
template <bool PACK>
__device__ __forceinline__ int qrow(int lane) { return PACK ? (lane & 7) : (lane & 15); }
template <bool PACK>
__device__ __forceinline__ half8 qchunk(const uint8_t *qs, int lane, int i) {
  U8 t;
  t.v = lds16(qs + qrow<PACK>(lane) * kQRow + (32 * i + 8 * (lane >> 4)) * 2);
  return t.h;
}

// x[lane] + x[lane ^ 8] within each 16-lane row (DPP row rotate by 8).
__device__ __forceinline__ f4 add_row_half(f4 x) {
  f4 r;
#pragma unroll
  for (int k = 0; k < 4; ++k)
    r[k] = x[k] + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x[k]), 0x128, 0xF, 0xF, false));
  return r;
}

constexpr half4 kOnes = half4{(_Float16)1, (_Float16)1, (_Float16)1, (_Float16)1};

// ---------------------------------------------------------------- items
// Exact block tile: 16 tokens of fp16 K and V.
template <bool PACK>
__device__ __forceinline__ void exact_tile(const AttnParams &p, State &st, const uint8_t *qs, const uint8_t *ip,
                                           uint32_t tvalid, int lane) {
  const int kg = lane >> 4;
  U8 a[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) a[i].v = lds16(ip + lane * 64 + 16 * i);
  f4 S = {0, 0, 0, 0};
#pragma unroll
  for (int i = 0; i < 4; ++i) S = mfma32(a[i].h, qchunk<PACK>(qs, lane, i), S);
  const bool full = tvalid == 0xFFFFu;
  const uint32_t mine = (tvalid >> (4 * kg)) & 0xFu;
  half4 P4;
  float alpha;
  tile_softmax(p, st, S, full, mine, P4, alpha);
  const f4 pb = mfma16(kOnes, P4, f4{0, 0, 0, 0});
#pragma unroll
  for (int i = 0; i < 4; ++i) a[i].v = lds16(ip + 4096 + lane * 64 + 16 * i);
#pragma unroll
  for (int j = 0; j < 8; ++j)
    st.O[j] = mfma16(as_h4(a[j >> 1].u[2 * (j & 1)], a[j >> 1].u[2 * (j & 1) + 1]), P4, st.O[j]);
  st.l += pb[0];
}

// State of the scalar-code block being read.
struct IntBlock {
  half8 qh[4], ql[4];  // q * s as two fp16 terms
  f4 c0;               // per-block logit constant
  f4 acc[8], pb;       // block-local P.V on codes and sum of P
};

// PACK: lanes of columns 0..7 keep the high term of q * s of their head in qh,
// lanes of columns 8..15 the low term (ql is unused); one MFMA chain then holds both.
template <int BITS, bool PACK>
__device__ __forceinline__ void int_header(IntBlock &ib, const uint8_t *qs, const uint8_t *ip, int lane) {
  const int kg = lane >> 4;
  half8 qB[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) qB[i] = qchunk<PACK>(qs, lane, i);
  U8 sK[4], zK[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    sK[i].v = lds16(ip + kg * 64 + 16 * i);
    zK[i].v = lds16(ip + 256 + kg * 64 + 16 * i);
  }
  // q * s as two fp16 terms hi + lo (q * s and q * s - hi are exact in fp32)
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    ib.qh[i] = qB[i] * sK[i].h;
#pragma unroll
    for (int e = 0; e < 8; ++e)
      ib.ql[i][e] = (_Float16)__builtin_fmaf((float)qB[i][e], (float)sK[i].h[e], -(float)ib.qh[i][e]);
  }
  f4 c0 = {0, 0, 0, 0};
  if (PACK) {
    const bool lo = (lane & 8) != 0;
    const half8 zero8 = half8{0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ib.qh[i] = lo ? ib.ql[i] : ib.qh[i];
      c0 = mfma32(zK[i].h, lo ? zero8 : qB[i], c0);  // the zero-point term once per head
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      U8 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) o.u[e] = opaque(neg_off_pair<BITS>(4 * i + e));
      c0 = mfma32(o.h, ib.qh[i], c0);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) c0 = mfma32(zK[i].h, qB[i], c0);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      U8 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) o.u[e] = opaque(neg_off_pair<BITS>(4 * i + e));
      c0 = mfma32(o.h, ib.qh[i], c0);
      c0 = mfma32(o.h, ib.ql[i], c0);
    }
  }
  ib.c0 = c0;
#pragma unroll
  for (int j = 0; j < 8; ++j) ib.acc[j] = f4{0, 0, 0, 0};
  ib.pb = f4{0, 0, 0, 0};
}

// One 16-token tile of an int block: key codes at kt, value codes at vt (LDS).
template <int BITS, bool PACK>
__device__ __forceinline__ void int_tile(const AttnParams &p, State &st, IntBlock &ib, const uint8_t *kt,
                                         const uint8_t *vt, uint32_t tvalid, int lane) {
  constexpr int NW = Unpack<BITS>::kWords;
  const int kg = lane >> 4;
  const uint8_t *kc = kt + lane * (4 * BITS);
  const uint8_t *vc = vt + lane * (4 * BITS);
  Mag mg;
  if (BITS != 8) {
    mg.e64 = opaque(E64);
    mg.e16 = opaque(E16);
    mg.e4 = opaque(E4);
  }
  uint32_t kw[NW];
  if (NW >= 4) {
#pragma unroll
    for (int q = 0; q < NW; q += 4) {
      const uint4 a = lds16(kc + 4 * q);
      kw[q] = a.x; kw[q + 1] = a.y; kw[q + 2] = a.z; kw[q + 3] = a.w;
    }
  } else {
    const uint2 a = *(const uint2 *)kc;
    kw[0] = a.x; kw[1] = a.y;
  }
  uint32_t vw[NW];  // value codes, read now so that the softmax hides the latency
  if (NW >= 4) {
#pragma unroll
    for (int q = 0; q < NW; q += 4) {
      const uint4 a = lds16(vc + 4 * q);
      vw[q] = a.x; vw[q + 1] = a.y; vw[q + 2] = a.z; vw[q + 3] = a.w;
    }
  } else {
    const uint2 a = *(const uint2 *)vc;
    vw[0] = a.x; vw[1] = a.y;
  }
  f4 S = ib.c0;
  if (PACK) {  // one chain: high terms in columns 0..7, low terms in 8..15
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      U8 a;
#pragma unroll
      for (int e = 0; e < 4; ++e) a.u[e] = Unpack<BITS>::pair(kw, 4 * i + e, mg);
      S = mfma32(a.h, ib.qh[i], S);
    }
    S = add_row_half(S);
  } else {  // two independent chains (q*s high and low terms)
    f4 S2 = {0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      U8 a;
#pragma unroll
      for (int e = 0; e < 4; ++e) a.u[e] = Unpack<BITS>::pair(kw, 4 * i + e, mg);
      S = mfma32(a.h, ib.qh[i], S);
      S2 = mfma32(a.h, ib.ql[i], S2);
    }
    S += S2;
  }
  const bool full = tvalid == 0xFFFFu;
  const uint32_t mine = (tvalid >> (4 * kg)) & 0xFu;
  half4 P4;
  float alpha;
  if (tile_softmax(p, st, S, full, mine, P4, alpha)) {
#pragma unroll
    for (int j = 0; j < 8; ++j) ib.acc[j] *= alpha;
    ib.pb *= alpha;
  }
  ib.pb = mfma16(kOnes, P4, ib.pb);
#pragma unroll
  for (int j = 0; j < 8; ++j)
    ib.acc[j] = mfma16(as_h4(Unpack<BITS>::pair(vw, 2 * j, mg), Unpack<BITS>::pair(vw, 2 * j + 1, mg)), P4, ib.acc[j]);
}

// End of an int block: O[d][h] += s_d * (acc - off * sum p) + z_d * sum p,
// d = 16j + 4kg + r, with the value scale/zero at vsz (LDS).
template <int BITS>
__device__ __forceinline__ void int_epilogue(State &st, IntBlock &ib, const uint8_t *vsz, int lane) {
  const uint8_t *sz = vsz + (lane >> 4) * 64;
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {  // two halves keep fewer scale/zero registers live
    U8 sV[2], zV[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      sV[i].v = lds16(sz + 32 * hh + 16 * i);
      zV[i].v = lds16(sz + 256 + 32 * hh + 16 * i);
    }
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const int j = 4 * hh + jj;
      const float off = v_off<BITS>(j);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int n = 4 * jj + r;
        const float x = fmaf(-off, ib.pb[r], ib.acc[j][r]);
        st.O[j][r] = fmaf((float)sV[n >> 3].h[n & 7], x, fmaf((float)zV[n >> 3].h[n & 7], ib.pb[r], st.O[j][r]));
      }
    }
  }
  st.l += ib.pb[0];
}

// Centroid block: one item with both records.
template <bool PACK>
__device__ __forceinline__ void centroid_item(const AttnParams &p, State &st, const uint8_t *qs, const uint8_t *ip,
                                              uint64_t valid, int lane) {
  const int kg = lane >> 4, m16 = lane & 15;
  // logits of the 4 key centroids: rows 4kg + r of A hold centroid r
  f4 sc = {0, 0, 0, 0};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    U8 a;
    a.v = lds16(ip + ((m16 & 3) * D + 8 * kg + 32 * i) * 2);
    sc = mfma32(a.h, qchunk<PACK>(qs, lane, i), sc);
  }
  const uint32_t *kid = (const uint32_t *)(ip + KC * D * 2);
  const uint32_t *vid = (const uint32_t *)(ip + kCentBytes + KC * D * 2);
  const uint32_t ki = (kid[lane >> 4] >> (2 * (lane & 15))) & 3u;
  const uint32_t vi = (vid[lane >> 4] >> (2 * (lane & 15))) & 3u;
  U8 vc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) vc[i].v = kg == 0 ? lds16(ip + kCentBytes + m16 * 64 + 16 * i) : make_uint4(0, 0, 0, 0);
  const bool on = (valid >> lane) & 1ull;
  float cnt[4][4], used[4];
#pragma unroll
  for (int a = 0; a < 4; ++a) {
    float tot = 0.f;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      cnt[a][b] = (float)__popcll(__ballot(on && ki == (uint32_t)a && vi == (uint32_t)b));
      tot += cnt[a][b];
    }
    used[a] = tot;
  }
  float bm = kNegInf;
#pragma unroll
  for (int a = 0; a < 4; ++a)
    if (used[a] > 0.f) bm = vmax(bm, sc[a]);
  rescale_factor(st, bm * p.sl2);
  float pk[4];
#pragma unroll
  for (int a = 0; a < 4; ++a) pk[a] = used[a] > 0.f ? __builtin_amdgcn_exp2f(fmaf(sc[a], p.sl2, -st.m)) : 0.f;
  _Float16 wh[4];
  float lsum = 0.f;
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    float w = 0.f;
#pragma unroll
    for (int a = 0; a < 4; ++a) w = fmaf(cnt[a][b], pk[a], w);
    wh[b] = (_Float16)w;
    lsum += (float)wh[b];
  }
  // O[d][h] += sum_v W[v][h] * vc[v][d]: rows k = 4kg + r, only kg == 0 carries data
  const half4 zero4 = half4{(_Float16)0, (_Float16)0, (_Float16)0, (_Float16)0};
  const half4 Bw = kg == 0 ? half4{wh[0], wh[1], wh[2], wh[3]} : zero4;
#pragma unroll
  for (int j = 0; j < 8; ++j)
    st.O[j] = mfma16(as_h4(vc[j >> 1].u[2 * (j & 1)], vc[j >> 1].u[2 * (j & 1) + 1]), Bw, st.O[j]);
  st.l += lsum;
}

// Runs: process items of one level until the next item has another level (left in
// `it`, already popped) or the sequence ends (returns false).
template <bool PACK>
__device__ __forceinline__ bool exact_run(const AttnParams &p, State &st, const uint8_t *qs, Pipe &pp,
                                          Item &it, uint64_t &valid, const uint8_t *&ip, int lane) {
  do {
    exact_tile<PACK>(p, st, qs, ip, it.tvalid(), lane);
    pp.release(it);
    if (!pp.pop(it, valid, ip)) return false;
  } while (it.lv() == GKV_EXACT);
  return true;
}

template <int BITS, bool PACK>
__device__ __forceinline__ bool int_run(const AttnParams &p, State &st, const uint8_t *qs, Pipe &pp,
                                        Item &it, uint64_t &valid, const uint8_t *&ip, int lane) {
  IntBlock ib;
  do {
    const uint8_t *kq = ip;
    if (it.first()) {
      int_header<BITS, PACK>(ib, qs, kq, lane);
      kq += kSZBytes;
    }
    const int n = it.ntiles();
    const uint8_t *vq = kq + n * 256 * BITS;
    uint32_t tl = it.tiles();
#pragma unroll 1
    for (int j = 0; j < n; ++j) {
      const int t = __builtin_ctz(tl);
      tl &= tl - 1;
      int_tile<BITS, PACK>(p, st, ib, kq + j * 256 * BITS, vq + j * 256 * BITS, (uint32_t)(valid >> (16 * t)) & 0xFFFFu,
                     lane);
    }
    if (it.last()) int_epilogue<BITS>(st, ib, vq + n * 256 * BITS, lane);
    pp.release(it);
    if (!pp.pop(it, valid, ip)) return false;
  } while (it.lv() == BITS);
  return true;
}

template <bool PACK>
__device__ __forceinline__ bool centroid_run(const AttnParams &p, State &st, const uint8_t *qs, Pipe &pp,
                                             Item &it, uint64_t &valid, const uint8_t *&ip,
                                             int lane) {
  do {
    centroid_item<PACK>(p, st, qs, ip, valid, lane);
    pp.release(it);
    if (!pp.pop(it, valid, ip)) return false;
  } while (it.lv() == GKV_CENTROID);
  return true;
}

template <bool PACK>
__global__ void __launch_bounds__(kThreads, 2) attn_kernel(AttnParams p) {
  extern __shared__ __align__(16) uint8_t smem[];
  const int sidx = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int kg = lane >> 4, m16 = lane & 15;
  const int64_t u = (int64_t)b * p.Hkv + h;
  const int W = p.nsplit * kWaves, w = sidx * kWaves + wave;

  // the group's queries (rows of absent heads are zero)
  uint8_t *qs = smem + kWaves * kWaveLds;
  for (int i = threadIdx.x; i < 16 * (D / 8); i += kThreads) {
    const int g = i / (D / 8), c8 = (i % (D / 8)) * 8;
    const uint4 v = g < p.G ? *(const uint4 *)(p.q + (u * p.G + g) * D + c8) : make_uint4(0, 0, 0, 0);
    *(uint4 *)(qs + g * kQRow + c8 * 2) = v;
  }
  __syncthreads();
  State st;
#pragma unroll
  for (int j = 0; j < 8; ++j) st.O[j] = f4{0, 0, 0, 0};
  st.m = kNegInf;
  st.l = 0.f;

  // this wavefront's items, from the plan
  const int32_t *sp = p.split + u * (int64_t)(W + 1);
  const uint32_t istart = (uint32_t)uni(sp[w]), iend = (uint32_t)uni(sp[w + 1]);

  // ---------------- pipelined item loop
  Pipe pp;
  pp.ring = smem + wave * kWaveLds;
  pp.dring = smem + wave * kWaveLds + kRing;
  pp.ring_base = (uint32_t)uni((int32_t)(uintptr_t)pp.ring);
  pp.dlds = (uint32_t)uni((int32_t)(uintptr_t)pp.dring);
  pp.dsrc = p.plan + (u * p.icap + istart) * (int64_t)sizeof(ItemDesc);
  pp.nitems = iend - istart;
  pp.lane = lane;
  pp.issued = 0;
  pp.pk = pp.plin = pp.pchunk = 0;
  pp.pend = false;
  pp.pkp = pp.pvp = 0;
  pp.pmeta = pp.pgeo = 0;
  pp.ck = pp.clin = pp.hold = 0;
  if (pp.nitems) pp.fetch_chunk(0);
  pp.ccnt = pp.issued;
  // Items are processed in runs of one level, each run in a loop specialised for
  // that level (the constants of one level's path are then live only in its loop).
  Item it;
  uint64_t valid;
  const uint8_t *ip;
  bool more = pp.pop(it, valid, ip);
  while (more) {
    switch (it.lv()) {
      case GKV_EXACT: more = exact_run<PACK>(p, st, qs, pp, it, valid, ip, lane); break;
      case GKV_INT8: more = int_run<8, PACK>(p, st, qs, pp, it, valid, ip, lane); break;
      case GKV_INT4: more = int_run<4, PACK>(p, st, qs, pp, it, valid, ip, lane); break;
      case GKV_INT2: more = int_run<2, PACK>(p, st, qs, pp, it, valid, ip, lane); break;
      default: more = centroid_run<PACK>(p, st, qs, pp, it, valid, ip, lane); break;
    }
  }
  vm_wait<0>();

  // ---------------- merge the four wavefronts and write one partial per head
  __syncthreads();
  float(*so)[16][D + 1] = (float(*)[16][D + 1])smem;
  float *sm = (float *)(smem + kWaves * 16 * (D + 1) * 4);
  float *sl = sm + kWaves * 16;
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int r = 0; r < 4; ++r) so[wave][m16][16 * j + 4 * kg + r] = st.O[j][r];
  if (kg == 0) {
    sm[wave * 16 + m16] = st.m;
    sl[wave * 16 + m16] = st.l;
  }
  __syncthreads();
  float *out = p.part + (u * p.nsplit + sidx) * (int64_t)p.G * (D + 2);
  for (int i = threadIdx.x; i < p.G * D; i += kThreads) {
    const int g = i >> 7, d = i & 127;
    float M = kNegInf;
#pragma unroll
    for (int q = 0; q < kWaves; ++q) M = fmaxf(M, sm[q * 16 + g]);
    float L = 0.f, o = 0.f;
    if (M > kNegInf) {
#pragma unroll
      for (int q = 0; q < kWaves; ++q) {
        const float a = __builtin_amdgcn_exp2f(sm[q * 16 + g] - M);
        L = fmaf(sl[q * 16 + g], a, L);
        o = fmaf(so[q][g][d], a, o);
      }
    }
    out[g * (D + 2) + 2 + d] = o;
    if (d == 0) {
      out[g * (D + 2)] = M;
      out[g * (D + 2) + 1] = L;
    }
  }
}

// ---------------------------------------------------------------- merge
// One workgroup per (head, (b, KV head)), one thread per channel: the partials
// (m_s, l_s, o_s) of the nsplit workgroups combine to o = sum_s a_s o_s / sum_s a_s l_s
// with a_s = 2^(m_s - max_s m_s).
__global__ void __launch_bounds__(D) merge_kernel(const float *part, float *out, int nsplit, int G) {
  __shared__ float sa[kMaxWaves / kWaves], sl[kMaxWaves / kWaves];
  __shared__ float sinv;
  const int g = blockIdx.x, d = threadIdx.x;
  const int64_t u = blockIdx.y;
  const int64_t stride = (int64_t)G * (D + 2);
  const float *base = part + u * nsplit * stride + g * (D + 2);
  for (int s2 = d; s2 < nsplit; s2 += D) {
    sa[s2] = base[s2 * stride];
    sl[s2] = base[s2 * stride + 1];
  }
  __syncthreads();
  if (d == 0) {
    float M = kNegInf;
    for (int s2 = 0; s2 < nsplit; ++s2) M = fmaxf(M, sa[s2]);
    float L = 0.f;
    for (int s2 = 0; s2 < nsplit; ++s2) {
      const float a = sa[s2] == kNegInf ? 0.f : __builtin_amdgcn_exp2f(sa[s2] - M);
      sa[s2] = a;
      L = fmaf(a, sl[s2], L);
    }
    sinv = 1.0f / L;
  }
  __syncthreads();
  float o = 0.f;
  int s2 = 0;
  for (; s2 + 8 <= nsplit; s2 += 8) {
    float v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = base[(s2 + k) * stride + 2 + d];
#pragma unroll
    for (int k = 0; k < 8; ++k) o = fmaf(sa[s2 + k], v[k], o);
  }
  for (; s2 < nsplit; ++s2) o = fmaf(sa[s2], base[s2 * stride + 2 + d], o);
  out[(u * G + g) * D + d] = o * sinv;
}

// ---------------------------------------------------------------- plan
// One workgroup per (b, KV head).  A visit is one block and the tokens of it that
// are read: all valid tokens of a dense read minus the residual rows, or the
// selected pages of a Compressed-Quest read.  The plan kernel describes the visits,
// splits them over the W wavefronts by a balance cost (visit v goes to the
// wavefront that owns the midpoint of its cost interval), and expands every visit
// into its pipeline items, written in order; each wavefront's items are the items
// of its visits.
constexpr int kPlanThreads = 1024;

struct VisitDesc {
  uint64_t kp, vp;  // addresses of the K and V records
  uint64_t valid;   // tokens of the block that are read (bit t = token t)
  int32_t level;    // storage level of both records
  uint32_t cost;    // balance cost (bits 0..23) | number of items (bits 24..31)
};
static_assert(sizeof(VisitDesc) == 32, "descriptor size");
// Balance cost of a visit: the measured time of its parts on one wavefront sharing
// its SIMD (about 8 cycles per unit).  Exact tiles are bound by the wavefront's
// share of the bandwidth (8 KB each), int tiles by the dequantisation and softmax
// work rather than by their bytes.
constexpr uint32_t kCostExactTile = 500, kCostInt8Tile = 450, kCostInt4Tile = 300, kCostInt2Tile = 210,
                   kCostCentroid = 565, kCostIntBlock = 240;

__device__ __forceinline__ uint32_t balance_cost(int lv, uint64_t va) {
  uint32_t tiles = 0;
  for (int t = 0; t < 4; ++t) tiles += ((va >> (16 * t)) & 0xFFFFull) != 0;
  if (!tiles) return 0;
  if (lv == GKV_CENTROID) return kCostCentroid;
  if (lv == GKV_EXACT) return tiles * kCostExactTile;
  const uint32_t per = lv == 8 ? kCostInt8Tile : (lv == 4 ? kCostInt4Tile : kCostInt2Tile);
  return kCostIntBlock + tiles * per;
}

__device__ __forceinline__ uint64_t token_mask(int64_t left) {  // tokens of a block below `left`
  return left >= P ? ~0ull : ((1ull << left) - 1);
}

// Inclusive scan over the workgroup; `total` receives the sum over all threads.
__device__ __forceinline__ uint64_t block_scan(uint64_t x, uint64_t *sh, uint64_t &total) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  constexpr int NW = kPlanThreads / 64;
  for (int o = 1; o < 64; o <<= 1) {
    const uint64_t y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) sh[wv] = x;
  __syncthreads();
  if (wv == 0) {
    uint64_t t = lane < NW ? sh[lane] : 0;
    for (int o = 1; o < NW; o <<= 1) {
      const uint64_t y = __shfl_up(t, o);
      if (lane >= o) t += y;
    }
    if (lane < NW) sh[NW + lane] = t;
  }
  __syncthreads();
  const uint64_t before = wv ? sh[NW + wv - 1] : 0;
  total = sh[2 * NW - 1];
  __syncthreads();
  return x + before;
}

// Number of items of a visit (as visit_items writes them).
__device__ __forceinline__ uint32_t visit_item_count(int lv, uint64_t valid) {
  uint32_t tiles = 0;
  for (int t = 0; t < 4; ++t)
    if ((valid >> (16 * t)) & 0xFFFFull) tiles |= 1u << t;
  if (!tiles) return 0;
  if (lv == GKV_CENTROID) return 1;
  if (lv == GKV_EXACT) return __builtin_popcount(tiles);
  const int tg = group_tiles(lv);
  uint32_t k = 0;
  while (tiles) {
    const uint32_t t = __builtin_ctz(tiles);
    uint32_t n = 1;
    while ((int)n < tg && ((tiles >> (t + n)) & 1u)) ++n;
    tiles &= ~(((1u << n) - 1) << t);
    ++k;
  }
  return k;
}

// Writes the items of a visit (at most 4), in order, to out[]; returns their number.
__device__ __forceinline__ int visit_items(const VisitDesc &v, ItemDesc *out) {
  uint32_t tiles = 0;
  for (int t = 0; t < 4; ++t)
    if ((v.valid >> (16 * t)) & 0xFFFFull) tiles |= 1u << t;
  if (!tiles) return 0;
  const uint32_t lv = (uint32_t)v.level;
  auto put = [&](int i, uint32_t kind, bool first, bool last, uint32_t taken, uint32_t n, uint32_t tv,
                 uint32_t size, uint32_t ninstr, uint32_t units) {
    out[i].kp = v.kp;
    out[i].vp = v.vp;
    out[i].valid = v.valid;
    out[i].meta = kind | (lv << 2) | ((uint32_t)first << 7) | ((uint32_t)last << 8) | (taken << 9) | (n << 13) |
                  (tv << 16);
    out[i].geo = (size / 16) | (ninstr << 10) | (units << 16);
  };
  if (lv == GKV_CENTROID) {
    put(0, kCentroid, true, true, tiles, 1, 0, 2 * kCentBytes, 2 * ((kCentBytes / 16 + 63) / 64), kCentBytes / 16);
    return 1;
  }
  int k = 0;
  if (lv == GKV_EXACT) {
    for (int t = 0; t < 4; ++t)
      if ((tiles >> t) & 1u)
        put(k++, kExactTile, true, true, 1u << t, 1, (uint32_t)((v.valid >> (16 * t)) & 0xFFFFull), 2 * 4096, 8, 256);
    return k;
  }
  const int tg = group_tiles((int)lv);
  uint32_t left = tiles;
  bool first = true;
  while (left) {
    const uint32_t t = __builtin_ctz(left);
    uint32_t n = 1;
    while ((int)n < tg && ((left >> (t + n)) & 1u)) ++n;
    const uint32_t taken = ((1u << n) - 1) << t;
    left &= ~taken;
    const bool last = left == 0;
    const uint32_t cu = n * 16 * lv;  // units per code segment (a multiple of 32)
    put(k++, kIntGroup, first, last, taken, n, 0, 2 * 16 * cu + (first ? kSZBytes : 0) + (last ? kSZBytes : 0),
        2 * ((cu + 63) / 64) + (first ? 1 : 0) + (last ? 1 : 0), cu);
    first = false;
  }
  return k;
}

// Visit v of a dense read: block v (v < nblk), else residual pseudo-block v - nblk.
__device__ __forceinline__ VisitDesc dense_visit(const AttnParams &p, int64_t u, int64_t nblk, int64_t v) {
  VisitDesc d;
  if (v < nblk) {
    d.level = p.level[u * p.nblk_cap + v];
    d.kp = (uint64_t)(uintptr_t)(p.arena + p.koff[u * p.nblk_cap + v]);
    d.vp = (uint64_t)(uintptr_t)(p.arena + p.voff[u * p.nblk_cap + v]);
    d.valid = token_mask(p.T - v * P);
    if (p.nres) d.valid &= ~p.res_mask[u * p.nblk_cap + v];
  } else {
    const int64_t rb = v - nblk;
    const uint8_t *kp = p.res_rows + (u * p.nrb_cap + rb) * (2 * kExactBytes);
    d.level = GKV_EXACT;
    d.kp = (uint64_t)(uintptr_t)kp;
    d.vp = (uint64_t)(uintptr_t)(kp + kExactBytes);
    d.valid = token_mask(p.nres - rb * P);
  }
  d.cost = balance_cost(d.level, d.valid) | (visit_item_count(d.level, d.valid) << 24);
  return d;
}

// Wavefront owning the midpoint of cost interval [e, e + c) of a total, in fp64
// (every operand is an integer below 2^53, and the floor of a monotone quotient
// keeps the owners non-decreasing along the visits).
__device__ __forceinline__ int midpoint_owner(int W, uint64_t e, uint32_t c, uint64_t total) {
  if (!total) return 0;
  const double o = __builtin_floor(((double)W * (double)(2 * e + c)) / (2.0 * (double)total));
  return o < (double)W ? (int)o : W - 1;
}

// Dense plan when every thread holds at most kPlanRegs visits: the visits stay in
// registers through the cost scan and the item expansion.
constexpr int kPlanRegs = 4;
__device__ __forceinline__ void plan_dense_regs(const AttnParams &p, int64_t u, int64_t nblk, int64_t nvis, int W,
                                                ItemDesc *items, int32_t *split, uint64_t *sh, uint32_t *lastc) {
  const int64_t per = (nvis + kPlanThreads - 1) / kPlanThreads;
  const int64_t v0 = threadIdx.x * per, v1 = v0 + per < nvis ? v0 + per : nvis;
  VisitDesc dv[kPlanRegs];
  uint64_t mine = 0;
  uint32_t last = 0;
#pragma unroll
  for (int j = 0; j < kPlanRegs; ++j)
    if (v0 + j < v1) {
      dv[j] = dense_visit(p, u, nblk, v0 + j);
      const uint32_t c = dv[j].cost;
      mine += ((uint64_t)(c & 0xFFFFFFu) << 24) | (c >> 24);
      last = c & 0xFFFFFFu;
    }
  lastc[threadIdx.x] = last;  // read by the next thread after the scan's barriers
  uint64_t tot;
  const uint64_t excl = block_scan(mine, sh, tot) - mine;
  const uint64_t total = tot >> 24;
  const uint32_t nitems = (uint32_t)(tot & 0xFFFFFFu);
  if (v0 >= v1) return;
  uint64_t ecost = excl >> 24;
  uint32_t eitem = (uint32_t)(excl & 0xFFFFFFu);
  int prev = -1;
  if (v0 > 0) prev = midpoint_owner(W, ecost - lastc[threadIdx.x - 1], lastc[threadIdx.x - 1], total);
#pragma unroll
  for (int j = 0; j < kPlanRegs; ++j)
    if (v0 + j < v1) {
      const uint32_t c = dv[j].cost & 0xFFFFFFu;
      const int own = midpoint_owner(W, ecost, c, total);
      for (int ww = prev + 1; ww <= own; ++ww) split[ww] = (int32_t)eitem;
      eitem += visit_items(dv[j], items + eitem);
      if (v0 + j == nvis - 1)
        for (int ww = own + 1; ww <= W; ++ww) split[ww] = (int32_t)nitems;
      prev = own;
      ecost += c;
    }
}

__global__ void __launch_bounds__(kPlanThreads) plan_kernel(AttnParams p) {
  __shared__ uint64_t sh[2 * kPlanThreads / 64];
  __shared__ uint32_t lastc[kPlanThreads];
  __shared__ int s_cnt;
  const int64_t u = blockIdx.x;
  const int W = p.nsplit * kWaves;
  VisitDesc *desc = (VisitDesc *)p.visits + u * p.vcap;
  ItemDesc *items = (ItemDesc *)p.plan + u * p.icap;
  int32_t *split = p.split + u * (int64_t)(W + 1);
  const int64_t nblk = (p.T + P - 1) / P;
  const int8_t *lvl = p.level + u * p.nblk_cap;
  const int64_t *ko = p.koff + u * p.nblk_cap, *vo = p.voff + u * p.nblk_cap;
  int64_t nvis;
  if (!p.pages) {
    // dense: blocks 0..nblk-1, then the residual rows as exact pseudo-blocks; each
    // thread describes a contiguous run of visits
    nvis = nblk + (p.nres + P - 1) / P;
    const int64_t per = (nvis + kPlanThreads - 1) / kPlanThreads;
    if (nvis > 0 && per <= kPlanRegs) {
      plan_dense_regs(p, u, nblk, nvis, W, items, split, sh, lastc);
      return;
    }
    const int64_t v0 = threadIdx.x * per, v1 = v0 + per < nvis ? v0 + per : nvis;
#pragma unroll 4
    for (int64_t v = v0; v < v1; ++v) desc[v] = dense_visit(p, u, nblk, v);
  } else {
    // Compressed-Quest: the leading valid ranked pages (ascending) and the current
    // page; consecutive pages of one block form one visit
    const int32_t *pg = p.pages + u * p.topk;
    const int64_t cur = (p.T - 1) / 16;
    if (threadIdx.x == 0) s_cnt = p.topk;
    __syncthreads();
    for (int i = threadIdx.x; i < p.topk; i += kPlanThreads)
      if (pg[i] < 0 || pg[i] >= cur) atomicMin(&s_cnt, i);
    __syncthreads();
    const int cnt = s_cnt;
    const int n = cnt + 1;
    uint64_t vbase = 0;
    for (int base = 0; base < n; base += kPlanThreads) {
      const int i = base + threadIdx.x;
      int64_t blk = -1;
      bool start = false;
      if (i < n) {
        blk = (i < cnt ? pg[i] : cur) >> 2;
        start = i == 0 || ((i - 1 < cnt ? pg[i - 1] : cur) >> 2) != blk;
      }
      uint64_t tot;
      const uint64_t incl = block_scan(start ? 1 : 0, sh, tot);
      if (start) {
        uint32_t tl = 0;
        for (int j = i; j < n; ++j) {
          const int64_t pj = j < cnt ? pg[j] : cur;
          if ((pj >> 2) != blk) break;
          tl |= 1u << (pj & 3);
        }
        VisitDesc d;
        d.level = lvl[blk];
        d.kp = (uint64_t)(uintptr_t)(p.arena + ko[blk]);
        d.vp = (uint64_t)(uintptr_t)(p.arena + vo[blk]);
        uint64_t va = 0;
        for (int t = 0; t < 4; ++t)
          if (tl & (1u << t)) va |= 0xFFFFull << (16 * t);
        d.valid = va & token_mask(p.T - blk * P);
        d.cost = balance_cost(d.level, d.valid) | (visit_item_count(d.level, d.valid) << 24);
        desc[vbase + incl - 1] = d;
      }
      vbase += tot;
    }
    nvis = (int64_t)vbase;
  }
  __syncthreads();
  if (nvis == 0) {
    for (int ww = threadIdx.x; ww <= W; ww += kPlanThreads) split[ww] = 0;
    return;
  }
  // prefix cost and item count of each thread's run of visits (packed: cost in the
  // high bits, items in the low 24), then the owner and first item of every visit
  const int64_t per = (nvis + kPlanThreads - 1) / kPlanThreads;
  const int64_t v0 = threadIdx.x * per, v1 = v0 + per < nvis ? v0 + per : nvis;
  uint64_t mine = 0;
#pragma unroll 4
  for (int64_t v = v0; v < v1; ++v) {
    const uint32_t c = desc[v].cost;
    mine += ((uint64_t)(c & 0xFFFFFFu) << 24) | (c >> 24);
  }
  uint64_t tot;
  const uint64_t excl = block_scan(mine, sh, tot) - mine;
  const uint64_t total = tot >> 24;
  const uint32_t nitems = (uint32_t)(tot & 0xFFFFFFu);
  auto owner = [&](uint64_t e, uint32_t c) -> int { return midpoint_owner(W, e, c, total); };
  if (v0 < v1) {
    uint64_t ecost = excl >> 24;
    uint32_t eitem = (uint32_t)(excl & 0xFFFFFFu);
    int prev = -1;
    if (v0 > 0) {
      const uint32_t cp = desc[v0 - 1].cost & 0xFFFFFFu;
      prev = owner(ecost - cp, cp);
    }
    for (int64_t v = v0; v < v1; ++v) {
      const VisitDesc d = desc[v];
      const uint32_t c = d.cost & 0xFFFFFFu;
      const int own = owner(ecost, c);
      for (int ww = prev + 1; ww <= own; ++ww) split[ww] = (int32_t)eitem;
      eitem += visit_items(d, items + eitem);
      if (v == nvis - 1)
        for (int ww = own + 1; ww <= W; ++ww) split[ww] = (int32_t)nitems;
      prev = own;
      ecost += c;
    }
  }
}

}  // namespace

// ---------------------------------------------------------------- C ABI
// Workgroups per (b, KV head) for a call at context length T: enough wavefronts to
// fill the chip (2048 over all (b, KV head)), at most one per visit.
static int attn_nsplit(const gkv_cache *c, int32_t topk, int64_t T) {
  const int64_t units = (int64_t)c->B * c->Hkv;
  int64_t waves;
  if (topk > 0) {
    waves = (topk + 1 + 3) / 4;
  } else {
    const int64_t nvis = (T + P - 1) / P + (c->nres_cap + P - 1) / P;
    waves = 2048 / units;
    if (waves > nvis) waves = nvis;
  }
  if (waves < 1) waves = 1;
  if (waves > kMaxWaves) waves = kMaxWaves;
  return (int)((waves + kWaves - 1) / kWaves);
}

// Workspace layout, sized by the cache capacity so that it does not move as T grows:
// partials | wavefront splits | visit descriptors | item descriptors (at most 4
// items per visit; +1 KB: the descriptor copies read whole 1 KB chunks).
struct AttnLayout {
  int64_t split, visits, plan, total, vcap, icap;
  int ncap;
};
static int64_t align256(int64_t x) { return (x + 255) & ~(int64_t)255; }
static AttnLayout attn_layout(const gkv_cache *c, int32_t topk) {
  AttnLayout L;
  const int64_t units = (int64_t)c->B * c->Hkv;
  const int G = c->Hq / c->Hkv;
  L.ncap = attn_nsplit(c, topk, (int64_t)c->nblk_cap * P);
  L.vcap = topk > 0 ? (int64_t)topk + 1 : (int64_t)c->nblk_cap + (c->nres_cap + P - 1) / P;
  L.icap = 4 * L.vcap;
  L.split = align256(units * L.ncap * G * (D + 2) * 4);
  L.visits = L.split + align256(units * ((int64_t)L.ncap * kWaves + 1) * 4);
  L.plan = L.visits + align256(units * L.vcap * (int64_t)sizeof(VisitDesc));
  L.total = L.plan + units * L.icap * (int64_t)sizeof(ItemDesc) + 1024;
  return L;
}

int64_t gkv_attn_workspace(const gkv_cache *c, int32_t topk) { return attn_layout(c, topk).total; }

// Checks the call and fills the kernel parameters (q and out may be null for the
// stages that do not use them).
static gkv_status attn_setup(const uint16_t *q, const gkv_cache *c, const int32_t *pages, int32_t topk, void *ws,
                             int64_t ws_bytes, AttnParams &p) {
  gkv_status st = gkv_validate_cache(c);
  if (st) return st;
  if (!ws) return GKV_E_ARG;
  if (c->T <= 0) return GKV_E_SHAPE;
  if (pages) {
    if (topk <= 0) return GKV_E_ARG;
    if (c->page != 16) return GKV_E_UNSUPPORTED;
    if (c->nres) return GKV_E_UNSUPPORTED;
  } else {
    topk = 0;
  }
  const AttnLayout L = attn_layout(c, topk);
  if (ws_bytes < L.total) return GKV_E_WORKSPACE;
  p.q = q;
  p.level = c->level;
  p.koff = c->koff;
  p.voff = c->voff;
  p.arena = c->arena;
  p.res_mask = c->res_mask;
  p.res_rows = c->res_rows;
  p.pages = pages;
  p.part = (float *)ws;
  p.split = (int32_t *)((uint8_t *)ws + L.split);
  p.visits = (uint8_t *)ws + L.visits;
  p.plan = (uint8_t *)ws + L.plan;
  p.vcap = L.vcap;
  p.icap = L.icap;
  p.T = c->T;
  p.nblk_cap = c->nblk_cap;
  p.Hkv = c->Hkv;
  p.G = c->Hq / c->Hkv;
  p.nres = c->nres;
  p.nrb_cap = (c->nres_cap + P - 1) / P;
  p.topk = topk;
  p.nsplit = attn_nsplit(c, topk, c->T);
  p.sl2 = 1.4426950408889634f / sqrtf((float)D);
  return GKV_OK;
}

static void launch_plan(const AttnParams &p, const gkv_cache *c, hipStream_t s) {
  hipLaunchKernelGGL(plan_kernel, dim3(c->B * c->Hkv), dim3(kPlanThreads), 0, s, p);
}
static void launch_partials(const AttnParams &p, const gkv_cache *c, hipStream_t s) {
  const size_t lds = (size_t)kWaves * kWaveLds + 16 * kQRow;  // rings also hold the merge buffers
  if (p.G <= 8)
    hipLaunchKernelGGL(attn_kernel<true>, dim3(p.nsplit, c->Hkv, c->B), dim3(kThreads), lds, s, p);
  else
    hipLaunchKernelGGL(attn_kernel<false>, dim3(p.nsplit, c->Hkv, c->B), dim3(kThreads), lds, s, p);
}
static void launch_merge(const AttnParams &p, const gkv_cache *c, float *out, hipStream_t s) {
  hipLaunchKernelGGL(merge_kernel, dim3(p.G, c->Hkv * c->B), dim3(D), 0, s, (const float *)p.part, out, p.nsplit,
                     p.G);
}

extern "C" gkv_status gkv_attn_plan(const gkv_cache *c, const int32_t *pages, int32_t topk, void *ws, int64_t ws_bytes,
                                    void *stream) {
  AttnParams p;
  const gkv_status st = attn_setup(nullptr, c, pages, topk, ws, ws_bytes, p);
  if (st) return st;
  launch_plan(p, c, (hipStream_t)stream);
  return hipGetLastError() == hipSuccess ? GKV_OK : GKV_E_HIP;
}

extern "C" gkv_status gkv_attn_partials(const uint16_t *q, const gkv_cache *c, const int32_t *pages, int32_t topk,
                                        void *ws, int64_t ws_bytes, void *stream) {
  if (!q) return GKV_E_ARG;
  AttnParams p;
  const gkv_status st = attn_setup(q, c, pages, topk, ws, ws_bytes, p);
  if (st) return st;
  launch_partials(p, c, (hipStream_t)stream);
  return hipGetLastError() == hipSuccess ? GKV_OK : GKV_E_HIP;
}

extern "C" gkv_status gkv_attn_merge(const gkv_cache *c, const int32_t *pages, int32_t topk, float *out, void *ws,
                                     int64_t ws_bytes, void *stream) {
  if (!out) return GKV_E_ARG;
  AttnParams p;
  const gkv_status st = attn_setup(nullptr, c, pages, topk, ws, ws_bytes, p);
  if (st) return st;
  launch_merge(p, c, out, (hipStream_t)stream);
  return hipGetLastError() == hipSuccess ? GKV_OK : GKV_E_HIP;
}

extern "C" gkv_status gkv_graded_decode_attn(const uint16_t *q, const gkv_cache *c, const int32_t *pages,
                                             int32_t topk, float *out, void *ws, int64_t ws_bytes, void *stream) {
  if (!q || !out) return GKV_E_ARG;
  AttnParams p;
  const gkv_status st = attn_setup(q, c, pages, topk, ws, ws_bytes, p);
  if (st) return st;
  const hipStream_t s = (hipStream_t)stream;
  launch_plan(p, c, s);
  launch_partials(p, c, s);
  launch_merge(p, c, out, s);
  return hipGetLastError() == hipSuccess ? GKV_OK : GKV_E_HIP;
}
