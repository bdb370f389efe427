// Fused dequant + online-softmax GQA decode attention over a graded cache
// (sections 3.1, 3.5 and 3.7), and the split-context reduction.
//
// Three kernels per call.  The plan kernel describes every "visit" (a block and the
// tokens of it that are read: all valid tokens of a dense read minus the residual
// rows, or the selected pages of a Compressed-Quest read), splits the visits over the
// wavefronts by a balance cost, and writes the wavefronts' work lists.  The attention
// kernel runs nsplit workgroups of 4 wavefronts per (b, KV head); each wavefront keeps
// an online-softmax state for the up-to-16 query heads of the group in MFMA
// accumulator layout; the four wavefronts of a workgroup are merged in LDS into one
// partial (m, l, o) per head, and a merge kernel combines the partials of each
// (b, KV head).
//
// Memory pipeline: the plan kernel turns every visit into compute "items" (an
// exact 16-token tile, a group of int tiles, a centroid block) and copy "units": a
// unit fills one 4 KB slot of a wavefront's LDS ring with exactly four asynchronous
// global -> LDS loads (global_load_lds_dwordx4: every lane moves 16 B, so one
// instruction moves up to 1 KB).  The producer keeps every free slot filled; since
// every unit is four instructions and the producer's lead is fixed by the slots the
// consumer holds, the wait for a unit is a constant load count at each place the
// consumer pops one.  The descriptors arrive the same way, in 512-byte chunks
// copied half a chunk ahead.  The copies are issued from inline assembly so that
// the compiler does not add a full load-counter wait in front of every LDS read;
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

#include <mutex>

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
constexpr uint32_t E1024 = 0x64006400u, E256 = 0x5C005C00u, E64 = 0x54005400u, E16 = 0x4C004C00u,
                   E4 = 0x44004400u;

// The fp16 exponent words sit in registers (see Mag) so that each pair is one
// v_and_or_b32: that instruction cannot take two literal constants.
struct Mag {
  uint32_t e1024, e256, e64, e16, e4;
};

template <int BITS>
struct Unpack;

template <>
struct Unpack<8> {
  static constexpr int kWords = 8;
  __device__ static uint32_t pair(const uint32_t *w, int q, const Mag &) {  // codes 2q, 2q+1
    return perm(M1024, w[q >> 1], (q & 1) ? 0x04030402u : 0x04010400u);
  }
  __device__ static uint32_t kpair(const uint32_t *w, int q, const Mag &mg) { return pair(w, q, mg); }
};
template <>
struct Unpack<4> {
  static constexpr int kWords = 4;
  // Keys: nibbles 1, 5 | 3, 7 at 64 + c, nibbles 0, 4 | 2, 6 at 1024 + c (one shift
  // per word; the offsets fold into the per-block constant).
  __device__ static uint32_t kpair(const uint32_t *w, int q, const Mag &mg) {
    const uint32_t x = w[q >> 2];
    switch (q & 3) {
      case 0: return andor(x, 0x00F000F0u, mg.e64);
      case 1: return andor(x >> 8, 0x00F000F0u, mg.e64);
      case 2: return andor(x, 0x000F000Fu, mg.e1024);
      default: return andor(x >> 8, 0x000F000Fu, mg.e1024);
    }
  }
  // Values: small offsets (64 and 16), which the block epilogue subtracts in fp32.
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
  // Keys: every position keeps its own offset (they are folded into the per-block
  // constant), so only the high six bits need a shift.
  __device__ static uint32_t kpair(const uint32_t *w, int q, const Mag &mg) {
    const uint32_t x = w[q >> 3];
    switch (q & 7) {
      case 0: return andor(x, 0x03000300u, mg.e4);
      case 1: return andor(x >> 6, 0x03000300u, mg.e4);
      case 2: return andor(x, 0x00C000C0u, mg.e16);
      case 3: return andor(x >> 6, 0x00C000C0u, mg.e16);
      case 4: return andor(x, 0x00300030u, mg.e64);
      case 5: return andor(x >> 6, 0x00300030u, mg.e64);
      case 6: return andor(x, 0x00030003u, mg.e1024);
      default: return andor(x, 0x000C000Cu, mg.e256);
    }
  }
  // Values: the two pairs of one MFMA share an offset.
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
// Offset (as fp16 pair, negated) of key code pair q.
template <int BITS>
__device__ __forceinline__ uint32_t neg_off_pair(int q) {
  if (BITS == 8) return 0xE400E400u;  // -1024
  if (BITS == 4) return (q & 3) < 2 ? 0xD400D400u : 0xE400E400u;  // -64 / -1024
  const int r = q & 7;
  if (r < 6) return r < 2 ? 0xC400C400u : (r < 4 ? 0xCC00CC00u : 0xD400D400u);  // -4 / -16 / -64
  return r == 6 ? 0xE400E400u : 0xDC00DC00u;  // -1024 / -256
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
constexpr int kTagWords = 12;
constexpr uint64_t kTagMagic = 0x676b76706c616e31ull;  // marks a tag as written by a dense plan

struct AttnParams {
  const uint16_t *q;
  const int8_t *level;
  const int64_t *koff, *voff;
  const uint8_t *arena;
  const uint64_t *res_mask;
  const int32_t *res_off;
  const uint8_t *res_rows;
  const int32_t *pages;
  const int64_t *seq_len;  // tokens per sequence (-1: retired), or null: every sequence has T
  uint8_t *visits;  // visit descriptors (plan kernel scratch), vcap per (b, KV head)
  uint8_t *plan;    // item descriptors, icap per (b, KV head)
  uint8_t *units;   // unit descriptors, ucap per (b, KV head)
  int32_t *split;   // first item and first unit of each wavefront, 2 (W + 1) per (b, KV head)
  float *part;
  int64_t T;
  int nblk_cap, Hkv, G, nres, nrb_cap, topk, nsplit;
  int page;  // Compressed-Quest page tokens (16, 32 or 64)
  const float *cert;  // per-block certificate numbers {kerr, verr, vmax, 0} (dense reads)
  float *bound;       // when set: the attention error certificate per query head
  int fast;  // workgroups of each (b, KV head) dispatched first (see attn_grid)
  int64_t vcap, icap, ucap;
  float sl2;  // log2(e) / sqrt(D)
  // Plan reuse (dense reads of a cache with a version stamp): the workspace's tag holds
  // the key of the state whose plan it holds; the plan kernel skips when it matches,
  // the attention kernel writes it once the plan is complete.
  int cacheable;
  uint64_t *tag;
  uint64_t key[kTagWords];
};

// Tokens of (b, KV head) u: its sequence's length, 0 for a retired sequence.
__device__ __forceinline__ int64_t unit_T(const AttnParams &p, int64_t u) {
  if (!p.seq_len) return p.T;
  const int64_t t = p.seq_len[u / p.Hkv];
  return t > 0 ? t : 0;
}

// Tokens a dense plan covers in u: its length rounded up to whole blocks.  A sequence's
// last block is always exact (a partial block is never demoted), and the attention
// kernel masks that block's tokens past the length at run time, so one plan serves
// every length inside the block (appends that open no block keep the plan).
__device__ __forceinline__ int64_t plan_T(const AttnParams &p, int64_t u) {
  return (unit_T(p, u) + P - 1) / P * P;
}

constexpr int kSlotBytes = 4096;  // one copy unit
constexpr int kSlots = 4;         // ring slots per wavefront
constexpr int kRing = kSlots * kSlotBytes;
constexpr int kChunk = 32;        // descriptors per 512-byte chunk
// per wavefront: ring | unit-descriptor chunks (2 x 512) | item-descriptor chunks
// (2 x 512) | value scale/zero of the current int block (512)
constexpr int kWaveLds = kRing + 4 * 512 + 512;
constexpr int kMaxWaves = 1024;   // wavefronts per (b, KV head)
// partial per workgroup and head: m, l, o[D], then the certificate sums c1, c2, c3
constexpr int kPart = D + 5;


// ---------------------------------------------------------------- async copies
// Every copy carries the nontemporal hint: each cache byte is read once per step, and
// on gfx950 the hint lifts a streaming read from about 6.2 to about 7.0 TB/s (the
// attention kernel's achieved rate rose by a tenth with it).
// lds_wave_base is wave-uniform (it goes to M0; lane l writes 16 bytes at +16 l); the
// readfirstlane folds away when the compiler already holds it in a scalar register.
__device__ __forceinline__ void dma16(const void *g, uint32_t lds_wave_base) {
  const uint32_t m0v = __builtin_amdgcn_readfirstlane(lds_wave_base);
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off nt" ::"v"(g), "s"(m0v) : "memory", "m0");
}
// Four 1 KB copies into one ring slot with one M0: a -> slot [0, 2K), b -> slot [2K, 4K)
// (the instruction offset moves the global and the LDS address together).
__device__ __forceinline__ void dma4(const uint8_t *a, const uint8_t *b, uint32_t slot) {
  const uint32_t m0v = __builtin_amdgcn_readfirstlane(slot);
  asm volatile(
      "s_mov_b32 m0, %2\n\t"
      "global_load_lds_dwordx4 %0, off nt\n\t"
      "global_load_lds_dwordx4 %0, off offset:1024 nt\n\t"
      "global_load_lds_dwordx4 %1, off offset:2048 nt\n\t"
      "global_load_lds_dwordx4 %1, off offset:3072 nt" ::"v"(a),
      "v"(b - 2048), "s"(m0v)
      : "memory", "m0");
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

// ---------------------------------------------------------------- items and units
// Items, in the order the consumer computes them, and the copy units they read:
//   exact tile:   unit [K tile 4 KB], unit [V tile 4 KB]
//   int group:    (first of a block: unit [K scale/zero | V scale/zero]), then for
//                 int2 unit [K codes of n tiles | V codes of n tiles], for int4 and
//                 int8 unit [K codes of n tiles], unit [V codes of n tiles]  (n
//                 consecutive read tiles of one block, at most 4 KB of codes per record)
//   centroid:     unit [K record | V record]
//   mean:         unit [K row | V row]
enum ItemKind { kExactTile = 0, kIntGroup = 1, kCentroid = 2, kMean = 3 };

// Item descriptor.  meta: kind (2 bits) | level (5) | first (1) | last (1) | tile
// mask (4) | tile count (3) | exact tile's valid-token bits (16).
struct ItemDesc {
  uint32_t meta, pad;
  uint64_t valid;  // tokens of the block that are read
};
static_assert(sizeof(ItemDesc) == 16, "descriptor size");

// Copy unit: part A (slot bytes [0, 2K)) from address a, part B ([2K, 4K)) from b.
// In each part the first load moves n0 16-byte lanes from the part's address and
// the second n1 lanes from the address + 1 KB; n1 = 0 stands for one lane that
// re-reads the part's first 16 bytes, so that every unit is four loads (an empty
// part B is one such lane at part A's address).
struct UnitDesc {
  uint64_t a;  // address (bits 0..47) | n0 (bits 48..55) | n1 (bits 56..63), part A
  uint64_t b;  // the same for part B
};
static_assert(sizeof(UnitDesc) == 16, "descriptor size");

__device__ __forceinline__ int meta_kind(uint32_t m) { return m & 3u; }
__device__ __forceinline__ int meta_lv(uint32_t m) { return (m >> 2) & 31u; }
__device__ __forceinline__ bool meta_first(uint32_t m) { return (m >> 7) & 1u; }
__device__ __forceinline__ bool meta_last(uint32_t m) { return (m >> 8) & 1u; }
__device__ __forceinline__ uint32_t meta_tiles(uint32_t m) { return (m >> 9) & 15u; }
__device__ __forceinline__ int meta_ntiles(uint32_t m) { return (m >> 13) & 7u; }
__device__ __forceinline__ uint32_t meta_tvalid(uint32_t m) { return m >> 16; }

// Consecutive read tiles per int item: up to 4 KB of codes per record (int8: 2 tiles,
// int4 and int2: a whole block).  int2 items read one unit (K codes | V codes, 2 KB
// each); int4 and int8 items read a K unit and a V unit.
__device__ __forceinline__ int group_tiles(int lv) { return lv == 8 ? 2 : 4; }

// Issues the four loads of a unit into the slot at LDS address `slot`.
__device__ __forceinline__ void issue_part(uint64_t a, uint32_t dst, int lane) {
  const uint32_t n0 = (uint32_t)(a >> 48) & 255u, n1 = (uint32_t)(a >> 56);
  const uint8_t *pa = (const uint8_t *)(uintptr_t)(a & 0xFFFFFFFFFFFFull) + 16 * lane;
  if ((uint32_t)lane < n0) dma16(pa, dst);
  const uint32_t m1 = n1 ? n1 : 1u, o1 = n1 ? 1024u : 0u;
  if ((uint32_t)lane < m1) dma16(pa + o1, dst + 1024);
}
__device__ __forceinline__ void issue_unit(uint64_t a, uint64_t b, uint32_t slot, int lane) {
  if ((a >> 48) == 0x4040u && (b >> 48) == 0x4040u) {  // both parts full: 4 x 1 KB, one M0
    dma4((const uint8_t *)(uintptr_t)(a & 0xFFFFFFFFFFFFull) + 16 * lane,
         (const uint8_t *)(uintptr_t)(b & 0xFFFFFFFFFFFFull) + 16 * lane, slot);
    return;
  }
  issue_part(a, slot, lane);
  issue_part(b, slot + 2048, lane);
}

// ---------------------------------------------------------------- pipeline
// One wavefront's pipeline over its units and items.  The producer issues unit k
// into slot k % kSlots as soon as the consumer has released unit k - kSlots; the
// consumer pops the units of each item in order.  When the consumer pops unit k
// while holding H units, every unit up to min(n, released + kSlots) has been
// issued, so at least 4 (kSlots - 1 - H) loads follow unit k's unless the list ends
// first (then it waits for all).  Descriptor chunk c + 1 is copied when the cursor
// of its list reaches 32 c + 16 and waited for when it reaches 32 (c + 1).
struct Pipe {
  const uint8_t *ring;           // ring (LDS)
  const uint8_t *uchunk, *ichunk;  // descriptor chunks (LDS, 2 x 512 B each)
  const uint8_t *usrc, *isrc;    // this wavefront's unit and item descriptors (global)
  uint32_t ring_base, ulds, ilds;  // LDS addresses (wave-uniform)
  uint32_t nunits, nitems;
  uint32_t issued;  // load instructions issued
  uint32_t pk;      // units issued
  uint32_t ufetch;  // load count through the last unit-chunk copy
  uint32_t ck, rel; // units popped, released
  uint32_t ik;      // items read
  uint32_t ifetch;  // load count through the last item-chunk copy
  uint8_t *ebuf;    // value scale/zero of the current int block (LDS, 512 B)
  int lane;
  uint32_t blk;        // block index of the current item (0xFFFF: no block record)
  int64_t tlim;        // tokens of this (b, KV head): exact tiles of a dense plan are masked there
  const float *cert;   // this (b, KV head)'s certificate rows, or null

  __device__ __forceinline__ void fetch(const uint8_t *src, uint32_t lds, uint32_t c) {
    if (lane < 32) dma16(src + (size_t)c * 512 + 16 * lane, lds + (c & 1) * 512);
  }
  // local: the lists (at most one chunk each) were written into the chunk buffers by
  // this wavefront, and nothing is fetched
  __device__ __forceinline__ void start(int ln, bool local) {
    lane = ln;
    issued = pk = ck = rel = ik = 0;
    ufetch = ifetch = 0;
    if (nunits && !local) {
      fetch(usrc, ulds, 0);
      ufetch = ++issued;
    }
    if (nitems && !local) {
      fetch(isrc, ilds, 0);
      ifetch = ++issued;
    }
    vm_wait<0>();
  }
  __device__ __forceinline__ void pump() {
    while (pk < nunits && pk < rel + kSlots) {
      const uint32_t r = pk % kChunk;
      if (r == 0 && pk) wait_loads(issued - ufetch);  // chunk pk / 32 has landed
      if (r == kChunk / 2 && (pk / kChunk + 1) * kChunk < nunits) {
        fetch(usrc, ulds, pk / kChunk + 1);
        ufetch = ++issued;
      }
      const uint4 d = *(const uint4 *)(uchunk + ((pk / kChunk) & 1) * 512 + r * sizeof(UnitDesc));
      const uint64_t a = (uint64_t)uni64((int64_t)(((uint64_t)d.y << 32) | d.x));
      const uint64_t b = (uint64_t)uni64((int64_t)(((uint64_t)d.w << 32) | d.z));
      issue_unit(a, b, ring_base + (pk % kSlots) * kSlotBytes, lane);
      issued += 4;
      ++pk;
    }
  }
  // The next item's descriptor (false when the wavefront's items are done).
  template <bool CERT>
  __device__ __forceinline__ bool next_item(uint32_t &meta, uint64_t &valid) {
    if (ik == nitems) return false;
    const uint32_t r = ik % kChunk;
    if (r == 0 && ik) wait_loads(issued - ifetch);
    if (r == kChunk / 2 && (ik / kChunk + 1) * kChunk < nitems) {
      fetch(isrc, ilds, ik / kChunk + 1);
      ifetch = ++issued;
    }
    const uint4 d = *(const uint4 *)(ichunk + ((ik / kChunk) & 1) * 512 + r * sizeof(ItemDesc));
    meta = (uint32_t)uni((int32_t)d.x);
    valid = (uint64_t)uni64((int64_t)(((uint64_t)d.w << 32) | d.z));
    blk = (uint32_t)uni((int32_t)d.y);
    ++ik;
    return true;
  }
  // Pop the next unit while holding H units; returns its slot once it has landed.
  template <int H>
  __device__ __forceinline__ const uint8_t *pop() {
    pump();
    const uint32_t k = ck++;
    if (k + kSlots - H > nunits) vm_wait<0>();
    else vm_wait<4 * (kSlots - 1 - H)>();
    return ring + (k % kSlots) * kSlotBytes;
  }
  // Releasing slots lets the next pump copy into them: every LDS read issued so far
  // (the items read their slots with ordinary loads, whose results the compiler may
  // consume after the copy is issued) must have returned first.
  __device__ __forceinline__ void release(uint32_t n) {
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    rel += n;
  }
};

// ---------------------------------------------------------------- per-wave state
struct State {
  f4 O[8];
  float m, l;
  float c1, c2, c3;  // certificate sums: sum_b p_b verr_b, sum_b p_b e^eps_b, sum_b p_b e^-eps_b
  float es;          // eps_b = es * kerr_b in log2 units: ||q|| log2(e) / sqrt(D)
};

// Adds block mass pb (this lane's head) with certificate numbers kerr, verr.
__device__ __forceinline__ void cert_add(State &st, float pb, float kerr, float verr) {
  const float x = st.es * kerr;
  st.c1 = fmaf(pb, verr, st.c1);
  st.c2 = fmaf(pb, __builtin_amdgcn_exp2f(x), st.c2);
  st.c3 = fmaf(pb, __builtin_amdgcn_exp2f(-x), st.c3);
}

// Maximum over the 4 lanes of a head (lanes m16 + 16 kg): the row-swap permutes
// pair lane l with l ^ 32 and l ^ 16.
__device__ __forceinline__ float wave_max16(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = vmax(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return vmax(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

__device__ __forceinline__ float wave_sum16(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
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
    st.c1 *= alpha;
    st.c2 *= alpha;
    st.c3 *= alpha;
    st.m = mn;
  }
  return alpha;
}

// Probabilities of one tile (this lane's 4 token rows of its head) against the
// running maximum.  Only when some logit lies more than kRescale above it (always on
// the first tile, with m = -inf) does the wavefront take the tile maximum over the
// head's lanes and rescale.  Returns true when it rescaled (alpha holds the factor).
__device__ __forceinline__ bool tile_softmax(const AttnParams &p, State &st, f4 S, uint32_t tvalid, int kg,
                                             half4 &P4, float &alpha) {
  const bool full = tvalid == 0xFFFFu;
  float x[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) x[r] = fmaf(S[r], p.sl2, -st.m);
  uint32_t mine = 15u;
  if (!full) {  // tokens that are not read (a uniform branch: most tiles are full)
    uint32_t t = tvalid;
    asm volatile("" : "+s"(t));  // keeps the mask work inside the branch
    mine = (t >> (4 * kg)) & 15u;
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (!(mine & (1u << r))) x[r] = kNegInf;
  }
  const bool big = vmax(vmax(x[0], x[1]), vmax(x[2], x[3])) > kRescale;
  const bool resc = __any(big);
  alpha = 1.0f;
  if (resc) {
    float bm = kNegInf;
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (mine & (1u << r)) bm = vmax(bm, S[r]);
    alpha = rescale_factor(st, wave_max16(bm) * p.sl2);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      x[r] = fmaf(S[r], p.sl2, -st.m);
      if (!(mine & (1u << r))) x[r] = kNegInf;
    }
  }
  P4 = half4{(_Float16)__builtin_amdgcn_exp2f(x[0]), (_Float16)__builtin_amdgcn_exp2f(x[1]),
             (_Float16)__builtin_amdgcn_exp2f(x[2]), (_Float16)__builtin_amdgcn_exp2f(x[3])};
  return resc;
}

// Probabilities of two tiles of one block at once (this lane's 4 token rows of its
// head in each), with one rescale decision for the pair: P8 holds tile A's rows in
// elements 0..3 and tile B's in 4..7.
__device__ __forceinline__ bool pair_softmax(const AttnParams &p, State &st, f4 SA, f4 SB, uint32_t tvA,
                                             uint32_t tvB, int kg, half8 &P8, float &alpha) {
  const bool full = (tvA & tvB) == 0xFFFFu;
  float x[8];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    x[r] = fmaf(SA[r], p.sl2, -st.m);
    x[4 + r] = fmaf(SB[r], p.sl2, -st.m);
  }
  uint32_t mine = 0xFFu;
  if (!full) {  // tokens that are not read (a uniform branch: most pairs are full)
    uint32_t a = tvA, b = tvB;
    asm volatile("" : "+s"(a), "+s"(b));  // keeps the mask work inside the branch
    mine = ((a >> (4 * kg)) & 15u) | (((b >> (4 * kg)) & 15u) << 4);
#pragma unroll
    for (int r = 0; r < 8; ++r)
      if (!(mine & (1u << r))) x[r] = kNegInf;
  }
  const bool big = vmax(vmax(vmax(x[0], x[1]), vmax(x[2], x[3])), vmax(vmax(x[4], x[5]), vmax(x[6], x[7]))) > kRescale;
  const bool resc = __any(big);
  alpha = 1.0f;
  if (resc) {
    float bm = kNegInf;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      if (mine & (1u << r)) bm = vmax(bm, SA[r]);
      if (mine & (1u << (4 + r))) bm = vmax(bm, SB[r]);
    }
    alpha = rescale_factor(st, wave_max16(bm) * p.sl2);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      x[r] = fmaf(SA[r], p.sl2, -st.m);
      x[4 + r] = fmaf(SB[r], p.sl2, -st.m);
    }
#pragma unroll
    for (int r = 0; r < 8; ++r)
      if (!(mine & (1u << r))) x[r] = kNegInf;
  }
#pragma unroll
  for (int r = 0; r < 8; ++r) P8[r] = (_Float16)__builtin_amdgcn_exp2f(x[r]);
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
constexpr half8 kOnes8 = half8{(_Float16)1, (_Float16)1, (_Float16)1, (_Float16)1,
                               (_Float16)1, (_Float16)1, (_Float16)1, (_Float16)1};

// ---------------------------------------------------------------- items
// Exact block tile: 16 tokens of fp16 K and V.
template <bool PACK, bool CERT>
__device__ __forceinline__ void exact_tile(const AttnParams &p, State &st, const uint8_t *qs, Pipe &pp,
                                           uint32_t tvalid, int lane) {
  const int kg = lane >> 4;
  const uint8_t *kt = pp.template pop<0>();
  U8 a[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) a[i].v = lds16(kt + lane * 64 + 16 * i);
  f4 S = {0, 0, 0, 0};
#pragma unroll
  for (int i = 0; i < 4; ++i) S = mfma32(a[i].h, qchunk<PACK>(qs, lane, i), S);
  half4 P4;
  float alpha;
  tile_softmax(p, st, S, tvalid, kg, P4, alpha);
  const f4 pb = mfma16(kOnes, P4, f4{0, 0, 0, 0});
  const uint8_t *vt = pp.template pop<1>();
#pragma unroll
  for (int i = 0; i < 4; ++i) a[i].v = lds16(vt + lane * 64 + 16 * i);
#pragma unroll
  for (int j = 0; j < 8; ++j)
    st.O[j] = mfma16(as_h4(a[j >> 1].u[2 * (j & 1)], a[j >> 1].u[2 * (j & 1) + 1]), P4, st.O[j]);
  st.l += pb[0];
  if (CERT) {  // exact rows: no logit or value error
    st.c2 += pb[0];
    st.c3 += pb[0];
  }
  pp.release(2);
}

// State of the scalar-code block being read.
struct IntBlock {
  half8 qh[4], ql[4];  // q * s as two fp16 terms
  f4 c0;               // per-block logit constant
  f4 acc[8], pb;       // block-local P.V on codes and sum of P
  f4 ps, pz;           // values grouped per token: sum of P * scale and of P * zero
  float kerr, verr;    // certificate numbers of the block
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
  // q * s as two fp16 terms hi + lo: hi = fp16(q * s), lo = fp16(q * s - hi).  The
  // fused fp16 multiply-add rounds the exact q * s - hi once, so two packed
  // instructions give both terms of two channels
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    ib.qh[i] = qB[i] * sK[i].h;
    ib.ql[i] = __builtin_elementwise_fma(qB[i], sK[i].h, -ib.qh[i]);
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

// This lane's code words of one tile (LDS).
template <int BITS>
__device__ __forceinline__ void tile_words(const uint8_t *c, uint32_t *w) {
  constexpr int NW = Unpack<BITS>::kWords;
  if (NW >= 4) {
#pragma unroll
    for (int q = 0; q < NW; q += 4) {
      const uint4 a = lds16(c + 4 * q);
      w[q] = a.x; w[q + 1] = a.y; w[q + 2] = a.z; w[q + 3] = a.w;
    }
  } else {
    const uint2 a = *(const uint2 *)c;
    w[0] = a.x; w[1] = a.y;
  }
}

// Logits of one tile of an int block from its key code words.
template <int BITS, bool PACK>
__device__ __forceinline__ f4 int_logits(const IntBlock &ib, const uint32_t *kw, const Mag &mg) {
  f4 S = ib.c0;
  if (PACK) {  // one chain: high terms in columns 0..7, low terms in 8..15
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      U8 a;
#pragma unroll
      for (int e = 0; e < 4; ++e) a.u[e] = Unpack<BITS>::kpair(kw, 4 * i + e, mg);
      S = mfma32(a.h, ib.qh[i], S);
    }
    S = add_row_half(S);
  } else {  // two independent chains (q*s high and low terms)
    f4 S2 = {0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      U8 a;
#pragma unroll
      for (int e = 0; e < 4; ++e) a.u[e] = Unpack<BITS>::kpair(kw, 4 * i + e, mg);
      S = mfma32(a.h, ib.qh[i], S);
      S2 = mfma32(a.h, ib.ql[i], S2);
    }
    S += S2;
  }
  return S;
}

// Per-token value scale and zero of this lane's 4 tokens of block tile ti (VTOK: the
// block's value header, scale[64] then zero[64] in token order, at ebuf).
__device__ __forceinline__ void tok_sz(const uint8_t *ebuf, int ti, int kg, U4 &sv, U4 &zv) {
  *(uint2 *)sv.u = *(const uint2 *)(ebuf + 2 * (16 * ti + 4 * kg));
  *(uint2 *)zv.u = *(const uint2 *)(ebuf + 128 + 2 * (16 * ti + 4 * kg));
}

// One 16-token tile of an int block: key codes at kt, value codes at vt (LDS).  With
// VTOK (values grouped per token) P is scaled by each token's value scale before the
// P.V product, and sum P * scale and sum P * zero are kept for the block epilogue.
template <int BITS, bool PACK, bool VTOK>
__device__ __forceinline__ void int_tile(const AttnParams &p, State &st, IntBlock &ib, const uint8_t *kt,
                                         const uint8_t *vt, uint32_t tvalid, const Mag &mg, int lane, int ti,
                                         const uint8_t *ebuf) {
  constexpr int NW = Unpack<BITS>::kWords;
  const int kg = lane >> 4;
  uint32_t kw[NW], vw[NW];  // value codes read now so that the softmax hides the latency
  tile_words<BITS>(kt + lane * (4 * BITS), kw);
  tile_words<BITS>(vt + lane * (4 * BITS), vw);
  const f4 S = int_logits<BITS, PACK>(ib, kw, mg);
  half4 P4;
  float alpha;
  if (tile_softmax(p, st, S, tvalid, kg, P4, alpha)) {
#pragma unroll
    for (int j = 0; j < 8; ++j) ib.acc[j] *= alpha;
    ib.pb *= alpha;
    if (VTOK) {
      ib.ps *= alpha;
      ib.pz *= alpha;
    }
  }
  ib.pb = mfma16(kOnes, P4, ib.pb);
  half4 PV = P4;
  if (VTOK) {
    U4 sv, zv;
    tok_sz(ebuf, ti, kg, sv, zv);
    PV = P4 * sv.h;  // one rounding of the exact fp16 product
    ib.ps = mfma16(kOnes, PV, ib.ps);
    ib.pz = mfma16(zv.h, P4, ib.pz);  // every row of A holds the 4 tokens' zeros
  }
#pragma unroll
  for (int j = 0; j < 8; ++j)
    ib.acc[j] = mfma16(as_h4(Unpack<BITS>::pair(vw, 2 * j, mg), Unpack<BITS>::pair(vw, 2 * j + 1, mg)), PV, ib.acc[j]);
}

// Two consecutive tiles of an int block (tile B's codes follow tile A's).  P.V runs
// as one 32-deep MFMA per channel group: the contraction index k = 8 kg + e takes
// tile A's token 4 kg + e for e < 4 and tile B's token 4 kg + e - 4 for e >= 4, in
// both operands, so each lane's operands are its own registers of the two tiles.
template <int BITS, bool PACK, bool VTOK>
__device__ __forceinline__ void int_tile2(const AttnParams &p, State &st, IntBlock &ib, const uint8_t *kt,
                                          const uint8_t *vt, uint32_t tvA, uint32_t tvB, const Mag &mg, int lane,
                                          int ta, int tb, const uint8_t *ebuf) {
  constexpr int NW = Unpack<BITS>::kWords;
  constexpr int TB = 256 * BITS;  // code bytes of one tile and tensor
  const int kg = lane >> 4;
  uint32_t kwA[NW], kwB[NW], vwA[NW], vwB[NW];
  tile_words<BITS>(kt + lane * (4 * BITS), kwA);
  tile_words<BITS>(kt + TB + lane * (4 * BITS), kwB);
  tile_words<BITS>(vt + lane * (4 * BITS), vwA);
  tile_words<BITS>(vt + TB + lane * (4 * BITS), vwB);
  const f4 SA = int_logits<BITS, PACK>(ib, kwA, mg);
  const f4 SB = int_logits<BITS, PACK>(ib, kwB, mg);
  half8 P8;
  float alpha;
  if (pair_softmax(p, st, SA, SB, tvA, tvB, kg, P8, alpha)) {
#pragma unroll
    for (int j = 0; j < 8; ++j) ib.acc[j] *= alpha;
    ib.pb *= alpha;
    if (VTOK) {
      ib.ps *= alpha;
      ib.pz *= alpha;
    }
  }
  ib.pb = mfma32(kOnes8, P8, ib.pb);
  half8 PV = P8;
  if (VTOK) {
    U4 sA, zA, sB, zB;
    tok_sz(ebuf, ta, kg, sA, zA);
    tok_sz(ebuf, tb, kg, sB, zB);
    U8 s8, z8;
    s8.u[0] = sA.u[0]; s8.u[1] = sA.u[1]; s8.u[2] = sB.u[0]; s8.u[3] = sB.u[1];
    z8.u[0] = zA.u[0]; z8.u[1] = zA.u[1]; z8.u[2] = zB.u[0]; z8.u[3] = zB.u[1];
    PV = P8 * s8.h;
    ib.ps = mfma32(kOnes8, PV, ib.ps);
    ib.pz = mfma32(z8.h, P8, ib.pz);
  }
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    U8 a;
    a.u[0] = Unpack<BITS>::pair(vwA, 2 * j, mg);
    a.u[1] = Unpack<BITS>::pair(vwA, 2 * j + 1, mg);
    a.u[2] = Unpack<BITS>::pair(vwB, 2 * j, mg);
    a.u[3] = Unpack<BITS>::pair(vwB, 2 * j + 1, mg);
    ib.acc[j] = mfma32(a.h, PV, ib.acc[j]);
  }
}

// End of an int block: O[d][h] += s_d * (acc - off * sum p) + z_d * sum p,
// d = 16j + 4kg + r, with the value scale/zero at vsz (LDS).  With VTOK the scales
// are already inside acc: O[d][h] += acc - off * sum p s + sum p z.
template <int BITS, bool VTOK>
__device__ __forceinline__ void int_epilogue(State &st, IntBlock &ib, const uint8_t *vsz, int lane) {
  if (VTOK) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float off = v_off<BITS>(j);
#pragma unroll
      for (int r = 0; r < 4; ++r) st.O[j][r] += fmaf(-off, ib.ps[r], ib.acc[j][r]) + ib.pz[r];
    }
    st.l += ib.pb[0];
    return;
  }
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

// Centroid block: one unit with both records (K at +0, V at +2 KB).
template <bool PACK, bool CERT>
__device__ __forceinline__ void centroid_item(const AttnParams &p, State &st, const uint8_t *qs, const uint8_t *ip,
                                              uint64_t valid, int lane, const float *cb) {
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
  const uint32_t *vid = (const uint32_t *)(ip + 2048 + KC * D * 2);
  const uint32_t ki = (kid[lane >> 4] >> (2 * (lane & 15))) & 3u;
  const uint32_t vi = (vid[lane >> 4] >> (2 * (lane & 15))) & 3u;
  U8 vc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) vc[i].v = kg == 0 ? lds16(ip + 2048 + m16 * 64 + 16 * i) : make_uint4(0, 0, 0, 0);
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
  if (CERT) cert_add(st, lsum, cb[0], cb[1]);
}

// One-centroid block: one unit with the key row at +0 and the value row at +2 KB.
// All read tokens share one key and one value, so the block adds one logit per head
// with weight (tokens read) x exp, and that weight times the value row.
template <bool PACK, bool CERT>
__device__ __forceinline__ void mean_item(const AttnParams &p, State &st, const uint8_t *qs, const uint8_t *ip,
                                          uint64_t valid, int lane, const float *cb) {
  const int kg = lane >> 4;
  // every row of A is the key row, so each output row holds the logit of the column's head
  f4 sc = {0, 0, 0, 0};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    U8 a;
    a.v = lds16(ip + (8 * kg + 32 * i) * 2);
    sc = mfma32(a.h, qchunk<PACK>(qs, lane, i), sc);
  }
  rescale_factor(st, sc[0] * p.sl2);
  const float w = (float)__popcll(valid) * __builtin_amdgcn_exp2f(fmaf(sc[0], p.sl2, -st.m));
  // O[channel 16j + 4kg + r][head] += w * v[channel]
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    U4 v;
    *(uint2 *)v.u = *(const uint2 *)(ip + 2048 + (16 * j + 4 * kg) * 2);
#pragma unroll
    for (int r = 0; r < 4; ++r) st.O[j][r] = fmaf(w, (float)v.h[r], st.O[j][r]);
  }
  st.l += w;
  if (CERT) cert_add(st, w, cb[0], cb[1]);
}

// Runs: process items of one level until the next item has another level (its
// descriptor left in meta/valid) or the items end (returns false).
template <bool PACK, bool CERT>
__device__ __forceinline__ bool exact_run(const AttnParams &p, State &st, const uint8_t *qs, Pipe &pp,
                                          uint32_t &meta, uint64_t &valid, int lane) {
  do {
    uint32_t tv = meta_tvalid(meta);
    if (pp.blk != 0xFFFFu) {  // a block's tile: its tokens at or past the length are not read
      const int64_t left = pp.tlim - (int64_t)pp.blk * P - 16 * __builtin_ctz(meta_tiles(meta));
      tv &= left >= 16 ? 0xFFFFu : (left <= 0 ? 0u : (1u << left) - 1u);
    }
    exact_tile<PACK, CERT>(p, st, qs, pp, tv, lane);
    if (!pp.template next_item<CERT>(meta, valid)) return false;
  } while (meta_lv(meta) == GKV_EXACT);
  return true;
}

template <int BITS, bool PACK, bool CERT, bool VTOK, bool QUEST>
__device__ __forceinline__ bool int_run(const AttnParams &p, State &st, const uint8_t *qs, Pipe &pp,
                                        uint32_t &meta, uint64_t &valid, int lane) {
  IntBlock ib;
  Mag mg;  // the exponent words, once per run
  if (BITS != 8) {
    mg.e1024 = opaque(E1024);
    mg.e256 = opaque(E256);
    mg.e64 = opaque(E64);
    mg.e16 = opaque(E16);
    mg.e4 = opaque(E4);
  }
  do {
    if (meta_first(meta)) {
      if (CERT) {
        ib.kerr = pp.cert[pp.blk * 4];
        ib.verr = pp.cert[pp.blk * 4 + 1];
      }
      const uint8_t *sz = pp.template pop<0>();
      int_header<BITS, PACK>(ib, qs, sz, lane);
      if (VTOK) {
        ib.ps = f4{0, 0, 0, 0};
        ib.pz = f4{0, 0, 0, 0};
      }
      *(uint2 *)(pp.ebuf + 8 * lane) = *(const uint2 *)(sz + 2048 + 8 * lane);  // V scale/zero, kept
      pp.release(1);
    }
    const int n = meta_ntiles(meta);
    // K and V codes in one unit (V at +2048): int2 items, and in a Compressed-Quest read
    // every item with at most 2 KB of codes per tensor
    const bool one_unit = BITS == 2 || (QUEST && n * 256 * BITS <= 2048);
    const uint8_t *kq = pp.template pop<0>();
    const uint8_t *vq = one_unit ? kq + 2048 : pp.template pop<1>();
    uint32_t tl = meta_tiles(meta);
    int j = 0;
#pragma unroll 1
    for (; j + 1 < n; j += 2) {  // tiles in pairs
      const int ta = __builtin_ctz(tl);
      tl &= tl - 1;
      const int tb = __builtin_ctz(tl);
      tl &= tl - 1;
      int_tile2<BITS, PACK, VTOK>(p, st, ib, kq + j * 256 * BITS, vq + j * 256 * BITS,
                                  (uint32_t)(valid >> (16 * ta)) & 0xFFFFu, (uint32_t)(valid >> (16 * tb)) & 0xFFFFu,
                                  mg, lane, ta, tb, pp.ebuf);
    }
    if (j < n) {
      const int ta = __builtin_ctz(tl);
      int_tile<BITS, PACK, VTOK>(p, st, ib, kq + j * 256 * BITS, vq + j * 256 * BITS,
                                 (uint32_t)(valid >> (16 * ta)) & 0xFFFFu, mg, lane, ta, pp.ebuf);
    }
    if (meta_last(meta)) {
      int_epilogue<BITS, VTOK>(st, ib, pp.ebuf, lane);
      if (CERT) cert_add(st, ib.pb[0], ib.kerr, ib.verr);
    }
    pp.release(one_unit ? 1 : 2);
    if (!pp.template next_item<CERT>(meta, valid)) return false;
  } while (meta_lv(meta) == BITS);
  return true;
}

template <bool PACK, bool CERT>
__device__ __forceinline__ bool centroid_run(const AttnParams &p, State &st, const uint8_t *qs, Pipe &pp,
                                             uint32_t &meta, uint64_t &valid, int lane) {
  do {
    centroid_item<PACK, CERT>(p, st, qs, pp.template pop<0>(), valid, lane, CERT ? pp.cert + pp.blk * 4 : nullptr);
    pp.release(1);
    if (!pp.template next_item<CERT>(meta, valid)) return false;
  } while (meta_lv(meta) == GKV_CENTROID);
  return true;
}

// A run of n = 2..8 one-centroid blocks whose records lie back to back in one unit
// (block g: key row at 512 g, value row at 512 g + 256), with cnt_g = (cnt >> 8 g) &
// 255 tokens read.  Row m of the logit MFMA's A is block m & 7's key row, so lane
// (kg, m) gets the logits of blocks 4 (kg & 1) + r; the weights cnt_g * p_g of
// blocks 4 kg + e (kg < 2) then form the B operand of one 16-deep P.V MFMA per
// channel group, whose contraction index runs over the blocks.  The slot bytes past
// the run are stale and never enter an MFMA: those key rows, weights and value
// operands are selected to zero (with stale key rows in the logit MFMA the results
// were measured to vary between identical calls).
template <bool PACK, bool CERT>
__device__ __forceinline__ void mean_run_item(const AttnParams &p, State &st, const uint8_t *qs, const uint8_t *ip,
                                              int n, uint64_t cnt, int lane, const float *cb) {
  const int kg = lane >> 4, m16 = lane & 15;
  f4 sc = {0, 0, 0, 0};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    U8 a;
    a.v = (m16 & 7) < n ? lds16(ip + 512 * (m16 & 7) + (8 * kg + 32 * i) * 2) : make_uint4(0, 0, 0, 0);
    sc = mfma32(a.h, qchunk<PACK>(qs, lane, i), sc);
  }
  float c[4];
  float bm = kNegInf;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int g = 4 * (kg & 1) + r;
    c[r] = (float)((cnt >> (8 * g)) & 255u);  // 0 for blocks >= n
    if (c[r] > 0.f) bm = vmax(bm, sc[r]);
  }
  rescale_factor(st, wave_max16(bm) * p.sl2);
  _Float16 wh[4];
  float lsum = 0.f;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const float w = c[r] > 0.f && kg < 2 ? c[r] * __builtin_amdgcn_exp2f(fmaf(sc[r], p.sl2, -st.m)) : 0.f;
    wh[r] = (_Float16)w;
    lsum += (float)wh[r];
  }
  const half4 Bw = half4{wh[0], wh[1], wh[2], wh[3]};
#pragma unroll
  for (int j = 0; j < 8; ++j) {  // O[16 j + row][head] += sum_g v_g[16 j + row] w_g[head]
    half4 av;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int g = 4 * kg + e;
      av[e] = kg < 2 && g < n ? *(const _Float16 *)(ip + 512 * g + 256 + 2 * (16 * j + m16)) : (_Float16)0;
    }
    st.O[j] = mfma16(av, Bw, st.O[j]);
  }
  st.l += wave_sum16(lsum);
  if (CERT) {
    float c1 = 0.f, c2 = 0.f, c3 = 0.f;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int g = 4 * kg + r;
      if (kg < 2 && g < n) {
        const float pb = (float)wh[r], x = st.es * cb[4 * g];
        c1 = fmaf(pb, cb[4 * g + 1], c1);
        c2 = fmaf(pb, __builtin_amdgcn_exp2f(x), c2);
        c3 = fmaf(pb, __builtin_amdgcn_exp2f(-x), c3);
      }
    }
    st.c1 += wave_sum16(c1);
    st.c2 += wave_sum16(c2);
    st.c3 += wave_sum16(c3);
  }
}

template <bool PACK, bool CERT>
__device__ __forceinline__ bool mean_run(const AttnParams &p, State &st, const uint8_t *qs, Pipe &pp,
                                         uint32_t &meta, uint64_t &valid, int lane) {
  do {
    const int n = meta_ntiles(meta) + 1;
    if (n > 1)
      mean_run_item<PACK, CERT>(p, st, qs, pp.template pop<0>(), n, valid, lane,
                                CERT ? pp.cert + pp.blk * 4 : nullptr);
    else
      mean_item<PACK, CERT>(p, st, qs, pp.template pop<0>(), valid, lane, CERT ? pp.cert + pp.blk * 4 : nullptr);
    pp.release(1);
    if (!pp.template next_item<CERT>(meta, valid)) return false;
  } while (meta_lv(meta) == GKV_MEAN);
  return true;
}

// Compressed-Quest reads take no plan: each wavefront writes its own item and unit
// lists (defined with the plan code below).
__device__ __forceinline__ uint2 quest_lists(const AttnParams &p, int64_t u, int w, int W, int lane,
                                             ItemDesc *items, UnitDesc *units);

template <bool PACK, bool CERT, bool VTOK, bool QUEST>
__global__ void __launch_bounds__(kThreads, 2) attn_kernel(AttnParams p) {
  extern __shared__ __align__(16) uint8_t smem[];
  // Workgroup L of the one-dimensional grid serves (b, KV head) L % units as its
  // workgroup L / units, so that the workgroups dispatched first cover every (b, KV head).
  const int units = (int)gridDim.x / p.nsplit;
  const int sidx = (int)blockIdx.x / units, h = (int)blockIdx.x % units % p.Hkv, b = (int)blockIdx.x % units / p.Hkv;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int kg = lane >> 4, m16 = lane & 15;
  const int64_t u = (int64_t)b * p.Hkv + h;
  const int W = p.nsplit * kWaves, w = sidx * kWaves + wave;
  if (p.cacheable && blockIdx.x == 0 && threadIdx.x == 0) {
    // the plan kernel of this call has finished: the workspace now holds the plan of
    // this key (vector stores; read by later calls' plan kernels)
#pragma unroll
    for (int i = 0; i < kTagWords; ++i) p.tag[i] = p.key[i];
  }

  // the group's queries (rows of absent heads are zero): one 16-byte piece per thread,
  // loaded here and stored to LDS once the wavefront's lists are set up, so that the
  // loads of both are in flight together
  static_assert(16 * (D / 8) == kThreads, "one query piece per thread");
  uint8_t *qs = smem + kWaves * kWaveLds;
  const int qg = threadIdx.x / (D / 8), qc8 = (threadIdx.x % (D / 8)) * 8;
  const uint4 qv = qg < p.G ? *(const uint4 *)(p.q + (u * p.G + qg) * D + qc8) : make_uint4(0, 0, 0, 0);

  // ---------------- this wavefront's item and unit lists
  Pipe pp;
  uint8_t *wl = smem + wave * kWaveLds;
  pp.ring = wl;
  pp.uchunk = wl + kRing;
  pp.ichunk = wl + kRing + 1024;
  pp.ebuf = wl + kRing + 2048;
  pp.ring_base = (uint32_t)uni((int32_t)(uintptr_t)pp.ring);
  pp.ulds = (uint32_t)uni((int32_t)(uintptr_t)pp.uchunk);
  pp.ilds = (uint32_t)uni((int32_t)(uintptr_t)pp.ichunk);
  pp.cert = CERT ? p.cert + u * p.nblk_cap * 4 : nullptr;
  pp.blk = 0xFFFFu;
  pp.tlim = uni64(unit_T(p, u));
  if (QUEST) {
    // Compressed-Quest: this wavefront's share of the read pages, listed in LDS here
    const uint2 n = quest_lists(p, u, w, W, lane, (ItemDesc *)pp.ichunk, (UnitDesc *)pp.uchunk);
    pp.isrc = pp.usrc = nullptr;
    pp.nitems = (uint32_t)uni((int32_t)n.x);
    pp.nunits = (uint32_t)uni((int32_t)n.y);
    pp.start(lane, true);
  } else {
    // this wavefront's items and units, from the plan
    const int32_t *isp = p.split + u * (int64_t)(2 * (W + 1)), *usp = isp + (W + 1);
    const uint32_t i0 = (uint32_t)uni(isp[w]), i1 = (uint32_t)uni(isp[w + 1]);
    const uint32_t u0 = (uint32_t)uni(usp[w]), u1 = (uint32_t)uni(usp[w + 1]);
    pp.isrc = p.plan + (u * p.icap + i0) * (int64_t)sizeof(ItemDesc);
    pp.usrc = p.units + (u * p.ucap + u0) * (int64_t)sizeof(UnitDesc);
    pp.nitems = i1 - i0;
    pp.nunits = u1 - u0;
    pp.start(lane, false);
  }
  *(uint4 *)(qs + qg * kQRow + qc8 * 2) = qv;
  __syncthreads();
  State st;
#pragma unroll
  for (int j = 0; j < 8; ++j) st.O[j] = f4{0, 0, 0, 0};
  st.m = kNegInf;
  st.l = 0.f;
  st.c1 = st.c2 = st.c3 = 0.f;
  st.es = 0.f;
  if (CERT) {  // ||q|| of this lane's head, for eps_b = ||q|| kerr_b / sqrt(D)
    float qq = 0.f;
    for (int c8 = 0; c8 < D; c8 += 8) {
      U8 t;
      t.v = lds16(qs + qrow<PACK>(lane) * kQRow + c8 * 2);
#pragma unroll
      for (int e = 0; e < 8; ++e) qq = fmaf((float)t.h[e], (float)t.h[e], qq);
    }
    st.es = __builtin_sqrtf(qq) * p.sl2;  // sl2 = log2(e) / sqrt(D)
  }

  // ---------------- pipelined item loop
  // Items are processed in runs of one level, each run in a loop specialised for
  // that level (the constants of one level's path are then live only in its loop).
  uint32_t meta;
  uint64_t valid;
  bool more = pp.template next_item<CERT>(meta, valid);
  while (more) {
    switch (meta_lv(meta)) {
      case GKV_EXACT: more = exact_run<PACK, CERT>(p, st, qs, pp, meta, valid, lane); break;
      case GKV_INT8: more = int_run<8, PACK, CERT, VTOK, QUEST>(p, st, qs, pp, meta, valid, lane); break;
      case GKV_INT4: more = int_run<4, PACK, CERT, VTOK, QUEST>(p, st, qs, pp, meta, valid, lane); break;
      case GKV_INT2: more = int_run<2, PACK, CERT, VTOK, QUEST>(p, st, qs, pp, meta, valid, lane); break;
      case GKV_CENTROID: more = centroid_run<PACK, CERT>(p, st, qs, pp, meta, valid, lane); break;
      default: more = mean_run<PACK, CERT>(p, st, qs, pp, meta, valid, lane); break;
    }
  }
  vm_wait<0>();

  // ---------------- merge the four wavefronts and write one partial per head
  __syncthreads();
  float(*so)[16][D + 1] = (float(*)[16][D + 1])smem;
  float *sm = (float *)(smem + kWaves * 16 * (D + 1) * 4);
  float *sl = sm + kWaves * 16;
  float *scs = sl + kWaves * 16;  // certificate sums [3][kWaves * 16]
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int r = 0; r < 4; ++r) so[wave][m16][16 * j + 4 * kg + r] = st.O[j][r];
  if (kg == 0) {
    sm[wave * 16 + m16] = st.m;
    sl[wave * 16 + m16] = st.l;
    if (CERT) {
      scs[wave * 16 + m16] = st.c1;
      scs[kWaves * 16 + wave * 16 + m16] = st.c2;
      scs[2 * kWaves * 16 + wave * 16 + m16] = st.c3;
    }
  }
  __syncthreads();
  float *out = p.part + (u * p.nsplit + sidx) * (int64_t)p.G * kPart;
  for (int i = threadIdx.x; i < p.G * D; i += kThreads) {
    const int g = i >> 7, d = i & 127;
    float M = kNegInf;
#pragma unroll
    for (int q = 0; q < kWaves; ++q) M = fmaxf(M, sm[q * 16 + g]);
    float L = 0.f, o = 0.f, cc = 0.f;  // cc: certificate sum d (d < 3)
    if (M > kNegInf) {
#pragma unroll
      for (int q = 0; q < kWaves; ++q) {
        const float a = __builtin_amdgcn_exp2f(sm[q * 16 + g] - M);
        L = fmaf(sl[q * 16 + g], a, L);
        o = fmaf(so[q][g][d], a, o);
        if (CERT && d < 3) cc = fmaf(scs[d * kWaves * 16 + q * 16 + g], a, cc);
      }
    }
    out[g * kPart + 2 + d] = o;
    if (d == 0) {
      out[g * kPart] = M;
      out[g * kPart + 1] = L;
    }
    if (CERT && d < 3) out[g * kPart + D + 2 + d] = cc;
  }
}

// ---------------------------------------------------------------- merge
// One workgroup per (head, (b, KV head)), one thread per channel: the partials
// (m_s, l_s, o_s) of the nsplit workgroups combine to o = sum_s a_s o_s / sum_s a_s l_s
// with a_s = 2^(m_s - max_s m_s).
__global__ void __launch_bounds__(D) merge_kernel(const float *part, float *out, int nsplit, int G, float *bound,
                                                  const float *cert, int nblk_cap, int nblk,
                                                  const int64_t *seq_len, int Hkv) {
  __shared__ float sa[kMaxWaves / kWaves], sl[kMaxWaves / kWaves];
  __shared__ float sinv, svm[D];
  const int g = blockIdx.x, d = threadIdx.x;
  const int64_t u = blockIdx.y;
  const int64_t stride = (int64_t)G * kPart;
  const float *base = part + u * nsplit * stride + g * kPart;
  for (int s2 = d; s2 < nsplit; s2 += D) {
    sa[s2] = base[s2 * stride];
    sl[s2] = base[s2 * stride + 1];
  }
  if (seq_len) {  // this sequence's blocks
    const int64_t t = seq_len[u / Hkv];
    nblk = t > 0 ? (int)((t + P - 1) / P) : 0;
  }
  if (bound) {  // max_b vmax_b over the blocks of this (b, KV head)
    float vm = 0.f;
    for (int b = d; b < nblk; b += D) vm = fmaxf(vm, cert[(u * nblk_cap + b) * 4 + 2]);
    svm[d] = vm;
  }
  __syncthreads();
  if (d < 64) {  // the first wavefront: the split weights a_s and L, lane d over splits d, d + 64, ...
    float M = kNegInf;
    for (int s2 = d; s2 < nsplit; s2 += 64) M = fmaxf(M, sa[s2]);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) M = fmaxf(M, __shfl_xor(M, o));
    float L = 0.f;
    for (int s2 = d; s2 < nsplit; s2 += 64) {
      const float a = sa[s2] == kNegInf ? 0.f : __builtin_amdgcn_exp2f(sa[s2] - M);
      sa[s2] = a;
      L = fmaf(a, sl[s2], L);
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) L += __shfl_xor(L, o);
    if (d == 0) sinv = L > 0.f ? 1.0f / L : 0.f;  // an empty sequence reads nothing: its output is zero
    // lane 0 reads the weights the wavefront's lanes wrote (LDS keeps one wavefront's order)
    if (d == 0 && bound && !(L > 0.f)) bound[u * G + g] = 0.f;
    if (d == 0 && bound && L > 0.f) {  // section 3.6: sum_b a_b verr_b + min(2, M+/M- - M-/M+) max_j ||v_j||
      float c1 = 0.f, c2 = 0.f, c3 = 0.f, vm = 0.f;
      for (int s2 = 0; s2 < nsplit; ++s2) {
        c1 = fmaf(sa[s2], base[s2 * stride + D + 2], c1);
        c2 = fmaf(sa[s2], base[s2 * stride + D + 3], c2);
        c3 = fmaf(sa[s2], base[s2 * stride + D + 4], c3);
      }
      for (int i = 0; i < D; ++i) vm = fmaxf(vm, svm[i]);
      const float r = c2 / c3;
      bound[u * G + g] = c1 / L + fminf(2.f, r - 1.0f / r) * vm;
    }
  }
  __syncthreads();
  float o = 0.f;
  int s2 = 0;
  for (; s2 + 16 <= nsplit; s2 += 16) {
    float v[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) v[k] = base[(s2 + k) * stride + 2 + d];
#pragma unroll
    for (int k = 0; k < 16; ++k) o = fmaf(sa[s2 + k], v[k], o);
  }
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
// Dense reads: up to 8 workgroups per (b, KV head).  A visit is one block and the
// tokens of it that are read: all valid tokens minus the residual rows.  The plan
// kernel describes the visits, splits them over the W wavefronts by a balance cost
// (visit v goes to the wavefront that owns the midpoint of its cost interval), and
// expands every visit into its pipeline items, written in order; each wavefront's
// items are the items of its visits.  Compressed-Quest reads have no plan kernel:
// their wavefronts list their own pages (quest_lists).
constexpr int kPlanThreads = 1024;

struct VisitDesc {
  uint64_t kp, vp;  // addresses of the K and V records
  uint64_t valid;   // tokens of the block that are read (bit t = token t)
  int16_t level;    // storage level of both records; a run of n one-centroid blocks
                    // (dense reads) carries n - 1 in bits 8..10 and 8-bit token counts
                    // per block in `valid`
  uint16_t blk;     // block index (0xFFFF: residual rows or a Compressed-Quest visit)
  uint32_t cost;    // balance cost (bits 0..23) | items (bits 24..26) | units (bits 27..30)
};
static_assert(sizeof(VisitDesc) == 32, "descriptor size");
// Balance cost of a visit: the measured time of its parts on one wavefront sharing
// its SIMD (about 8 cycles per unit).  Exact tiles are bound by the wavefront's
// share of the bandwidth (8 KB each), int tiles by the dequantisation and softmax
// work rather than by their bytes.
constexpr uint32_t kCostExactTile = 551, kCostInt8Tile = 426, kCostInt4Tile = 340, kCostInt2Tile = 306,
                   kCostCentroid = 799, kCostIntBlock = 248, kCostMean = 300, kCostMeanRun = 260,
                   kCostMeanRunBlock = 45;

// Blocks in a one-centroid run (1 for every other visit) and the visit's level.
__device__ __forceinline__ int run_blocks(int lv) { return ((lv >> 8) & 7) + 1; }
__device__ __forceinline__ int run_level(int lv) { return lv & 0xFF; }

__device__ __forceinline__ uint32_t balance_cost(int lv, uint64_t va) {
  if (run_blocks(lv) > 1) return kCostMeanRun + kCostMeanRunBlock * run_blocks(lv);
  uint32_t tiles = 0;
  for (int t = 0; t < 4; ++t) tiles += ((va >> (16 * t)) & 0xFFFFull) != 0;
  if (!tiles) return 0;
  if (lv == GKV_CENTROID) return kCostCentroid;
  if (lv == GKV_MEAN) return kCostMean;
  if (lv == GKV_EXACT) return tiles * kCostExactTile;
  const uint32_t per = lv == 8 ? kCostInt8Tile : (lv == 4 ? kCostInt4Tile : kCostInt2Tile);
  return kCostIntBlock + tiles * per;
}

__device__ __forceinline__ uint64_t token_mask(int64_t left) {  // tokens of a block below `left`
  return left >= P ? ~0ull : (left <= 0 ? 0ull : ((1ull << left) - 1));
}

// Wavefront inclusive scan of a 32-bit value in lane order: DPP row shifts within
// each row of 16 lanes, then row broadcasts between rows.
template <int CTRL, int ROWS>
__device__ __forceinline__ uint32_t dpp_add(uint32_t x) {
  return x + (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, ROWS, 0xF, true);
}
__device__ __forceinline__ uint32_t wave_scan32(uint32_t x) {
  x = dpp_add<0x111, 0xF>(x);  // row_shr:1
  x = dpp_add<0x112, 0xF>(x);  // row_shr:2
  x = dpp_add<0x114, 0xF>(x);  // row_shr:4
  x = dpp_add<0x118, 0xF>(x);  // row_shr:8
  x = dpp_add<0x142, 0xA>(x);  // row_bcast:15 into rows 1, 3
  x = dpp_add<0x143, 0xC>(x);  // row_bcast:31 into rows 2, 3
  return x;
}

// Inclusive scan over the workgroup of packed scan keys (cost | units | items, see
// scan_key); `total` receives the sum over all threads.  The three fields are scanned
// as 32-bit values, which equals the 64-bit sum since no field overflows.
__device__ __forceinline__ uint64_t block_scan(uint64_t x, uint64_t *sh, uint64_t &total) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  constexpr int NW = kPlanThreads / 64;
  uint32_t c = wave_scan32((uint32_t)(x >> 35)), un = wave_scan32((uint32_t)(x >> 17) & 0x3FFFFu),
           it = wave_scan32((uint32_t)x & 0x1FFFFu);
  uint32_t *s32 = (uint32_t *)sh;  // [3][NW] wave totals, then [3][NW] exclusive wave offsets
  if (lane == 63) {
    s32[wv] = c;
    s32[NW + wv] = un;
    s32[2 * NW + wv] = it;
  }
  __syncthreads();
  if (wv == 0 && lane < 3 * NW) {  // 48 lanes: three 16-wave scans
    const int f = lane / NW, q = lane % NW;
    uint32_t t = s32[lane];
    for (int o = 1; o < NW; o <<= 1) {
      const uint32_t y = __shfl_up(t, o);
      if (q >= o) t += y;
    }
    s32[3 * NW + f * NW + q] = t;  // inclusive over waves
  }
  __syncthreads();
  const uint32_t *inc = s32 + 3 * NW;
  if (wv) {
    c += inc[wv - 1];
    un += inc[NW + wv - 1];
    it += inc[2 * NW + wv - 1];
  }
  total = ((uint64_t)inc[NW - 1] << 35) | ((uint64_t)inc[2 * NW - 1] << 17) | inc[3 * NW - 1];
  __syncthreads();
  return ((uint64_t)c << 35) | ((uint64_t)un << 17) | it;
}

// Items and units of a visit (as visit_items writes them): items | units << 3.
__device__ __forceinline__ uint32_t visit_counts(int lv, uint64_t valid, bool kv_one = false) {
  if (run_blocks(lv) > 1) return 1u | (1u << 3);
  uint32_t tiles = 0;
  for (int t = 0; t < 4; ++t)
    if ((valid >> (16 * t)) & 0xFFFFull) tiles |= 1u << t;
  if (!tiles) return 0;
  if (lv == GKV_CENTROID || lv == GKV_MEAN) return 1u | (1u << 3);
  if (lv == GKV_EXACT) return (uint32_t)__builtin_popcount(tiles) * (1u | (2u << 3));
  const int tg = group_tiles(lv);
  uint32_t k = 0, m = 1;  // items; units (the scale/zero unit first)
  while (tiles) {
    const uint32_t t = __builtin_ctz(tiles);
    uint32_t n = 1;
    while ((int)n < tg && ((tiles >> (t + n)) & 1u)) ++n;
    tiles &= ~(((1u << n) - 1) << t);
    ++k;
    m += lv == 2 || (kv_one && n * 256 * (uint32_t)lv <= 2048) ? 1u : 2u;  // K and V codes in one unit or two
  }
  return k | (m << 3);
}

// A unit of part A (ba bytes from a) and part B (bb bytes from b); each part at most
// 2 KB, part A at least 16 bytes.
__device__ __forceinline__ uint64_t unit_part(uint64_t a, uint32_t bytes) {
  const uint32_t n0 = (bytes < 1024 ? bytes : 1024) / 16, n1 = (bytes > 1024 ? bytes - 1024 : 0) / 16;
  return a | ((uint64_t)n0 << 48) | ((uint64_t)n1 << 56);
}
__device__ __forceinline__ UnitDesc unit_desc(uint64_t a, uint32_t ba, uint64_t b, uint32_t bb) {
  UnitDesc d;
  d.a = unit_part(a, ba);
  d.b = bb ? unit_part(b, bb) : unit_part(a, 16);
  return d;
}

// Writes the items and units of a visit, in order.
__device__ __forceinline__ void visit_items(const VisitDesc &v, ItemDesc *items, UnitDesc *units, bool kv_one = false) {
  uint32_t tiles = 0;
  for (int t = 0; t < 4; ++t)
    if ((v.valid >> (16 * t)) & 0xFFFFull) tiles |= 1u << t;
  if (!tiles) return;
  const uint32_t lv = (uint32_t)run_level(v.level);
  if (run_blocks(v.level) > 1) {  // one-centroid run: one item, one unit of back-to-back records
    const uint32_t n = (uint32_t)run_blocks(v.level), bytes = 512 * n;
    items[0].meta = kMean | (lv << 2) | (1u << 7) | (1u << 8) | ((n - 1) << 13);
    items[0].pad = v.blk;
    items[0].valid = v.valid;
    units[0] = unit_desc(v.kp, bytes < 2048 ? bytes : 2048, v.kp + 2048, bytes > 2048 ? bytes - 2048 : 0);
    return;
  }
  auto put = [&](int i, uint32_t kind, bool first, bool last, uint32_t taken, uint32_t n, uint32_t tv) {
    items[i].meta = kind | (lv << 2) | ((uint32_t)first << 7) | ((uint32_t)last << 8) | (taken << 9) | (n << 13) |
                    (tv << 16);
    items[i].pad = v.blk;
    items[i].valid = v.valid;
  };
  if (lv == GKV_CENTROID) {
    put(0, kCentroid, true, true, tiles, 1, 0);
    units[0] = unit_desc(v.kp, kCentBytes, v.vp, kCentBytes);
    return;
  }
  if (lv == GKV_MEAN) {
    put(0, kMean, true, true, tiles, 0, 0);
    units[0] = unit_desc(v.kp, kMeanBytes, v.vp, kMeanBytes);
    return;
  }
  int k = 0, m = 0;
  if (lv == GKV_EXACT) {
    for (int t = 0; t < 4; ++t)
      if ((tiles >> t) & 1u) {
        put(k++, kExactTile, true, true, 1u << t, 1, (uint32_t)((v.valid >> (16 * t)) & 0xFFFFull));
        units[m++] = unit_desc(v.kp + 4096 * t, 2048, v.kp + 4096 * t + 2048, 2048);
        units[m++] = unit_desc(v.vp + 4096 * t, 2048, v.vp + 4096 * t + 2048, 2048);
      }
    return;
  }
  units[m++] = unit_desc(v.kp, kSZBytes, v.vp, kSZBytes);
  const int tg = group_tiles((int)lv);
  uint32_t left = tiles;
  bool first = true;
  while (left) {
    const uint32_t t = __builtin_ctz(left);
    uint32_t n = 1;
    while ((int)n < tg && ((left >> (t + n)) & 1u)) ++n;
    const uint32_t taken = ((1u << n) - 1) << t;
    left &= ~taken;
    put(k++, kIntGroup, first, left == 0, taken, n, 0);
    const uint32_t off = kSZBytes + t * 256 * lv, span = n * 256 * lv;
    if (lv == 2 || (kv_one && span <= 2048)) {  // the K and V codes share one unit (V at +2048)
      units[m++] = unit_desc(v.kp + off, span, v.vp + off, span);
    } else {
      const uint32_t pa = span < 2048 ? span : 2048, pb = span - pa;
      units[m++] = unit_desc(v.kp + off, pa, v.kp + off + 2048, pb);
      units[m++] = unit_desc(v.vp + off, pa, v.vp + off + 2048, pb);
    }
    first = false;
  }
}

// Read pages per wavefront of a Compressed-Quest read: at most 8 tiles, so that a
// wavefront's items and units fit one 32-entry descriptor chunk each (a tile costs at
// most 3 units: an int8 page alone in its block takes its scale/zero unit and a K and
// a V unit).
// With residual rows a page also brings the residual tiles holding its tokens' rows
// (a 16-token page's rows span at most 2 tiles, 4 units), so a wavefront takes half as
// many pages.
__host__ __device__ __forceinline__ int quest_pages_per_wave(int page, bool residual) {
  return (residual ? 4 : 8) / (page / 16);
}

// A 64-bit value of lane l (l uniform).
__device__ __forceinline__ int64_t lane64(int64_t x, int l) {
  const uint32_t lo = __builtin_amdgcn_readlane((int)(uint32_t)x, l);
  const uint32_t hi = __builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)x >> 32), l);
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Wavefront w of W of (b, KV head) u in a Compressed-Quest read: the read slots are
// the topk selected pages (ascending; an entry below 0 or at or past the current
// page, such as the -1 padding, reads nothing) and then the current page
// (T - 1) / page.  The wavefront takes slots [w n / W, (w + 1) n / W) of those
// n = topk + 1, joins consecutive pages of one block into one visit, and writes the
// visits' items and units (as the dense plan expands its visits) into `items` and
// `units` (LDS).  Lane s loads slot i0 + s's page and then its block's table entries,
// so the lists cost two dependent memory round trips whatever the wavefront's page
// count; the visits are then built from registers.  An int4/int8 item with at most 2 KB
// of codes per tensor copies its K and V codes in one unit.  Returns (items, units).
__device__ __forceinline__ uint2 quest_lists(const AttnParams &p, int64_t u, int w, int W, int lane,
                                             ItemDesc *items, UnitDesc *units) {
  const int32_t *pg = p.pages + u * p.topk;
  const int64_t Tu = unit_T(p, u);
  if (Tu == 0) return make_uint2(0, 0);  // an empty or retired sequence reads nothing
  const int64_t cur = (Tu - 1) / p.page;
  const int n = p.topk + 1;
  const int i0 = (int)(((int64_t)w * n) / W), i1 = (int)(((int64_t)(w + 1) * n) / W);
  // page pg lies in block pg >> pshift and covers tiles page_tiles(pg) of it
  const int pshift = p.page == 16 ? 2 : (p.page == 32 ? 1 : 0), tpp = p.page / 16;
  auto page_tiles = [&](int64_t q) { return ((1u << tpp) - 1) << ((q & ((1 << pshift) - 1)) * tpp); };
  // this lane's slot: its page (-1: nothing to read) and its block's table entries
  const int si = i0 + lane;
  int64_t q = -1;
  if (si < i1) {
    if (si < p.topk) {
      const int64_t x = pg[si];
      q = x >= 0 && x < cur ? x : -1;
    } else {
      q = cur;
    }
  }
  int64_t lv = 0, kof = 0, vof = 0, bmask = 0, roff = 0;
  if (q >= 0) {
    const int64_t blk = u * p.nblk_cap + (q >> pshift);
    lv = p.level[blk];
    kof = p.koff[blk];
    vof = p.voff[blk];
    if (p.nres) {
      bmask = (int64_t)p.res_mask[blk];
      roff = p.res_off[u * (p.nblk_cap + 1) + (q >> pshift)];
    }
  }
  const int ns = i1 - i0;
  uint32_t ni = 0, nu = 0;
  for (int s = 0; s < ns;) {
    const int64_t q0 = lane64(q, s);
    if (q0 < 0) {
      ++s;
      continue;
    }
    const int64_t blk = q0 >> pshift;
    uint32_t tl = page_tiles(q0);
    int t = s + 1;
    for (; t < ns; ++t) {
      const int64_t qt = lane64(q, t);
      if (qt < 0) continue;
      if ((qt >> pshift) != blk) break;
      tl |= page_tiles(qt);
    }
    VisitDesc d;
    d.level = (int16_t)__builtin_amdgcn_readlane((int)lv, s);
    d.blk = 0xFFFF;
    d.kp = (uint64_t)(uintptr_t)(p.arena + lane64(kof, s));
    d.vp = (uint64_t)(uintptr_t)(p.arena + lane64(vof, s));
    uint64_t va = 0;
    for (int tt = 0; tt < 4; ++tt)
      if (tl & (1u << tt)) va |= 0xFFFFull << (16 * tt);
    d.valid = va & token_mask(Tu - blk * P);
    d.cost = 0;
    // residual rows override their tokens (section 3.4): the graded tiles skip them
    // and the exact tiles of the residual that hold their rows are read instead
    uint64_t bm = 0, rm = 0;
    if (p.nres) {
      bm = (uint64_t)lane64(bmask, s);
      rm = bm & d.valid;
      d.valid &= ~bm;
    }
    const uint32_t c = visit_counts(d.level, d.valid, true);
    if (lane == 0) visit_items(d, items + ni, units + nu, true);
    ni += c & 7u;
    nu += c >> 3;
    if (rm) {
      const int32_t r0 = __builtin_amdgcn_readlane((int)roff, s);
      auto row_of = [&](uint64_t t) { return r0 + __popcll(bm & ((1ull << t) - 1)); };
      while (rm) {  // the read tokens' rows, ascending: one exact tile item per 16 rows
        const int rt = row_of(__builtin_ctzll(rm)) >> 4;
        uint32_t tv = 0;
        while (rm) {
          const int r = row_of(__builtin_ctzll(rm));
          if ((r >> 4) != rt) break;
          tv |= 1u << (r & 15);
          rm &= rm - 1;
        }
        const uint64_t kp = (uint64_t)(uintptr_t)(p.res_rows + (u * p.nrb_cap + (rt >> 2)) * (2 * kExactBytes) +
                                                  4096 * (rt & 3));
        if (lane == 0) {
          items[ni].meta = kExactTile | ((uint32_t)GKV_EXACT << 2) | (1u << 7) | (1u << 8) |
                           ((1u << (rt & 3)) << 9) | (1u << 13) | (tv << 16);
          items[ni].pad = 0xFFFF;
          items[ni].valid = 0;
          units[nu] = unit_desc(kp, 2048, kp + 2048, 2048);
          units[nu + 1] = unit_desc(kp + kExactBytes, 2048, kp + kExactBytes + 2048, 2048);
        }
        ni += 1;
        nu += 2;
      }
    }
    s = t;
  }
  return make_uint2(ni, nu);
}

// Tokens read from block b of a dense read (residual rows excluded).
__device__ __forceinline__ uint64_t dense_tokens(const AttnParams &p, int64_t u, int64_t b) {
  uint64_t va = token_mask(plan_T(p, u) - b * P);
  if (p.nres) va &= ~p.res_mask[u * p.nblk_cap + b];
  return va;
}

// Whether one-centroid block b continues the run of block b - 1: both one-centroid
// and read, inside one aligned group of 8 blocks, each block's value row right after
// its key row and block b's key row right after block b - 1's value row.
__device__ __forceinline__ bool mean_joins(const AttnParams &p, int64_t u, int64_t b) {
  if ((b & 7) == 0) return false;
  const int64_t i = u * p.nblk_cap + b;
  if (p.level[i] != GKV_MEAN || p.level[i - 1] != GKV_MEAN) return false;
  const int64_t k0 = p.koff[i - 1], k1 = p.koff[i];
  if (p.voff[i - 1] != k0 + kMeanBytes || k1 != k0 + 2 * kMeanBytes || p.voff[i] != k1 + kMeanBytes) return false;
  return dense_tokens(p, u, b - 1) != 0 && dense_tokens(p, u, b) != 0;
}

// One-centroid block v of a dense read, with jn the plan's bitmap of mean_joins: a
// block that continues a run is read by the run's first block (no items, no cost); a
// first block takes the run's following blocks and their token counts.
__device__ __forceinline__ void mean_run_visit(const AttnParams &p, int64_t u, int64_t v, const uint32_t *jn,
                                               VisitDesc &d) {
  const uint32_t grp = (jn[v >> 5] >> (v & 24)) & 255u;  // the joins bits of v's aligned group of 8
  const int o = (int)(v & 7);
  if ((grp >> o) & 1u) {
    d.valid = 0;
    return;
  }
  const int n = 1 + __builtin_ctz(~(grp >> (o + 1)) | (1u << (7 - o)));  // following set bits, to the group end
  if (n == 1) return;
  uint64_t cnt = 0;
  for (int g = 0; g < n; ++g) cnt |= (uint64_t)__popcll(dense_tokens(p, u, v + g)) << (8 * g);
  d.valid = cnt;
  d.level = (int16_t)(GKV_MEAN | ((n - 1) << 8));
}

// Position, in a range of n blocks, of visit v.  The aligned groups of 8 blocks are
// visited from the four quarters of the range in turn (a transpose of the first
// 4 * (n / 32) groups; the blocks after them keep their places), so that every
// wavefront's contiguous share holds blocks of the whole ladder: the old centroid and
// int2 blocks, whose dequantisation keeps the VALU busy, beside int8 and exact blocks,
// bound by their bytes.  The two wavefronts that share a SIMD then carry like mixes;
// with shares of one level each, an int4 wavefront beside an int2 one ended 13 us after
// the same int4 share beside a centroid one.  A group's blocks keep their order, so
// one-centroid runs stay whole.
__device__ __forceinline__ int64_t visit_block(int64_t v, int64_t n) {
  const int64_t q = n / 32;  // groups per quarter
  if (v >= 32 * q) return v;
  const int64_t g = v >> 3;
  return (((g & 3) * q + (g >> 2)) << 3) | (v & 7);
}

// Visit v of a dense read.  The blocks 0..nblk-1 and after them the residual
// pseudo-blocks form one range, visited in the order of visit_block, so that the
// residual's exact tiles spread over the last wavefronts' shares too.
__device__ __forceinline__ VisitDesc dense_visit(const AttnParams &p, int64_t u, int64_t nblk, int64_t v,
                                                 const uint32_t *jn) {
  VisitDesc d;
  v = visit_block(v, nblk + (p.nres + P - 1) / P);
  if (v < nblk) {
    const int64_t b = v;
    d.level = p.level[u * p.nblk_cap + b];
    d.blk = (uint16_t)b;
    d.kp = (uint64_t)(uintptr_t)(p.arena + p.koff[u * p.nblk_cap + b]);
    d.vp = (uint64_t)(uintptr_t)(p.arena + p.voff[u * p.nblk_cap + b]);
    d.valid = token_mask(plan_T(p, u) - b * P);
    if (p.nres) d.valid &= ~p.res_mask[u * p.nblk_cap + b];
    if (jn && d.level == GKV_MEAN && d.valid) mean_run_visit(p, u, b, jn, d);
  } else {
    const int64_t rb = v - nblk;
    const uint8_t *kp = p.res_rows + (u * p.nrb_cap + rb) * (2 * kExactBytes);
    d.level = GKV_EXACT;
    d.blk = 0xFFFF;
    d.kp = (uint64_t)(uintptr_t)kp;
    d.vp = (uint64_t)(uintptr_t)(kp + kExactBytes);
    d.valid = token_mask(p.nres - rb * P);
  }
  d.cost = balance_cost(d.level, d.valid) | (visit_counts(d.level, d.valid) << 24);
  return d;
}

// Wavefront owning the midpoint of cost interval [e, e + c) of a total, in fp64
// (every operand is an integer below 2^53, and the floor of a monotone quotient
// keeps the owners non-decreasing along the visits).
// The first W1 wavefronts (those of the workgroups dispatched first, which win the
// issue arbitration against the later ones on their SIMDs) get kFastCap capacity
// units, the others kSlowCap (measured: 1.33 times the work in the same time).
// The position is scaled by cap / (2 total), taken once per plan (a product with a
// positive constant is monotone, so the owners stay non-decreasing).
constexpr double kFastCap = 23.0, kSlowCap = 17.25;
__device__ __forceinline__ double owner_scale(int W, int W1, uint64_t total) {
  return total ? (kFastCap * W1 + kSlowCap * (W - W1)) / (2.0 * (double)total) : 0.0;
}
__device__ __forceinline__ int midpoint_owner(int W, int W1, uint64_t e, uint32_t c, double scale) {
  const double x = (double)(2 * e + c) * scale;
  const double o = x < kFastCap * W1 ? __builtin_floor(x * (1.0 / kFastCap))
                                     : W1 + __builtin_floor((x - kFastCap * W1) * (1.0 / kSlowCap));
  return o < (double)W ? (int)o : W - 1;
}

// Cost, units and items of a visit packed for one prefix scan: cost (bits 35..63) |
// units (17..34) | items (0..16); the totals fit while a (b, KV head) has at most
// 32767 visits (checked on the host).
__device__ __forceinline__ uint64_t scan_key(uint32_t cost) {
  return ((uint64_t)(cost & 0xFFFFFFu) << 35) | ((uint64_t)((cost >> 27) & 15u) << 17) | ((cost >> 24) & 7u);
}
__device__ __forceinline__ uint64_t key_cost(uint64_t k) { return k >> 35; }
__device__ __forceinline__ uint32_t key_units(uint64_t k) { return (uint32_t)(k >> 17) & 0x3FFFFu; }
__device__ __forceinline__ uint32_t key_items(uint64_t k) { return (uint32_t)k & 0x1FFFFu; }

// Where a plan writes: the wavefronts' splits and the item and unit lists.
struct PlanOut {
  ItemDesc *items;
  UnitDesc *units;
  int32_t *isplit, *usplit;
  int W, W1;       // wavefronts, wavefronts of the workgroups dispatched first
  uint64_t total;  // scan key of all visits
  double scale;    // owner_scale of the total cost
};

// Visit v, whose scan key interval starts at e: the splits of the wavefronts whose
// first visit it is, and its items and units.
__device__ __forceinline__ void place_visit(const PlanOut &o, const VisitDesc &d, int64_t v, int64_t nvis,
                                            uint64_t &e, int &prev) {
  const uint32_t c = d.cost & 0xFFFFFFu;
  const int own = midpoint_owner(o.W, o.W1, key_cost(e), c, o.scale);
  for (int ww = prev + 1; ww <= own; ++ww) {
    o.isplit[ww] = (int32_t)key_items(e);
    o.usplit[ww] = (int32_t)key_units(e);
  }
  visit_items(d, o.items + key_items(e), o.units + key_units(e));
  if (v == nvis - 1)
    for (int ww = own + 1; ww <= o.W; ++ww) {
      o.isplit[ww] = (int32_t)key_items(o.total);
      o.usplit[ww] = (int32_t)key_units(o.total);
    }
  prev = own;
  e += scan_key(d.cost);
}

// Owner of the visit before v0 (cost interval ending at e), -1 for v0 == 0.
__device__ __forceinline__ int prev_owner(const PlanOut &o, int64_t v0, uint64_t e, uint32_t prev_cost) {
  if (v0 == 0) return -1;
  const uint32_t c = prev_cost & 0xFFFFFFu;
  return midpoint_owner(o.W, o.W1, key_cost(e) - c, c, o.scale);
}

// A dense plan runs gridDim.y workgroups per (b, KV head): each scans the costs and
// counts of all visits (cheap) and expands only the visits of its slice of threads.
__device__ __forceinline__ bool own_slice() {
  return (int)((threadIdx.x * gridDim.y) / kPlanThreads) == (int)blockIdx.y;
}

// The bitmap of one-centroid runs of a dense plan (bit b: block b continues block
// b - 1's run), built by every thread for its visits [v0, v1) when any is set (a
// workgroup-uniform flag); null otherwise.
__device__ __forceinline__ const uint32_t *build_joins(const AttnParams &p, int64_t u, int64_t nblk, int64_t v0,
                                                       int64_t v1, bool any, uint32_t *joins) {
  if (!any) return nullptr;
  for (int64_t w = threadIdx.x; w < (nblk + 31) / 32; w += kPlanThreads) joins[w] = 0;
  __syncthreads();
  for (int64_t b = v0; b < v1 && b < nblk; ++b)
    if (mean_joins(p, u, b)) atomicOr(&joins[b >> 5], 1u << (b & 31));
  __syncthreads();
  return joins;
}

// Dense plan when every thread holds at most kPlanRegs visits: the visits stay in
// registers through the scan and the expansion.
constexpr int kPlanRegs = 4;
__device__ __forceinline__ void plan_dense_regs(const AttnParams &p, int64_t u, int64_t nblk, int64_t nvis,
                                                PlanOut o, uint64_t *sh, uint32_t *lastc, uint32_t *joins) {
  const int64_t per = (nvis + kPlanThreads - 1) / kPlanThreads;
  const int64_t v0 = threadIdx.x * per, v1 = v0 + per < nvis ? v0 + per : nvis;
  VisitDesc dv[kPlanRegs];
  bool any_mean = false;
#pragma unroll
  for (int j = 0; j < kPlanRegs; ++j)
    if (v0 + j < v1) {
      dv[j] = dense_visit(p, u, nblk, v0 + j, nullptr);
      any_mean |= dv[j].blk != 0xFFFFu && dv[j].level == GKV_MEAN;  // a block, not residual rows
    }
  // one-centroid runs, only when the cache holds one-centroid blocks
  if (const uint32_t *jn = build_joins(p, u, nblk, v0, v1, __syncthreads_or(any_mean), joins)) {
#pragma unroll
    for (int j = 0; j < kPlanRegs; ++j)
      if (v0 + j < v1 && dv[j].blk != 0xFFFFu && dv[j].level == GKV_MEAN && dv[j].valid) {
        mean_run_visit(p, u, dv[j].blk, jn, dv[j]);
        dv[j].cost = balance_cost(dv[j].level, dv[j].valid) | (visit_counts(dv[j].level, dv[j].valid) << 24);
      }
  }
  uint64_t mine = 0;
  uint32_t last = 0;
#pragma unroll
  for (int j = 0; j < kPlanRegs; ++j)
    if (v0 + j < v1) {
      mine += scan_key(dv[j].cost);
      last = dv[j].cost;
    }
  lastc[threadIdx.x] = last;  // read by the next thread after the scan's barriers
  uint64_t e = block_scan(mine, sh, o.total) - mine;
  o.scale = owner_scale(o.W, o.W1, key_cost(o.total));
  if (v0 >= v1 || !own_slice()) return;
  int prev = prev_owner(o, v0, e, v0 > 0 ? lastc[threadIdx.x - 1] : 0u);
#pragma unroll
  for (int j = 0; j < kPlanRegs; ++j)
    if (v0 + j < v1) place_visit(o, dv[j], v0 + j, nvis, e, prev);
}

__global__ void __launch_bounds__(kPlanThreads) plan_kernel(AttnParams p) {
  __shared__ uint64_t sh[3 * kPlanThreads / 64];  // block_scan: 6 x 16 32-bit words
  __shared__ uint32_t lastc[kPlanThreads];
  __shared__ uint32_t joins[32768 / 32];  // one-centroid run bits (nblk < 32768)
  __shared__ int s_same;
  if (p.cacheable) {  // the workspace may already hold this plan
    if (threadIdx.x == 0) {
      int same = 1;
#pragma unroll
      for (int i = 0; i < kTagWords; ++i) same &= p.tag[i] == p.key[i];
      s_same = same;
    }
    __syncthreads();
    if (s_same) return;
  }
  // the plan is rewritten: the tag is stale until an attention kernel validates it
  // (no workgroup of this launch can see this launch's key in it)
  if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) p.tag[0] = 0;
  const int64_t u = blockIdx.x;
  const int W = p.nsplit * kWaves;
  PlanOut o;
  o.items = (ItemDesc *)p.plan + u * p.icap;
  o.units = (UnitDesc *)p.units + u * p.ucap;
  o.isplit = p.split + u * (int64_t)(2 * (W + 1));
  o.usplit = o.isplit + (W + 1);
  o.W = W;
  o.W1 = p.fast * kWaves;
  const int64_t Tu = unit_T(p, u);
  const int64_t nblk = (Tu + P - 1) / P;
  // blocks 0..nblk-1, then the residual rows as exact pseudo-blocks; each thread
  // describes a contiguous run of visits
  const int64_t nvis = Tu ? nblk + (p.nres + P - 1) / P : 0;
  if (nvis == 0) {  // an empty or retired sequence: every wavefront's lists are empty
    if (blockIdx.y == 0)
      for (int ww = threadIdx.x; ww <= W; ww += kPlanThreads) o.isplit[ww] = o.usplit[ww] = 0;
    return;
  }
  const int64_t per = (nvis + kPlanThreads - 1) / kPlanThreads;
  if (per <= kPlanRegs) {
    plan_dense_regs(p, u, nblk, nvis, o, sh, lastc, joins);
    return;
  }
  const int64_t v0 = threadIdx.x * per, v1 = v0 + per < nvis ? v0 + per : nvis;
  bool any_mean = false;
  for (int64_t v = v0; v < v1 && v < nblk; ++v) any_mean |= p.level[u * p.nblk_cap + v] == GKV_MEAN;
  const uint32_t *jn = build_joins(p, u, nblk, v0, v1, __syncthreads_or(any_mean), joins);
  uint64_t mine = 0;
  for (int64_t v = v0; v < v1; ++v) mine += scan_key(dense_visit(p, u, nblk, v, jn).cost);
  uint64_t e = block_scan(mine, sh, o.total) - mine;
  o.scale = owner_scale(o.W, o.W1, key_cost(o.total));
  if (v0 >= v1 || !own_slice()) return;
  int prev = prev_owner(o, v0, e, v0 > 0 ? dense_visit(p, u, nblk, v0 - 1, jn).cost : 0u);
  for (int64_t v = v0; v < v1; ++v) place_visit(o, dense_visit(p, u, nblk, v, jn), v, nvis, e, prev);
}

}  // namespace

// ---------------------------------------------------------------- C ABI
// Workgroups per (b, KV head) for a call at context length T: enough wavefronts to
// fill the chip (2048 over all (b, KV head)), at most one per visit.
static int attn_nsplit(const gkv_cache *c, int32_t topk, int64_t T, bool layout) {
  const int64_t units = (int64_t)c->B * c->Hkv;
  int64_t waves;
  if (topk > 0) {
    // one read page per wavefront while the chip holds them (2048 wavefronts over all
    // (b, KV head)); never more pages per wavefront than its descriptor chunk holds
    waves = topk + 1;
    // the workspace is sized for a cache that may get residual rows (more wavefronts)
    const int ppw = quest_pages_per_wave(c->page ? c->page : 16, layout ? c->nres_cap > 0 : c->nres > 0);
    const int64_t room = 2048 / units, least = (topk + 1 + ppw - 1) / ppw;
    if (waves > room) waves = room > least ? room : least;
    if (waves > kMaxWaves) waves = kMaxWaves;  // still >= least (checked on the host)
    return (int)((waves + kWaves - 1) / kWaves);
  } else {
    const int64_t nvis = (T + P - 1) / P + (c->nres_cap + P - 1) / P;
    waves = 2048 / units;
    if (waves > nvis) waves = nvis;
  }
  if (waves < 1) waves = 1;
  if (waves > kMaxWaves) waves = kMaxWaves;
  return (int)((waves + kWaves - 1) / kWaves);
}

int gkv_device_cus() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 1;
  static int cache[64];
  if (!cache[dev]) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 1;
    cache[dev] = n;
  }
  return cache[dev];
}

// Workgroups of each (b, KV head) that are dispatched first.  With two attention
// workgroups per CU and the whole grid resident at once, workgroups 0 .. CUs-1 of the
// one-dimensional grid take the first slot of every CU; their wavefronts win the
// issue arbitration on their SIMDs (the older wavefront goes first) and run about a
// fifth faster, so the split gives them more work.  Otherwise all count the same.
static int attn_fast(int nsplit, int64_t units) {
  const int64_t cus = gkv_device_cus(), nb = (int64_t)nsplit * units;
  if (nb <= cus || nb > 2 * cus) return nsplit;
  return (int)(cus / units);
}

// Workspace layout, sized by the cache capacity so that it does not move as T grows:
// plan tag | partials | wavefront splits (items, units) | visit descriptors | item
// descriptors | unit descriptors (+512 B: the descriptor copies read whole 512-byte
// chunks).
struct AttnLayout {
  int64_t part, split, visits, plan, units, total, vcap, icap, ucap;
  int ncap;
};
static int64_t align256(int64_t x) { return (x + 255) & ~(int64_t)255; }
static AttnLayout attn_layout(const gkv_cache *c, int32_t topk) {
  AttnLayout L;
  const int64_t units = (int64_t)c->B * c->Hkv;
  const int G = c->Hq / c->Hkv;
  L.ncap = attn_nsplit(c, topk, (int64_t)c->nblk_cap * P, true);
  // a dense plan's lists; Compressed-Quest reads keep theirs in LDS
  L.vcap = topk > 0 ? 0 : (int64_t)c->nblk_cap + (c->nres_cap + P - 1) / P;
  L.icap = 4 * L.vcap;  // at most 4 items per visit
  L.ucap = 8 * L.vcap;  // at most 8 units per visit (an exact block)
  L.part = 256;  // the plan tag (kTagWords words) comes first
  L.split = L.part + align256(units * L.ncap * G * kPart * 4);
  L.visits = L.split + align256(units * 2 * ((int64_t)L.ncap * kWaves + 1) * 4);
  L.plan = L.visits + align256(units * L.vcap * (int64_t)sizeof(VisitDesc));
  L.units = L.plan + align256(units * L.icap * (int64_t)sizeof(ItemDesc));
  L.total = L.units + units * L.ucap * (int64_t)sizeof(UnitDesc) + 512;
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
    if (c->page != 16 && c->page != 32 && c->page != 64) return GKV_E_UNSUPPORTED;
  } else {
    topk = 0;
  }
  if (topk > 0) {  // the wavefronts that share the read pages, at most kMaxWaves
    const int ppw = quest_pages_per_wave(c->page, c->nres_cap > 0);
    if ((topk + 1 + ppw - 1) / ppw > kMaxWaves) return GKV_E_UNSUPPORTED;
  }
  const AttnLayout L = attn_layout(c, topk);
  if (L.vcap > 32767) return GKV_E_UNSUPPORTED;  // the dense plan's packed prefix sums
  if (ws_bytes < L.total) return GKV_E_WORKSPACE;
  p.q = q;
  p.level = c->level;
  p.koff = c->koff;
  p.voff = c->voff;
  p.arena = c->arena;
  p.res_mask = c->res_mask;
  p.res_off = c->res_off;
  p.res_rows = c->res_rows;
  p.pages = pages;
  p.seq_len = c->seq_len;
  p.tag = (uint64_t *)ws;
  p.part = (float *)((uint8_t *)ws + L.part);
  p.split = (int32_t *)((uint8_t *)ws + L.split);
  p.visits = (uint8_t *)ws + L.visits;
  p.plan = (uint8_t *)ws + L.plan;
  p.units = (uint8_t *)ws + L.units;
  p.vcap = L.vcap;
  p.icap = L.icap;
  p.ucap = L.ucap;
  p.T = c->T;
  p.nblk_cap = c->nblk_cap;
  p.Hkv = c->Hkv;
  p.G = c->Hq / c->Hkv;
  p.nres = c->nres;
  p.nrb_cap = (c->nres_cap + P - 1) / P;
  p.topk = topk;
  p.page = c->page ? c->page : 16;
  p.cert = c->cert;
  p.bound = nullptr;
  p.nsplit = attn_nsplit(c, topk, c->T, false);
  p.fast = attn_fast(p.nsplit, (int64_t)c->B * c->Hkv);
  p.sl2 = 1.4426950408889634f / sqrtf((float)D);
  // the key of the planned state: a dense plan depends on the tables (version stamp
  // and addresses), the block count, the residual count and the split
  p.cacheable = !pages && c->version != 0;
  const uint64_t key[kTagWords] = {c->version,
                                   (uint64_t)((c->T + P - 1) / P),
                                   (uint64_t)(uint32_t)c->nres | ((uint64_t)(uint32_t)p.nsplit << 32),
                                   (uint64_t)(uint32_t)p.fast | ((uint64_t)(uint32_t)c->nblk_cap << 32),
                                   (uint64_t)(uintptr_t)c->level,
                                   (uint64_t)(uintptr_t)c->koff,
                                   (uint64_t)(uintptr_t)c->voff,
                                   (uint64_t)(uintptr_t)c->arena,
                                   (uint64_t)(uintptr_t)c->res_mask,
                                   (uint64_t)(uintptr_t)c->res_rows,
                                   (uint64_t)(uint32_t)c->B | ((uint64_t)(uint32_t)c->Hkv << 32),
                                   kTagMagic};
  for (int i = 0; i < kTagWords; ++i) p.key[i] = key[i];
  return GKV_OK;
}

static void launch_plan(const AttnParams &p, const gkv_cache *c, hipStream_t s) {
  if (p.pages) return;  // Compressed-Quest reads list their pages in the attention kernel
  // one workgroup per 256 visits of a (b, KV head), at most 8
  const int64_t nvis = (p.T + P - 1) / P + (p.nres + P - 1) / P;
  const int slices = (int)(nvis / 256 < 1 ? 1 : (nvis / 256 > 8 ? 8 : nvis / 256));
  hipLaunchKernelGGL(plan_kernel, dim3(c->B * c->Hkv, slices), dim3(kPlanThreads), 0, s, p);
}
static void launch_partials(const AttnParams &p, const gkv_cache *c, hipStream_t s) {
  const size_t lds = (size_t)kWaves * kWaveLds + 16 * kQRow;  // rings also hold the merge buffers
  const dim3 grid(p.nsplit * c->Hkv * c->B);
  // the certificate sums, per-token value groups and Compressed-Quest lists are
  // separate instantiations: the plain dense decode keeps its registers and code
  const bool pack = p.G <= 8, cert = p.bound != nullptr, vtok = c->v_per_token != 0;
  const bool quest = p.pages != nullptr && !cert;  // the certificate is a dense read
  const dim3 blk(kThreads);
#define GKV_ATTN(a, b, c2, d) hipLaunchKernelGGL((attn_kernel<a, b, c2, d>), grid, blk, lds, s, p)
  if (quest) {
    if (vtok) {
      if (pack) GKV_ATTN(true, false, true, true);
      else GKV_ATTN(false, false, true, true);
    } else {
      if (pack) GKV_ATTN(true, false, false, true);
      else GKV_ATTN(false, false, false, true);
    }
  } else if (vtok) {
    if (cert) {
      if (pack) GKV_ATTN(true, true, true, false);
      else GKV_ATTN(false, true, true, false);
    } else {
      if (pack) GKV_ATTN(true, false, true, false);
      else GKV_ATTN(false, false, true, false);
    }
  } else {
    if (cert) {
      if (pack) GKV_ATTN(true, true, false, false);
      else GKV_ATTN(false, true, false, false);
    } else {
      if (pack) GKV_ATTN(true, false, false, false);
      else GKV_ATTN(false, false, false, false);
    }
  }
#undef GKV_ATTN
}
static void launch_merge(const AttnParams &p, const gkv_cache *c, float *out, hipStream_t s) {
  hipLaunchKernelGGL(merge_kernel, dim3(p.G, c->Hkv * c->B), dim3(D), 0, s, (const float *)p.part, out, p.nsplit,
                     p.G, p.bound, p.cert, c->nblk_cap, (int)((c->T + P - 1) / P), (const int64_t *)c->seq_len,
                     c->Hkv);
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

extern "C" gkv_status gkv_graded_decode_attn_bound(const uint16_t *q, const gkv_cache *c, float *out, float *bound,
                                                   void *ws, int64_t ws_bytes, void *stream) {
  if (!q || !out || !bound || !c || !c->cert) return GKV_E_ARG;
  AttnParams p;
  const gkv_status st = attn_setup(q, c, nullptr, 0, ws, ws_bytes, p);
  if (st) return st;
  p.bound = bound;
  const hipStream_t s = (hipStream_t)stream;
  launch_plan(p, c, s);
  launch_partials(p, c, s);
  launch_merge(p, c, out, s);
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

// ---------------------------------------------------------------- no-allocation entry point
// For callers that cannot allocate (graph capture, fixed serving loops): the
// workspace is a file-scope device array that each GPU holds for the life of the
// process.  Host code never passes `scratch` itself (in host code its name stands for
// a host-side symbol, not a device address); the device address comes from
// hipGetSymbolAddress, taken once per device with that device current.
constexpr int64_t kScratchBytes = 32ll << 20;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

static std::mutex g_scratch_mu;
static void *g_scratch_ptr[64];

static gkv_status scratch_address(void **ptr) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return GKV_E_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return GKV_E_HIP;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return GKV_OK;
}

extern "C" int64_t gkv_noalloc_scratch_bytes() { return kScratchBytes; }

extern "C" gkv_status gkv_graded_decode_attn_noalloc(const uint16_t *q, const gkv_cache *c, const int32_t *pages,
                                                     int32_t topk, float *out, void *stream) {
  if (!q || !out) return GKV_E_ARG;
  const gkv_status st = gkv_validate_cache(c);
  if (st) return st;
  if (pages && topk <= 0) return GKV_E_ARG;
  if (attn_layout(c, pages ? topk : 0).total > kScratchBytes) return GKV_E_WORKSPACE;  // before any HIP call
  void *ws = nullptr;
  const gkv_status sa = scratch_address(&ws);
  if (sa) return sa;
  return gkv_graded_decode_attn(q, c, pages, topk, out, ws, kScratchBytes, stream);
}
