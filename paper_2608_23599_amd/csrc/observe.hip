// Causal attention-mass observer (section 3.1, Eq. 1-2, GQA aggregation, EMA) and
// the closed-form level allocation (section 3.3, Eq. allocation and b*).
//
// Observer, per (sequence b, KV head h), with R = n_obs * G query rows (row
// r = i * G + g is query head h * G + g at prompt position T - n_obs + i):
//   obs_logit_kernel  MFMA logits of every row against every key, one log-sum-exp
//                     per (block, row) over the block's visible keys (log2 units),
//                     and per (row, workgroup chunk of blocks) a running max and sum;
//   obs_row_kernel    per row the log-sum-exp over all chunks;
//   obs_mass_kernel   per block the mean over rows of exp2(lse_block - lse_row),
//                     blended into the mass with the EMA weight.
// Allocation: query_norm_kernel (largest query norm of each group, fp64) and
// alloc_kernel (key range of each block, then the threshold form of b*).
#include <hip/hip_runtime.h>

#include "gkv_internal.h"

#pragma clang fp contract(off)

using namespace gkv;

namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float f16x __attribute__((ext_vector_type(16)));

union H8 {
  half8 h;
  uint4 v;
};

constexpr int kObsWaves = 8;
constexpr int kObsThreads = 64 * kObsWaves;
constexpr int kObsBlocksPerWave = 128 / kObsWaves;
constexpr int kObsChunk = kObsWaves * kObsBlocksPerWave;  // blocks per workgroup
constexpr int kMaxRows = 512;
constexpr float kNegInf = -__builtin_huge_valf();
// A running sum may grow to this before its reference is moved to the block's maximum.
constexpr float kSumLimit = 0x1p64f;

__device__ __forceinline__ f16x mfma32x32(half8 a, half8 b, f16x c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

// The logits use 32 x 32 x 16 MFMAs: A = 32 keys x 16 channels, B = 16 channels x
// 32 query rows.  Lane l = 32 hf + j (j = l & 31, hf = l >> 5) supplies A row j
// and B column j, channels 16 c + 8 hf .. + 7 of channel chunk c (0..7), and holds
// accumulator element e of column j = query row j, key 8 (e >> 2) + 4 hf + (e & 3)
// of the 32-key half kt of the block.
//
// Query rows in LDS in operand order: tile rt (32 rows), chunk c, lane l -> 16 bytes
// at ((rt * 8 + c) * 64 + l) * 16, so that the 64 lanes of one read are contiguous.
__device__ __forceinline__ uint32_t qoff(int rt, int c, int l) { return (uint32_t)((rt * 8 + c) * 64 + l) * 16u; }

// This lane's key operands of one block (zero beyond T).  One load instruction takes
// 32 bytes of each of 32 key rows, so the four loads that share a 128-byte line rely
// on finding it in the caches: these are plain loads (with the nontemporal hint, lines
// left the caches early and the bytes fetched from HBM grew by a quarter).
__device__ __forceinline__ void load_keys(H8 (&a)[2][8], const uint16_t *kb, int64_t T, int blk, int j, int hf) {
#pragma unroll
  for (int kt = 0; kt < 2; ++kt) {
    const int64_t key = (int64_t)blk * P + 32 * kt + j;
    const int64_t kk = key < T ? key : T - 1;  // in bounds; replaced by zero below
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      const uint4 v = *(const uint4 *)(kb + kk * D + 16 * c + 8 * hf);
      a[kt][c].v = key < T ? v : make_uint4(0, 0, 0, 0);
    }
  }
}

// Logits of one (block, 32-row tile): acc[kt] = keys of half kt against the tile's rows;
// qt = this lane's operand of the tile's chunk 0 in LDS.
__device__ __forceinline__ void tile_logits(f16x (&acc)[2], const H8 (&a)[2][8], const uint8_t *qt) {
#pragma unroll
  for (int kt = 0; kt < 2; ++kt) acc[kt] = f16x{};
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    H8 qb;
    qb.v = *(const uint4 *)(qt + c * 1024);
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) acc[kt] = mfma32x32(a[kt][c].h, qb.h, acc[kt]);
  }
}

// This lane's query operands of one tile (qt = its operand of the tile's chunk 0).
__device__ __forceinline__ void load_q(H8 (&qb)[8], const uint8_t *qt) {
#pragma unroll
  for (int c = 0; c < 8; ++c) qb[c].v = *(const uint4 *)(qt + c * 1024);
}

// Logits of one (block, 32-row tile) from query operands already in registers.
__device__ __forceinline__ void tile_logits_q(f16x (&acc)[2], const H8 (&a)[2][8], const H8 (&qb)[8]) {
#pragma unroll
  for (int kt = 0; kt < 2; ++kt) acc[kt] = f16x{};
#pragma unroll
  for (int c = 0; c < 8; ++c)
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) acc[kt] = mfma32x32(a[kt][c].h, qb[c].h, acc[kt]);
}

// The two lanes of a row (l and l ^ 32) exchange and combine a value.
__device__ __forceinline__ float row_sum2(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(a[0]) + __uint_as_float(a[1]);
}
__device__ __forceinline__ float row_max2(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
}

// Key of accumulator element e of half kt for this lane (relative to the block start).
__device__ __forceinline__ int elem_key(int kt, int e, int hf) { return 32 * kt + 8 * (e >> 2) + 4 * hf + (e & 3); }

// sum over the row's visible keys of exp2(s * sl2 - ref); with MASKED only the keys
// key0 + k <= last (and < T) count.
template <bool MASKED>
__device__ __forceinline__ float tile_sum(const f16x (&acc)[2], float sl2, float ref, int64_t key0, int hf,
                                          int64_t last, int64_t T) {
  float x[32];
#pragma unroll
  for (int kt = 0; kt < 2; ++kt)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      float v = __builtin_amdgcn_exp2f(fmaf(acc[kt][e], sl2, -ref));
      if (MASKED) {
        const int64_t key = key0 + elem_key(kt, e, hf);
        v = key <= last && key < T ? v : 0.f;
      }
      x[16 * kt + e] = v;
    }
#pragma unroll
  for (int w = 16; w >= 1; w >>= 1)  // pairwise: a chain of depth 5
#pragma unroll
    for (int i = 0; i < w; ++i) x[i] += x[i + w];
  return row_sum2(x[0]);
}

template <bool MASKED>
__device__ __forceinline__ float tile_max(const f16x (&acc)[2], float sl2, int64_t key0, int hf, int64_t last,
                                          int64_t T) {
  float m = kNegInf;
#pragma unroll
  for (int kt = 0; kt < 2; ++kt)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int64_t key = key0 + elem_key(kt, e, hf);
      if (!MASKED || (key <= last && key < T)) m = fmaxf(m, acc[kt][e] * sl2);
    }
  return row_max2(m);
}

// Merges a block's log-sum-exp v (-inf: no visible key) into the running pair r of its
// row, moving the reference to the larger of the two; written with selects only.
__device__ __forceinline__ void merge_lse(float v, float2 &r) {
  const bool valid = v > kNegInf;
  const bool first = valid && r.y == 0.f;  // the row's first visible block
  const bool up = v > r.x;
  const float e = __builtin_amdgcn_exp2f(-__builtin_fabsf(v - r.x));  // 0 when v = -inf
  const float y = up ? fmaf(r.y, e, 1.f) : r.y + e;
  r.y = first ? 1.f : (valid ? y : r.y);
  r.x = first || (valid && up) ? v : r.x;
}

// General path for one (block, tile): the block's log-sum-exp against its own maximum
// (-inf when the row sees none of its keys), merged into the running pair r.
template <bool MASKED>
__device__ __forceinline__ float tile_lse_general(const f16x (&acc)[2], float sl2, int64_t key0, int hf,
                                                  int64_t last, int64_t T, float2 &r) {
  const float ref = tile_max<MASKED>(acc, sl2, key0, hf, last, T);
  const float ref0 = ref == kNegInf ? 0.f : ref;  // keeps the sum finite (it is 0 then)
  const float sum = tile_sum<MASKED>(acc, sl2, ref0, key0, hf, last, T);
  const float v = ref == kNegInf ? kNegInf : ref + __builtin_amdgcn_logf(sum);
  merge_lse(v, r);
  return v;
}

// One unmasked tile: sum_j exp2(x_j - ref) against the row's running reference
// ref = r.x, so that the block adds exactly that sum to r.y and its log-sum-exp is
// ref + log2(sum).  Every row starts at (ref, sum) = (0, 0).  The wavefront takes the
// general path (uniformly) when some row's sum exceeds kSumLimit, or is below
// 1 / kSumLimit while the row has no earlier block at or above the reference (so that
// no block of the row can lose its precision).  The log-sum-exp goes to lse[0] and the
// running pair to st[0].
__device__ __forceinline__ void finish_tile(const f16x (&acc)[2], float sl2, int64_t key0, int hf, int64_t T,
                                            float2 r, float *lse, float2 *st) {
  const float sum = tile_sum<false>(acc, sl2, r.x, key0, hf, 0, T);
  const bool ok = (sum <= kSumLimit) & ((sum >= 1.f / kSumLimit) | (r.y >= 1.f));
  float v;
  if (__builtin_expect(__builtin_amdgcn_ballot_w64(!ok) != 0, 0)) {
    v = tile_lse_general<false>(acc, sl2, key0, hf, 0, T, r);
  } else {
    r.y += sum;
    v = r.x + __builtin_amdgcn_logf(sum);  // -inf when every term is below fp32 range
  }
  lse[0] = v;
  st[0] = r;
}

// Logits and per-block log-sum-exp.  Each wavefront takes kObsBlocksPerWave blocks
// and, per block, every 32-row tile of the group's queries: 16 MFMAs give the 64 x 32
// logits, then sum_j exp2(x_j - ref) over the block's visible keys with ref the row's
// running reference (kept in LDS per wavefront and row with the running sum of
// exp2(lse - ref) over the wavefront's blocks).  While the vector ALUs work on tile
// rt, the MFMAs of tile rt + 1 are issued in the same basic block, so the matrix cores
// and the vector ALUs overlap.  The running pairs are merged over the workgroup into
// one (max, sum) per (row, workgroup chunk).
__global__ void __launch_bounds__(kObsThreads) obs_logit_kernel(const uint16_t *__restrict__ q_obs,
                                                                const uint16_t *__restrict__ k_src, int n_obs,
                                                                int G, int Hkv, int64_t T, int nblk, int Rpad,
                                                                float sl2, float *__restrict__ lse,
                                                                float2 *__restrict__ part) {
  extern __shared__ __align__(16) uint8_t qs[];
  float2 *stats = (float2 *)(qs + Rpad * 256);  // [kObsWaves][Rpad] running (reference, sum)
  const int h = blockIdx.y, b = blockIdx.z;
  const int64_t u = (int64_t)b * Hkv + h;
  const int R = n_obs * G, Hq = Hkv * G;
  for (int i = threadIdx.x; i < Rpad * 16; i += kObsThreads) {
    const int r = i >> 4, cc = i & 15;  // row, 8-channel chunk
    uint4 v = make_uint4(0, 0, 0, 0);
    if (r < R) {
      const int qi = r / G, g = r - qi * G;
      v = *(const uint4 *)(q_obs + (((int64_t)b * n_obs + qi) * Hq + h * G + g) * D + 8 * cc);
    }
    *(uint4 *)(qs + qoff(r >> 5, cc >> 1, (r & 31) + 32 * (cc & 1))) = v;
  }
  for (int i = threadIdx.x; i < kObsWaves * Rpad; i += kObsThreads) stats[i] = make_float2(0.f, 0.f);
  __syncthreads();
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, j = lane & 31, hf = lane >> 5;
  float2 *wst = stats + wv * Rpad + j;
  const uint16_t *kb = k_src + u * T * D;
  const int64_t first_masked = T - n_obs + 1;  // keys at or beyond this are hidden from some row
  const int blk0 = blockIdx.x * kObsChunk + wv * kObsBlocksPerWave;
  const int nb = blk0 >= nblk ? 0 : (nblk - blk0 < kObsBlocksPerWave ? nblk - blk0 : kObsBlocksPerWave);
  const int nt = Rpad / 32;
  const uint8_t *qlane = qs + lane * 16;
  H8 a[2][8];
  if (nb > 0) load_keys(a, kb, T, blk0, j, hf);
  for (int k = 0; k < nb; ++k) {
    // The keys of block blk are in flight: they were issued when the previous block's
    // last MFMAs were out.  (Touching the next block's lines a block ahead, to warm the
    // L2, made the fetched bytes grow by half: the lines a CU's waves touch ahead fill
    // its XCD's L2 and leave before they are read.)
    const int blk = blk0 + k;
    const int64_t key0 = (int64_t)blk * P;
    float *lse_blk = lse + (u * nblk + blk) * Rpad + j;
    f16x cur[2];
    tile_logits(cur, a, qlane);
    if (key0 + P > first_masked) {  // uniform: some row does not see every key of the block
      for (int rt = 0; rt < nt; ++rt) {
        if (rt > 0) tile_logits(cur, a, qlane + rt * 8192);
        const int row = 32 * rt + j;
        const int64_t last = T - n_obs + row / G;  // the last key this row sees
        float2 r = wst[32 * rt];
        const float v = tile_lse_general<true>(cur, sl2, key0, hf, last, T, r);
        lse_blk[32 * rt] = v;
        wst[32 * rt] = r;
      }
      if (k + 1 < nb) load_keys(a, kb, T, blk + 1, j, hf);
      continue;
    }
    // Unmasked: software-pipelined over the row tiles, unrolled by two so that the two
    // accumulator sets trade roles (tile rt in one set while the MFMAs of tile rt + 1
    // fill the other) without copies, which would wait for the MFMAs to drain.  The
    // query operands of a tile are read from LDS one tile ahead of its MFMAs.
    H8 qb[8];
    load_q(qb, qlane + (nt > 1 ? 8192 : 0));  // tile 1 (tile 0 is in cur)
    f16x alt[2];
    float2 r = wst[0];
    int rt = 0;
    for (; rt + 2 < nt; rt += 2) {
      tile_logits_q(alt, a, qb);
      load_q(qb, qlane + (rt + 2) * 8192);
      float2 r_next = wst[32 * (rt + 1)];
      finish_tile(cur, sl2, key0, hf, T, r, lse_blk + 32 * rt, wst + 32 * rt);
      r = r_next;
      tile_logits_q(cur, a, qb);
      load_q(qb, qlane + (rt + 3 < nt ? rt + 3 : nt - 1) * 8192);
      r_next = wst[32 * (rt + 2)];
      finish_tile(alt, sl2, key0, hf, T, r, lse_blk + 32 * (rt + 1), wst + 32 * (rt + 1));
      r = r_next;
    }
    if (rt + 1 < nt) {  // two tiles left: rt in cur, rt + 1 (operands in qb) still to compute
      tile_logits_q(alt, a, qb);
      const float2 r_next = wst[32 * (rt + 1)];
      if (k + 1 < nb) load_keys(a, kb, T, blk + 1, j, hf);  // the block's MFMAs are all issued
      finish_tile(cur, sl2, key0, hf, T, r, lse_blk + 32 * rt, wst + 32 * rt);
      r = r_next;
      finish_tile(alt, sl2, key0, hf, T, r, lse_blk + 32 * (rt + 1), wst + 32 * (rt + 1));
    } else {  // one tile left, in cur
      if (k + 1 < nb) load_keys(a, kb, T, blk + 1, j, hf);
      finish_tile(cur, sl2, key0, hf, T, r, lse_blk + 32 * rt, wst + 32 * rt);
    }
  }
  __syncthreads();
  // merge the wavefronts' running sums: one (max, sum) per (row, chunk)
  for (int r = threadIdx.x; r < R; r += kObsThreads) {
    float m = kNegInf;  // pairs with a zero sum hold no block
    for (int w = 0; w < kObsWaves; ++w) {
      const float2 p = stats[w * Rpad + r];
      if (p.y > 0.f) m = fmaxf(m, p.x);
    }
    float sm = 0.f;
    if (m != kNegInf)
      for (int w = 0; w < kObsWaves; ++w) {
        const float2 p = stats[w * Rpad + r];
        if (p.y > 0.f) sm += p.y * __builtin_amdgcn_exp2f(p.x - m);
      }
    part[(u * gridDim.x + blockIdx.x) * Rpad + r] = make_float2(m, sm);
  }
}

// One wavefront per row: the row's log-sum-exp over the chunks' (max, sum) pairs.
__global__ void __launch_bounds__(256) obs_row_kernel(const float2 *__restrict__ part, int R, int Rpad, int nslice,
                                                      int Hkv, float *__restrict__ row_lse) {
  const int lane = threadIdx.x & 63, r = blockIdx.x * 4 + (threadIdx.x >> 6), h = blockIdx.y, b = blockIdx.z;
  if (r >= R) return;
  const int64_t u = (int64_t)b * Hkv + h;
  float m = kNegInf, s = 0.f;
  for (int sl = lane; sl < nslice; sl += 64) {
    const float2 p = part[(u * nslice + sl) * Rpad + r];
    if (p.x == kNegInf) continue;
    if (p.x > m) {
      s = s * __builtin_amdgcn_exp2f(m - p.x) + p.y;
      m = p.x;
    } else {
      s += p.y * __builtin_amdgcn_exp2f(p.x - m);
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const float m2 = __shfl_xor(m, o), s2 = __shfl_xor(s, o);
    const float mm = fmaxf(m, m2);
    s = (m == kNegInf ? 0.f : s * __builtin_amdgcn_exp2f(m - mm)) + (m2 == kNegInf ? 0.f : s2 * __builtin_amdgcn_exp2f(m2 - mm));
    m = mm;
  }
  if (lane == 0) row_lse[u * Rpad + r] = m + __builtin_amdgcn_logf(s);  // every row sees key 0
}

// Per block: the mean over rows of the block's share exp2(lse_block - lse_row) of each
// row, blended into the mass with the EMA weight.  A workgroup takes 16 consecutive
// blocks of one (b, h), four per wavefront; lane l holds rows 4 l .. 4 l + 3 and
// 256 + 4 l .. + 3 (Rpad <= 512), so that one block is two 16-byte loads per lane, and
// every load of the wavefront is issued before the first is used.
constexpr int kMassWaveBlocks = 4;
constexpr int kMassBlocks = 4 * kMassWaveBlocks;  // per workgroup

__global__ void __launch_bounds__(256) obs_mass_kernel(const float *__restrict__ lse,
                                                       const float *__restrict__ row_lse, int R, int Rpad,
                                                       int nblk, int Hkv, float alpha, float *__restrict__ mass) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int h = blockIdx.y, b = blockIdx.z;
  const int64_t u = (int64_t)b * Hkv + h;
  const int blk0 = (blockIdx.x * 4 + wv) * kMassWaveBlocks;
  if (blk0 >= nblk) return;
  float rl[8];
  bool row_ok[8];
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const int r0 = 256 * c + 4 * lane;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      row_ok[4 * c + i] = r0 + i < R;
      rl[4 * c + i] = r0 + i < Rpad ? row_lse[u * Rpad + r0 + i] : 0.f;
    }
  }
  float4 v[kMassWaveBlocks][2];
#pragma unroll
  for (int k = 0; k < kMassWaveBlocks; ++k)
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int r0 = 256 * c + 4 * lane;  // r0 < Rpad implies r0 + 3 < Rpad (Rpad % 32 == 0)
      v[k][c] = blk0 + k < nblk && r0 < Rpad ? *(const float4 *)(lse + (u * nblk + blk0 + k) * Rpad + r0)
                                             : make_float4(kNegInf, kNegInf, kNegInf, kNegInf);
    }
#pragma unroll
  for (int k = 0; k < kMassWaveBlocks; ++k) {
    const float x[8] = {v[k][0].x, v[k][0].y, v[k][0].z, v[k][0].w, v[k][1].x, v[k][1].y, v[k][1].z, v[k][1].w};
    float acc = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (row_ok[i] && x[i] != kNegInf) acc += __builtin_amdgcn_exp2f(x[i] - rl[i]);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) acc += __shfl_xor(acc, o);
    if (lane == 0 && blk0 + k < nblk) {
      const float m = acc / (float)R;
      float *dst = mass + u * nblk + blk0 + k;
      *dst = alpha == 1.f ? m : (1.f - alpha) * *dst + alpha * m;
    }
  }
}

// Largest ||q|| over the group's observed queries, fp64, channel-ascending sums.
__global__ void __launch_bounds__(256) query_norm_kernel(const uint16_t *__restrict__ q_obs, int n_obs, int G,
                                                         int Hkv, double *__restrict__ qn) {
  __shared__ double best[256];
  const int h = blockIdx.x, b = blockIdx.y;
  const int R = n_obs * G, Hq = Hkv * G;
  double mx = 0.0;
  for (int r = threadIdx.x; r < R; r += 256) {
    const int qi = r / G, g = r - qi * G;
    const uint16_t *q = q_obs + (((int64_t)b * n_obs + qi) * Hq + h * G + g) * D;
    double acc = 0.0;
    for (int d = 0; d < D; ++d) {
      const double x = (double)__builtin_bit_cast(_Float16, q[d]);
      acc = acc + x * x;
    }
    const double n = __builtin_sqrt(acc);
    mx = n > mx ? n : mx;
  }
  best[threadIdx.x] = mx;
  __syncthreads();
  if (threadIdx.x == 0) {
    double m = 0.0;
    for (int i = 0; i < 256; ++i) m = best[i] > m ? best[i] : m;
    qn[(int64_t)b * Hkv + h] = m;
  }
}

// Level of one block: key range, then x = c ||q|| e N m / (2 tau) against 2^L - 1.
__global__ void __launch_bounds__(D) alloc_kernel(const uint16_t *__restrict__ k_src, const float *__restrict__ mass,
                                                  const double *__restrict__ qn, int Hkv, int64_t T, int nblk,
                                                  double c, double tau, int window, int rounding,
                                                  int8_t *__restrict__ levels) {
  __shared__ double rng[D];
  const int blk = blockIdx.x, h = blockIdx.y, b = blockIdx.z, d = threadIdx.x;
  const int64_t u = (int64_t)b * Hkv + h;
  const bool exact = blk >= nblk - window || (int64_t)(blk + 1) * P > T;
  if (exact) {
    if (d == 0) levels[u * nblk + blk] = GKV_EXACT;
    return;
  }
  // thread d reads channels 8 (d % 16) .. +7 of rows d / 16, d / 16 + 8, .. (eight
  // 16-byte streaming loads, each row of the block read by 16 neighbouring lanes), then
  // the eight row groups' minima and maxima meet in LDS: min and max are exact in fp16
  const int cg = d & 15, rg = d >> 4;
  const _Float16 *kb = (const _Float16 *)k_src + (u * T + (int64_t)blk * P + rg) * D + 8 * cg;
  half8 v[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) v[j] = __builtin_nontemporal_load((const half8 *)(kb + (int64_t)8 * j * D));
  half8 mn = v[0], mx = v[0];
#pragma unroll
  for (int j = 1; j < 8; ++j) {
    mn = __builtin_elementwise_min(mn, v[j]);
    mx = __builtin_elementwise_max(mx, v[j]);
  }
  __shared__ half8 smn[8][16], smx[8][16];
  smn[rg][cg] = mn;
  smx[rg][cg] = mx;
  __syncthreads();
  {
    const int c = d >> 3, e = d & 7;  // channel d = 8 c + e
    _Float16 lo = smn[0][c][e], hi = smx[0][c][e];
#pragma unroll
    for (int r = 1; r < 8; ++r) {
      lo = smn[r][c][e] < lo ? smn[r][c][e] : lo;
      hi = smx[r][c][e] > hi ? smx[r][c][e] : hi;
    }
    // the largest channel range (exact in fp64, and max needs no order): within each
    // wavefront by shuffles, then over the two wavefronts
    double r = (double)hi - (double)lo;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      const double t = __shfl_xor(r, o);
      r = t > r ? t : r;
    }
    if ((d & 63) == 0) rng[d >> 6] = r;
  }
  __syncthreads();
  if (d == 0) {
    double e = rng[0];
    for (int i = 1; i < D / 64; ++i) e = rng[i] > e ? rng[i] : e;
    double x = c * qn[u];
    x = x * e;
    x = x * (double)nblk;
    x = x * (double)mass[u * nblk + blk];
    x = x / (2.0 * tau);
    // b* <= n is x <= 2^n - 1: rounded up, level L takes b* <= L; rounded to the
    // nearest level (ties up), int4 takes b* <= 5 and int8 b* <= 11
    const double t4 = rounding ? 31.0 : 15.0, t8 = rounding ? 2047.0 : 255.0;
    int8_t lv = GKV_EXACT;
    if (x <= 1.0) lv = GKV_CENTROID;
    else if (x <= 3.0) lv = GKV_INT2;
    else if (x <= t4) lv = GKV_INT4;
    else if (x <= t8) lv = GKV_INT8;
    levels[u * nblk + blk] = lv;
  }
}

int rows_padded(int R) { return (R + 31) / 32 * 32; }
int64_t align256(int64_t x) { return (x + 255) & ~(int64_t)255; }

struct ObsLayout {
  int nblk, R, Rpad, nslice;
  int64_t lse, part, rows, total;
};

ObsLayout obs_layout(int B, int Hkv, int Hq, int64_t T, int n_obs) {
  ObsLayout L;
  const int64_t units = (int64_t)B * Hkv;
  L.nblk = (int)((T + P - 1) / P);
  L.R = n_obs * (Hq / Hkv);
  L.Rpad = rows_padded(L.R);
  L.nslice = (L.nblk + kObsChunk - 1) / kObsChunk;
  L.lse = 0;
  L.part = align256(units * L.nblk * L.Rpad * 4);
  L.rows = L.part + align256(units * L.nslice * L.Rpad * 8);
  L.total = L.rows + align256(units * L.Rpad * 4);
  return L;
}

gkv_status obs_check(int B, int Hkv, int Hq, int64_t T, int n_obs) {
  if (B <= 0 || Hkv <= 0 || Hq <= 0 || Hq % Hkv) return GKV_E_SHAPE;
  const int G = Hq / Hkv;
  if (G < 1 || G > 16) return GKV_E_SHAPE;
  if (T <= 0 || n_obs < 1 || n_obs > T) return GKV_E_SHAPE;
  if ((int64_t)n_obs * G > kMaxRows) return GKV_E_UNSUPPORTED;
  if ((T + P - 1) / P > (1ll << 24)) return GKV_E_UNSUPPORTED;
  return GKV_OK;
}

}  // namespace

extern "C" int64_t gkv_observe_ws_bytes(int32_t B, int32_t Hkv, int32_t Hq, int64_t T, int32_t n_obs) {
  if (obs_check(B, Hkv, Hq, T, n_obs)) return -1;
  return obs_layout(B, Hkv, Hq, T, n_obs).total;
}

extern "C" gkv_status gkv_observe_mass(const uint16_t *q_obs, int32_t n_obs, const uint16_t *k_src, int32_t B,
                                       int32_t Hkv, int32_t Hq, int64_t T, float alpha, float *mass, void *ws,
                                       int64_t ws_bytes, void *stream) {
  gkv_status st = obs_check(B, Hkv, Hq, T, n_obs);
  if (st) return st;
  if (!q_obs || !k_src || !mass || !ws) return GKV_E_ARG;
  if (!(alpha > 0.f && alpha <= 1.f)) return GKV_E_ARG;
  const ObsLayout L = obs_layout(B, Hkv, Hq, T, n_obs);
  if (ws_bytes < L.total) return GKV_E_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  uint8_t *w = (uint8_t *)ws;
  float *lse = (float *)(w + L.lse);
  float2 *part = (float2 *)(w + L.part);
  float *rows = (float *)(w + L.rows);
  const int G = Hq / Hkv;
  const float sl2 = 1.4426950408889634f / sqrtf((float)D);
  hipLaunchKernelGGL(obs_logit_kernel, dim3(L.nslice, Hkv, B), dim3(kObsThreads), L.Rpad * (256 + 8 * kObsWaves), s, q_obs,
                     k_src, n_obs, G, Hkv, T, L.nblk, L.Rpad, sl2, lse, part);
  hipLaunchKernelGGL(obs_row_kernel, dim3((L.R + 3) / 4, Hkv, B), dim3(256), 0, s, part, L.R, L.Rpad, L.nslice, Hkv,
                     rows);
  hipLaunchKernelGGL(obs_mass_kernel, dim3((L.nblk + kMassBlocks - 1) / kMassBlocks, Hkv, B), dim3(256), 0, s, lse,
                     rows, L.R, L.Rpad, L.nblk, Hkv, alpha, mass);
  return hipGetLastError() == hipSuccess ? GKV_OK : GKV_E_HIP;
}

extern "C" gkv_status gkv_query_norms(const uint16_t *q_obs, int32_t n_obs, int32_t B, int32_t Hkv, int32_t Hq,
                                      double *qn, void *stream) {
  if (B <= 0 || Hkv <= 0 || Hq <= 0 || Hq % Hkv || Hq / Hkv > 16 || n_obs < 1) return GKV_E_SHAPE;
  if (!q_obs || !qn) return GKV_E_ARG;
  hipLaunchKernelGGL(query_norm_kernel, dim3(Hkv, B), dim3(256), 0, (hipStream_t)stream, q_obs, n_obs, Hq / Hkv,
                     Hkv, qn);
  return hipGetLastError() == hipSuccess ? GKV_OK : GKV_E_HIP;
}

extern "C" gkv_status gkv_allocate_levels(const uint16_t *k_src, const float *mass, const double *qn, int32_t B,
                                          int32_t Hkv, int64_t T, double c, double tau, int32_t window,
                                          int32_t rounding, int8_t *levels, void *stream) {
  if (B <= 0 || Hkv <= 0 || T <= 0) return GKV_E_SHAPE;
  if (!k_src || !mass || !qn || !levels) return GKV_E_ARG;
  if (!(c > 0.0) || !(tau > 0.0) || window < 0) return GKV_E_ARG;
  if (rounding != GKV_ROUND_UP && rounding != GKV_ROUND_NEAREST) return GKV_E_ARG;
  const int64_t nblk = (T + P - 1) / P;
  if (nblk > (1ll << 24)) return GKV_E_UNSUPPORTED;
  hipLaunchKernelGGL(alloc_kernel, dim3((unsigned)nblk, Hkv, B), dim3(D), 0, (hipStream_t)stream, k_src, mass, qn,
                     Hkv, T, (int)nblk, c, tau, window, (int)rounding, levels);
  return hipGetLastError() == hipSuccess ? GKV_OK : GKV_E_HIP;
}
