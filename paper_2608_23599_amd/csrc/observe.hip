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
typedef float f4 __attribute__((ext_vector_type(4)));

union H8 {
  half8 h;
  uint4 v;
};

constexpr int kObsThreads = 512;  // 8 wavefronts
constexpr int kObsBlocksPerWave = 16;
constexpr int kObsChunk = 8 * kObsBlocksPerWave;  // blocks per workgroup
constexpr int kMaxRows = 512;
constexpr float kNegInf = -__builtin_huge_valf();

__device__ __forceinline__ f4 mfma32(half8 a, half8 b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// Query rows in LDS: row r holds 16 chunks of 8 channels; chunk c sits at position
// c ^ (r & 15), so that the 16 rows read by one MFMA operand fall in distinct banks.
__device__ __forceinline__ uint32_t qpos(int r, int c) { return (uint32_t)(r * 16 + (c ^ (r & 15))) * 16u; }

// This lane's key operands of one block: key 64 blk + 16 t + m16, channels
// 32 i + 8 kg .. + 7 (zero beyond T).
__device__ __forceinline__ void load_keys(H8 (&a)[4][4], const uint16_t *kb, int64_t T, int blk, int kg, int m16) {
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int64_t key = (int64_t)blk * P + 16 * t + m16;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      a[t][i].v = key < T ? *(const uint4 *)(kb + key * D + 32 * i + 8 * kg) : make_uint4(0, 0, 0, 0);
  }
}

// Sum and maximum over the 4 lanes of a row (lanes m16 + 16 kg): the row swaps pair
// lane l with l ^ 32, then with l ^ 16.
__device__ __forceinline__ float row_sum4(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}
__device__ __forceinline__ float row_max4(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

// Sum over the tile of exp2(s * sl2 - ref) across the 4 lanes of each row; with
// MASKED only the keys <= last (and < T) count.  key0 is the key of s[0][0] for kg = 0.
template <bool MASKED>
__device__ __forceinline__ float tile_sum(const f4 (&s)[4], float sl2, float ref, int64_t key0, int kg,
                                          int64_t last, int64_t T) {
  float x[16];
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[4 * t + e] = __builtin_amdgcn_exp2f(fmaf(s[t][e], sl2, -ref));
      if (MASKED) {
        const int64_t key = key0 + 16 * t + 4 * kg + e;
        x[4 * t + e] = key <= last && key < T ? x[4 * t + e] : 0.f;
      }
    }
#pragma unroll
  for (int w = 8; w >= 1; w >>= 1)  // pairwise: a chain of depth 4
#pragma unroll
    for (int j = 0; j < w; ++j) x[j] += x[j + w];
  return row_sum4(x[0]);
}

template <bool MASKED>
__device__ __forceinline__ float tile_max(const f4 (&s)[4], float sl2, int64_t key0, int kg, int64_t last,
                                          int64_t T) {
  float bm = kNegInf;
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int64_t key = key0 + 16 * t + 4 * kg + e;
      if (!MASKED || (key <= last && key < T)) bm = fmaxf(bm, s[t][e] * sl2);
    }
  return row_max4(bm);
}

// Log-sum-exp (log2 units) of one (block, 16-row tile): sum_j exp2(x_j - ref) with
// ref the row's running maximum, redone against the tile's own maximum when that
// sum overflows (always on a row's first block, where ref = -inf).
template <bool MASKED>
__device__ __forceinline__ float tile_lse(const f4 (&s)[4], float sl2, float ref, int64_t key0, int kg, int64_t last,
                                          int64_t T) {
  // a row's first block (ref = -inf) goes straight to the tile maximum
  float sum = __any(ref == kNegInf) ? __builtin_inff() : tile_sum<MASKED>(s, sl2, ref, key0, kg, last, T);
  if (__any(!(sum <= 0x1p100f))) {
    ref = tile_max<MASKED>(s, sl2, key0, kg, last, T);
    sum = ref == kNegInf ? 0.f : tile_sum<MASKED>(s, sl2, ref, key0, kg, last, T);
  }
  return sum > 0.f ? ref + __builtin_amdgcn_logf(sum) : kNegInf;
}

// Logits and per-block log-sum-exp.  Each wavefront takes kObsBlocksPerWave blocks
// and, per block, every 16-row tile of the group's queries: 16 MFMAs give the 64 x 16
// logits, then sum_j exp2(x_j - ref) over the block's visible keys with ref the row's
// running maximum of block log-sum-exps (kept in LDS per wavefront and row).  The
// block's log-sum-exp is ref + log2(sum), whatever ref is, as long as the sum neither
// overflows (then the tile is redone against the block's own maximum) nor loses all
// its terms (a block 2^-126 below an earlier one, whose share is below fp32
// resolution).  The running (max, sum) over the wavefront's blocks are merged over
// the workgroup into one (max, sum) per (row, workgroup chunk).
__global__ void __launch_bounds__(kObsThreads) obs_logit_kernel(const uint16_t *__restrict__ q_obs,
                                                                const uint16_t *__restrict__ k_src, int n_obs,
                                                                int G, int Hkv, int64_t T, int nblk, int Rpad,
                                                                float sl2, float *__restrict__ lse,
                                                                float2 *__restrict__ part) {
  extern __shared__ __align__(16) uint8_t qs[];
  float2 *stats = (float2 *)(qs + Rpad * 256);  // [8 wavefronts][Rpad] running (max, sum)
  const int h = blockIdx.y, b = blockIdx.z;
  const int64_t u = (int64_t)b * Hkv + h;
  const int R = n_obs * G, Hq = Hkv * G;
  for (int i = threadIdx.x; i < Rpad * 16; i += kObsThreads) {
    const int r = i >> 4, c = i & 15;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (r < R) {
      const int qi = r / G, g = r - qi * G;
      v = *(const uint4 *)(q_obs + (((int64_t)b * n_obs + qi) * Hq + h * G + g) * D + 8 * c);
    }
    *(uint4 *)(qs + qpos(r, c)) = v;
  }
  for (int i = threadIdx.x; i < 8 * Rpad; i += kObsThreads) stats[i] = make_float2(kNegInf, 0.f);
  __syncthreads();
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, kg = lane >> 4, m16 = lane & 15;
  float2 *wst = stats + wv * Rpad;
  const uint16_t *kb = k_src + u * T * D;
  const int64_t first_masked = T - n_obs + 1;  // keys at or beyond this are hidden from some row
  const int blk0 = blockIdx.x * kObsChunk + wv * kObsBlocksPerWave;
  const int nb = blk0 >= nblk ? 0 : (nblk - blk0 < kObsBlocksPerWave ? nblk - blk0 : kObsBlocksPerWave);
  H8 a[4][4];
  for (int k = 0; k < nb; ++k) {
    const int blk = blk0 + k;
    load_keys(a, kb, T, blk, kg, m16);
    const int64_t key0 = (int64_t)blk * P;
    const bool masked = key0 + P > first_masked;  // uniform: the block has hidden keys
    for (int rt = 0; rt < Rpad / 16; rt += 2) {  // two row tiles at a time (Rpad is a multiple of 32)
      int row[2];
      H8 qb[2][4];
      float2 run[2];
      f4 s[2][4];
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        row[p] = 16 * (rt + p) + m16;
#pragma unroll
        for (int i = 0; i < 4; ++i) qb[p][i].v = *(const uint4 *)(qs + qpos(row[p], 4 * i + kg));
        run[p] = wst[row[p]];
#pragma unroll
        for (int t = 0; t < 4; ++t) s[p][t] = f4{0, 0, 0, 0};
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)  // eight independent accumulation chains
#pragma unroll
        for (int p = 0; p < 2; ++p)
#pragma unroll
          for (int t = 0; t < 4; ++t) s[p][t] = mfma32(a[t][i].h, qb[p][i].h, s[p][t]);
      // s[p][t][e]: key 64 blk + 16 t + 4 kg + e, query row row[p]
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        const int64_t last = T - n_obs + row[p] / G;  // the last key this row sees
        const float v = masked ? tile_lse<true>(s[p], sl2, run[p].x, key0, kg, last, T)
                               : tile_lse<false>(s[p], sl2, run[p].x, key0, kg, last, T);
        if (kg == 0 && row[p] < R) {
          lse[(u * nblk + blk) * Rpad + row[p]] = v;
          if (v != kNegInf) {  // the wavefront's running (max, sum) of this row
            float2 r2 = run[p];
            if (v > r2.x) {
              r2.y = r2.y * __builtin_amdgcn_exp2f(r2.x - v) + 1.f;
              r2.x = v;
            } else {
              r2.y += __builtin_amdgcn_exp2f(v - r2.x);
            }
            wst[row[p]] = r2;
          }
        }
      }
    }
  }
  __syncthreads();
  // merge the wavefronts' running sums: one (max, sum) per (row, chunk)
  for (int r = threadIdx.x; r < R; r += kObsThreads) {
    float m = kNegInf;
    for (int w = 0; w < 8; ++w) m = fmaxf(m, stats[w * Rpad + r].x);
    float sm = 0.f;
    if (m != kNegInf)
      for (int w = 0; w < 8; ++w) {
        const float2 p = stats[w * Rpad + r];
        if (p.x != kNegInf) sm += p.y * __builtin_amdgcn_exp2f(p.x - m);
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

// One wavefront per block: mean over rows of the block's share of each row.
__global__ void __launch_bounds__(256) obs_mass_kernel(const float *__restrict__ lse,
                                                       const float *__restrict__ row_lse, int R, int Rpad,
                                                       int nblk, int Hkv, float alpha, float *__restrict__ mass) {
  const int lane = threadIdx.x & 63;
  const int blk = blockIdx.x * 4 + (threadIdx.x >> 6), h = blockIdx.y, b = blockIdx.z;
  if (blk >= nblk) return;
  const int64_t u = (int64_t)b * Hkv + h;
  float acc = 0.f;
  for (int r = lane; r < R; r += 64) {
    const float v = lse[(u * nblk + blk) * Rpad + r];
    if (v != kNegInf) acc += __builtin_amdgcn_exp2f(v - row_lse[u * Rpad + r]);
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) acc += __shfl_xor(acc, o);
  if (lane == 0) {
    const float m = acc / (float)R;
    float *dst = mass + u * nblk + blk;
    *dst = alpha == 1.f ? m : (1.f - alpha) * *dst + alpha * m;
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
  const uint16_t *kb = k_src + (u * T + (int64_t)blk * P) * D + d;
  double mn = (double)__builtin_bit_cast(_Float16, kb[0]), mx = mn;
  for (int t = 1; t < P; ++t) {
    const double x = (double)__builtin_bit_cast(_Float16, kb[(int64_t)t * D]);
    mn = x < mn ? x : mn;
    mx = x > mx ? x : mx;
  }
  rng[d] = mx - mn;  // exact in fp64
  __syncthreads();
  if (d == 0) {
    double e = rng[0];
    for (int i = 1; i < D; ++i) e = rng[i] > e ? rng[i] : e;
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
  hipLaunchKernelGGL(obs_logit_kernel, dim3(L.nslice, Hkv, B), dim3(kObsThreads), L.Rpad * (256 + 8 * 8), s, q_obs,
                     k_src, n_obs, G, Hkv, T, L.nblk, L.Rpad, sl2, lse, part);
  hipLaunchKernelGGL(obs_row_kernel, dim3((L.R + 3) / 4, Hkv, B), dim3(256), 0, s, part, L.R, L.Rpad, L.nslice, Hkv,
                     rows);
  hipLaunchKernelGGL(obs_mass_kernel, dim3((L.nblk + 3) / 4, Hkv, B), dim3(256), 0, s, lse, rows, L.R, L.Rpad,
                     L.nblk, Hkv, alpha, mass);
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
