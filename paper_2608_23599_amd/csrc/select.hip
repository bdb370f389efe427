// Compressed-Quest page ranking (section 3.5) and rate-distortion residual
// selection (section 3.4): scoring kernels write order-preserving 64-bit keys, a
// radix-select kernel picks the first k of the order (key descending, index
// ascending) and writes the winners in ascending index order.
#include <hip/hip_runtime.h>

#include "gkv_internal.h"

#pragma clang fp contract(off)

using namespace gkv;

void gkv_launch_rd_score(const gkv_cache *c, const uint16_t *v_src, const float *mass, uint64_t *keys,
                         hipStream_t stream);
int64_t gkv_attn_workspace(const gkv_cache *c, int32_t topk);

namespace {

__device__ __forceinline__ uint64_t order_key(double x) {
  x = x + 0.0;  // -0 -> +0
  uint64_t bits;
  __builtin_memcpy(&bits, &x, 8);
  return (bits >> 63) ? ~bits : (bits | 0x8000000000000000ull);
}

// Box upper bound of every ranked page for the G query heads of a KV head:
// UB_g(p) = sum_d q_gd * (q_gd >= 0 ? kmax_pd : kmin_pd), channel-ascending in fp64
// (each product of two fp16 values is exact, so the fused multiply-add rounds once,
// like a separate add); page score = max_g UB_g.  grid (ceil(npages/256), Hkv, B).
__global__ void __launch_bounds__(256) quest_score_kernel(const uint16_t *__restrict__ q,
                                                          const uint16_t *__restrict__ boxes, int64_t npage_cap,
                                                          int64_t npages, int Hkv, int G,
                                                          uint64_t *__restrict__ keys) {
  __shared__ double qs[16 * D];
  const int h = blockIdx.y, b = blockIdx.z;
  const int64_t u = (int64_t)b * Hkv + h;
  for (int i = threadIdx.x; i < G * D; i += 256) qs[i] = (double)__builtin_bit_cast(_Float16, q[u * G * D + i]);
  __syncthreads();
  const int64_t pg = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (pg >= npages) return;
  const uint32_t *bx = (const uint32_t *)(boxes + u * npage_cap * 2 * D);
  double acc[16];
#pragma unroll
  for (int g = 0; g < 16; ++g) acc[g] = 0.0;
  for (int d = 0; d < D; ++d) {
    const uint32_t pr = bx[box_index(pg, d) >> 1];
    const double lo = (double)__builtin_bit_cast(_Float16, (uint16_t)(pr & 0xFFFFu));
    const double hi = (double)__builtin_bit_cast(_Float16, (uint16_t)(pr >> 16));
#pragma unroll
    for (int g = 0; g < 16; ++g) {
      if (g < G) {
        const double qd = qs[g * D + d];
        acc[g] = __builtin_fma(qd, qd >= 0.0 ? hi : lo, acc[g]);
      }
    }
  }
  double best = acc[0];
#pragma unroll
  for (int g = 1; g < 16; ++g)
    if (g < G) best = acc[g] > best ? acc[g] : best;
  keys[u * npage_cap + pg] = order_key(best);
}

// Select the first k of the order (key desc, index asc) among keys[0..n) of one
// unit and write their indices ascending to out[0..k) (-1 padded).  Optionally
// sets the selected tokens' bits in a per-64 mask.  One workgroup per unit.
constexpr int kSelThreads = 1024;

__global__ void __launch_bounds__(kSelThreads) select_kernel(const uint64_t *__restrict__ keys, int64_t key_stride,
                                                             int64_t n, int k, int32_t *__restrict__ out,
                                                             int64_t out_stride, uint64_t *mask, int64_t mask_stride,
                                                             int64_t mask_words) {
  __shared__ uint32_t hist[256];
  __shared__ uint64_t sh_prefix, sh_pmask;
  __shared__ int64_t sh_remaining;
  __shared__ int64_t wsum[kSelThreads / 64][2];
  __shared__ int64_t sh_base[2];
  const int64_t u = blockIdx.x;
  const uint64_t *key = keys + u * key_stride;
  int32_t *o = out + u * out_stride;
  uint64_t *mk = mask ? mask + u * mask_stride : nullptr;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  if (mk)
    for (int64_t i = tid; i < mask_words; i += kSelThreads) mk[i] = 0;
  const int64_t need = n < k ? n : k;
  for (int64_t i = need + tid; i < k; i += kSelThreads) o[i] = -1;
  if (need == 0) return;
  // radix select of the threshold key (the need-th largest), 8 bits at a time
  if (tid == 0) {
    sh_prefix = 0;
    sh_pmask = 0;
    sh_remaining = need;
  }
  __syncthreads();
  for (int pass = 0; pass < 8; ++pass) {
    const int shift = 56 - 8 * pass;
    for (int i = tid; i < 256; i += kSelThreads) hist[i] = 0;
    __syncthreads();
    const uint64_t pre = sh_prefix, pm = sh_pmask;
    for (int64_t i = tid; i < n; i += kSelThreads) {
      const uint64_t kv = key[i];
      if ((kv & pm) == pre) atomicAdd(&hist[(kv >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (tid == 0) {
      int64_t rem = sh_remaining;
      int dig = 255;
      for (; dig > 0; --dig) {
        if ((int64_t)hist[dig] >= rem) break;
        rem -= hist[dig];
      }
      sh_remaining = rem;
      sh_prefix = pre | ((uint64_t)dig << shift);
      sh_pmask = pm | (0xFFull << shift);
    }
    __syncthreads();
  }
  const uint64_t thr = sh_prefix;
  const int64_t eq_take = sh_remaining;  // keys equal to thr to take, lowest index first
  // ordered compaction: selected = key > thr, or key == thr among the first eq_take
  if (tid == 0) {
    sh_base[0] = 0;  // selected so far
    sh_base[1] = 0;  // keys equal to thr so far
  }
  __syncthreads();
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int64_t c0 = 0; c0 < n; c0 += kSelThreads) {
    const int64_t i = c0 + tid;
    const bool in = i < n;
    const uint64_t kv = in ? key[i] : 0;
    const bool gt = in && kv > thr, eq = in && kv == thr;
    const uint64_t be = __ballot(eq);
    if (lane == 0) wsum[wv][0] = __popcll(be);
    __syncthreads();
    int64_t eq_rank = sh_base[1] + __popcll(be & below);
    for (int q = 0; q < wv; ++q) eq_rank += wsum[q][0];
    const bool sel = gt || (eq && eq_rank < eq_take);
    const uint64_t bs = __ballot(sel);
    if (lane == 0) wsum[wv][1] = __popcll(bs);
    __syncthreads();
    int64_t pos = sh_base[0] + __popcll(bs & below);
    for (int q = 0; q < wv; ++q) pos += wsum[q][1];
    if (sel) {
      o[pos] = (int32_t)i;
      if (mk) atomicOr((unsigned long long *)&mk[i >> 6], 1ull << (i & 63));
    }
    __syncthreads();
    if (tid == 0) {
      for (int q = 0; q < kSelThreads / 64; ++q) {
        sh_base[0] += wsum[q][1];
        sh_base[1] += wsum[q][0];
      }
    }
    __syncthreads();
  }
}

// Copy the exact key/value rows of the selected residual tokens into exact-format
// pseudo-blocks.  grid (ceil(nkeep/64), Hkv, B), 256 threads.
__global__ void __launch_bounds__(256) res_gather_kernel(const uint16_t *__restrict__ k_src,
                                                         const uint16_t *__restrict__ v_src, int64_t T,
                                                         const int32_t *__restrict__ res_idx, int nres_cap,
                                                         int nkeep, uint8_t *res_rows, int Hkv) {
  const int rb = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int64_t u = (int64_t)b * Hkv + h;
  const int nrb = (nres_cap + P - 1) / P;
  uint16_t *kr = (uint16_t *)(res_rows + (u * nrb + rb) * (2 * kExactBytes));
  uint16_t *vr = kr + kExactBytes / 2;
  for (int i = threadIdx.x; i < P * D; i += 256) {
    const int slot = i >> 7, d = i & 127;
    const int r = rb * P + slot;
    uint16_t kv = 0, vv = 0;
    if (r < nkeep) {
      const int64_t tok = res_idx[u * nres_cap + r];
      kv = k_src[(u * T + tok) * D + d];
      vv = v_src[(u * T + tok) * D + d];
    }
    {  // key element (slot, d)
      const int pg = slot >> 4, lane = ((d >> 3) & 3) * 16 + (slot & 15), n = ((d >> 5) << 3) | (d & 7);
      kr[(pg * 64 + lane) * 32 + n] = kv;
    }
    {  // value element (slot, d)
      const int pg = slot >> 4, lane = ((slot >> 2) & 3) * 16 + (d & 15), n = ((d >> 4) << 2) | (slot & 3);
      vr[(pg * 64 + lane) * 32 + n] = vv;
    }
  }
}

}  // namespace

// ---------------------------------------------------------------- C ABI
static int64_t quest_ws(const gkv_cache *c) { return (int64_t)c->B * c->Hkv * c->npage_cap * 8; }
static int64_t rd_ws(const gkv_cache *c) { return (int64_t)c->B * c->Hkv * (c->T > 0 ? c->T : 1) * 8; }

extern "C" int64_t gkv_workspace_bytes(const gkv_cache *c, int32_t op, int32_t topk) {
  if (gkv_validate_cache(c)) return -1;
  if (op == 0) return c->page ? quest_ws(c) : -1;
  if (op == 1) return gkv_attn_workspace(c, topk > 0 ? topk : 0);
  if (op == 2) return rd_ws(c);
  return -1;
}

extern "C" gkv_status gkv_quest_select(const uint16_t *q, const gkv_cache *c, int32_t topk, int32_t *pages, void *ws,
                                       int64_t ws_bytes, void *stream) {
  gkv_status st = gkv_validate_cache(c);
  if (st) return st;
  if (!q || !pages || !ws || topk <= 0) return GKV_E_ARG;
  if (!c->page) return GKV_E_ARG;
  if (c->T <= 0) return GKV_E_SHAPE;
  if (ws_bytes < quest_ws(c)) return GKV_E_WORKSPACE;
  const int G = c->Hq / c->Hkv;
  const int64_t ncur = (c->T - 1) / c->page;  // ranked pages
  if (ncur > c->npage_cap) return GKV_E_SHAPE;
  hipStream_t s = (hipStream_t)stream;
  uint64_t *keys = (uint64_t *)ws;
  if (ncur > 0) {
    dim3 grid((unsigned)((ncur + 255) / 256), c->Hkv, c->B);
    hipLaunchKernelGGL(quest_score_kernel, grid, dim3(256), 0, s, q, c->boxes, c->npage_cap, ncur, c->Hkv, G, keys);
  }
  hipLaunchKernelGGL(select_kernel, dim3(c->B * c->Hkv), dim3(kSelThreads), 0, s, (const uint64_t *)keys, c->npage_cap,
                     ncur, topk, pages, (int64_t)topk, (uint64_t *)nullptr, (int64_t)0, (int64_t)0);
  return hipGetLastError() == hipSuccess ? GKV_OK : GKV_E_HIP;
}

extern "C" gkv_status gkv_rd_residual_select(gkv_cache *c, const uint16_t *k_src, const uint16_t *v_src,
                                             const float *mass, int32_t nkeep, void *ws, int64_t ws_bytes,
                                             void *stream) {
  gkv_status st = gkv_validate_cache(c);
  if (st) return st;
  if (!k_src || !v_src || !mass || !ws || nkeep < 0) return GKV_E_ARG;
  if (c->T <= 0) return GKV_E_SHAPE;
  if (nkeep > c->nres_cap || nkeep > c->T) return GKV_E_SHAPE;
  if (ws_bytes < rd_ws(c)) return GKV_E_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  uint64_t *keys = (uint64_t *)ws;
  if (nkeep > 0) gkv_launch_rd_score(c, v_src, mass, keys, s);
  hipLaunchKernelGGL(select_kernel, dim3(c->B * c->Hkv), dim3(kSelThreads), 0, s, (const uint64_t *)keys, c->T, c->T,
                     nkeep, c->res_idx, (int64_t)c->nres_cap, c->res_mask, (int64_t)c->nblk_cap,
                     (int64_t)c->nblk_cap);
  if (nkeep > 0) {
    dim3 g2((unsigned)((nkeep + P - 1) / P), c->Hkv, c->B);
    hipLaunchKernelGGL(res_gather_kernel, g2, dim3(256), 0, s, k_src, v_src, c->T, (const int32_t *)c->res_idx,
                       c->nres_cap, nkeep, c->res_rows, c->Hkv);
  }
  if (hipGetLastError() != hipSuccess) return GKV_E_HIP;
  c->nres = nkeep;
  return GKV_OK;
}
