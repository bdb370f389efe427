// Block encoders of the precision ladder (section 3.2), monotone demotion, token
// append, and exact page boxes (section 3.5).
//
// Every arithmetic step whose result is stored (scales, zeros, codes, centroids,
// ids, boxes) is exact-reproducible: fp64 with one rounding per operation, no
// contraction into fused multiply-adds, channel/token-ascending sequential sums,
// and one round-to-nearest-even to fp16 (gkv::f64_to_f16).
#include <hip/hip_runtime.h>

#include "gkv_internal.h"

#pragma clang fp contract(off)

using namespace gkv;

namespace {

constexpr int kThreads = 256;
constexpr int XS = D + 1;  // padded LDS row stride (doubles) against bank conflicts

struct EncodeShared {
  uint16_t xh[P * D];      // source as fp16 bits [token][channel] (rows or exact record)
  uint8_t xc[P * D];       // source as codes (int-level record being demoted)
  double xs[D], xz[D];     // source scale / zero for xc
  int32_t src_int;         // 1: x = xc * xs + xz, 0: x = xh, 2: x = centroid[xc]
  int32_t src_tok;         // with src_int == 1: xs, xz are per token (index t), else per channel
  double sc[KC * D];       // source centroids (fp64) when src_int == 2
  double c[KC * XS];       // centroids (fp64)
  double dist[P * KC];     // token x centroid distances
  double s64[D], z64[D];   // new scale / zero
  uint16_t s16[D], z16[D];
  uint8_t codes[P * D];    // new codes (int levels)
  int32_t assign[P], prev[P];
  int32_t flag;
  double cert[2];  // block_cert results
};

// Exact fp64 value of source element (t, d): an fp16 value, or code * scale + zero
// (both products and the sum are exact in fp64).
__device__ __forceinline__ double getx(const EncodeShared &S, int t, int d) {
  if (S.src_int == 2) return S.sc[S.xc[t * D] * D + d];
  if (S.src_int) {
    const int g = S.src_tok ? t : d;
    const double prod = (double)S.xc[t * D + d] * S.xs[g];
    return prod + S.xz[g];
  }
  return (double)__builtin_bit_cast(_Float16, S.xh[t * D + d]);
}

// Load the 64 x 128 block starting at row0 of one (b,h) from token-major fp16 rows;
// rows at or beyond T_src read as zero.
__device__ void load_rows(EncodeShared &S, const uint16_t *src, int64_t T_src, int64_t row0) {
  if (threadIdx.x == 0) {
    S.src_int = 0;
    S.src_tok = 0;
  }
  for (int i = threadIdx.x; i < P * (D / 8); i += kThreads) {
    const int t = i / (D / 8), c8 = (i % (D / 8)) * 8;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (row0 + t < T_src) v = *(const uint4 *)(src + (row0 + t) * D + c8);
    *(uint4 *)(S.xh + t * D + c8) = v;
  }
}

// Load a record as the source (per_token: an int-level value record grouped per token).
__device__ void load_record(EncodeShared &S, const uint8_t *rec, int level, int tensor, bool per_token) {
  if (threadIdx.x == 0) S.src_tok = per_token && is_int_level(level);
  if (level == GKV_EXACT) {
    if (threadIdx.x == 0) S.src_int = 0;
    const uint16_t *hh = (const uint16_t *)rec;
    for (int ck = threadIdx.x; ck < 4 * 64; ck += kThreads) {
      const int pg = ck >> 6, l = ck & 63;
      for (int n = 0; n < 32; ++n) {
        int t, ch;
        chunk_coord(tensor, pg, l, n, t, ch);
        S.xh[t * D + ch] = hh[ck * 32 + n];
      }
    }
    return;
  }
  if (level == GKV_MEAN) {  // one centroid: every token reads it
    if (threadIdx.x == 0) S.src_int = 2;
    const uint16_t *cc = (const uint16_t *)rec;
    for (int d = threadIdx.x; d < D; d += kThreads) S.sc[d] = (double)__builtin_bit_cast(_Float16, cc[d]);
    for (int t = threadIdx.x; t < P; t += kThreads) S.xc[t * D] = 0;
    return;
  }
  if (level == GKV_CENTROID) {
    if (threadIdx.x == 0) S.src_int = 2;
    const uint16_t *cc = (const uint16_t *)rec;
    for (int i = threadIdx.x; i < KC * D; i += kThreads) {
      const int k = i >> 7, d = i & 127;
      S.sc[i] = (double)__builtin_bit_cast(_Float16, cc[tensor == GKV_KEYS ? k * D + d : vcent_index(k, d)]);
    }
    const uint8_t *idb = rec + KC * D * 2;
    for (int t = threadIdx.x; t < P; t += kThreads) S.xc[t * D] = (idb[t >> 2] >> (2 * (t & 3))) & 3;
    return;
  }
  if (threadIdx.x == 0) S.src_int = 1;
  const uint16_t *sz = (const uint16_t *)rec;
  if (per_token) {
    for (int t = threadIdx.x; t < P; t += kThreads) {
      S.xs[t] = (double)__builtin_bit_cast(_Float16, sz[t]);
      S.xz[t] = (double)__builtin_bit_cast(_Float16, sz[P + t]);
    }
  } else {
    for (int e = threadIdx.x; e < D; e += kThreads) {
      const int ch = sz_channel(tensor, e);
      S.xs[ch] = (double)__builtin_bit_cast(_Float16, sz[e]);
      S.xz[ch] = (double)__builtin_bit_cast(_Float16, sz[D + e]);
    }
  }
  const int bits = level;
  const uint32_t *w = (const uint32_t *)(rec + kSZBytes);
  for (int ck = threadIdx.x; ck < 4 * 64; ck += kThreads) {
    const int pg = ck >> 6, l = ck & 63;
    for (int n = 0; n < 32; ++n) {
      int t, ch;
      chunk_coord(tensor, pg, l, n, t, ch);
      const uint32_t word = w[ck * bits + code_word(bits, n)];
      S.xc[t * D + ch] = (uint8_t)((word >> code_pos(bits, n)) & ((1u << bits) - 1u));
    }
  }
}

// Exact level: store the fp16 source in chunk order (source must be fp16).
__device__ void write_exact(EncodeShared &S, uint8_t *dst, int tensor) {
  uint16_t *hh = (uint16_t *)dst;
  for (int ck = threadIdx.x; ck < 4 * 64; ck += kThreads) {
    const int pg = ck >> 6, l = ck & 63;
    uint32_t w[16];
    for (int n = 0; n < 32; n += 2) {
      int t0, c0, t1, c1;
      chunk_coord(tensor, pg, l, n, t0, c0);
      chunk_coord(tensor, pg, l, n + 1, t1, c1);
      w[n >> 1] = (uint32_t)S.xh[t0 * D + c0] | ((uint32_t)S.xh[t1 * D + c1] << 16);
    }
    uint4 *o = (uint4 *)(hh + ck * 32);
    for (int q = 0; q < 4; ++q) o[q] = make_uint4(w[4 * q], w[4 * q + 1], w[4 * q + 2], w[4 * q + 3]);
  }
}

// Scalar quantizer, one group per channel, or per token for a value block of a
// cache that groups values per token (section 3.2).
__device__ void encode_int(EncodeShared &S, uint8_t *dst, int bits, int tensor, bool per_token) {
  const double qmax = (double)((1 << bits) - 1);
  const int tid = threadIdx.x;
  if (tid < (per_token ? P : D)) {
    double mn = per_token ? getx(S, tid, 0) : getx(S, 0, tid), mx = mn;
    for (int i = 1; i < (per_token ? D : P); ++i) {
      const double v = per_token ? getx(S, tid, i) : getx(S, i, tid);
      mn = v < mn ? v : mn;
      mx = v > mx ? v : mx;
    }
    const double range = mx - mn;
    const uint16_t z = canon_zero(f64_to_f16(mn));
    const uint16_t s = canon_zero(f64_to_f16(range / qmax));
    S.z16[tid] = z;
    S.s16[tid] = s;
    S.z64[tid] = f16_to_f64(z);
    S.s64[tid] = f16_to_f64(s);
  }
  __syncthreads();
  for (int i = tid; i < P * D; i += kThreads) {
    const int t = i >> 7, d = i & 127, g = per_token ? t : d;
    const double s = S.s64[g];
    uint8_t code = 0;
    if (s != 0.0) {
      const double diff = getx(S, t, d) - S.z64[g];
      double r = __builtin_rint(diff / s);
      r = r < 0.0 ? 0.0 : r;
      r = r > qmax ? qmax : r;
      code = (uint8_t)r;
    }
    S.codes[t * D + d] = code;
  }
  __syncthreads();
  uint16_t *sz = (uint16_t *)dst;
  if (per_token) {  // scale[64], zero[64] in token order, then zeros
    for (int e = tid; e < 2 * D; e += kThreads) sz[e] = e < P ? S.s16[e] : (e < 2 * P ? S.z16[e - P] : 0);
  } else {
    for (int e = tid; e < D; e += kThreads) {
      const int ch = sz_channel(tensor, e);
      sz[e] = S.s16[ch];
      sz[D + e] = S.z16[ch];
    }
  }
  uint32_t *w = (uint32_t *)(dst + kSZBytes);
  for (int ck = tid; ck < 4 * 64; ck += kThreads) {
    const int pg = ck >> 6, l = ck & 63;
    uint32_t words[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int n = 0; n < 32; ++n) {
      int t, ch;
      chunk_coord(tensor, pg, l, n, t, ch);
      words[code_word(bits, n)] |= (uint32_t)S.codes[t * D + ch] << code_pos(bits, n);
    }
    for (int q = 0; q < bits; ++q) w[ck * bits + q] = words[q];
  }
}

// Squared distances of every token to every centroid, channel-ascending, no FMA.
__device__ void kmeans_dist(EncodeShared &S) {
  const int t = threadIdx.x >> 2, k = threadIdx.x & 3;  // 256 threads = 64 tokens x 4
  double acc = 0.0;
  for (int d = 0; d < D; ++d) {
    const double diff = getx(S, t, d) - S.c[k * XS + d];
    const double sq = diff * diff;
    acc = acc + sq;
  }
  S.dist[t * KC + k] = acc;
  __syncthreads();
  if (threadIdx.x < P) {
    const int tt = threadIdx.x;
    int best = 0;
    double bd = S.dist[tt * KC];
    for (int kk = 1; kk < KC; ++kk)
      if (S.dist[tt * KC + kk] < bd) {
        bd = S.dist[tt * KC + kk];
        best = kk;
      }
    S.assign[tt] = best;
  }
  __syncthreads();
}

// Deterministic 4-means Lloyd iteration, then fp16 centroids and re-assigned ids.
__device__ void encode_centroid(EncodeShared &S, uint8_t *dst, int tensor) {
  const int tid = threadIdx.x;
  for (int i = tid; i < KC * D; i += kThreads) {
    const int k = i >> 7, d = i & 127;
    S.c[k * XS + d] = getx(S, k * (P / KC), d);
  }
  __syncthreads();
  for (int it = 0; it < 10; ++it) {
    kmeans_dist(S);
    if (tid == 0) S.flag = 0;
    __syncthreads();
    if (it > 0 && tid < P && S.assign[tid] != S.prev[tid]) atomicOr(&S.flag, 1);
    __syncthreads();
    if (it > 0 && S.flag == 0) break;  // assignment repeated: converged
    if (tid < P) S.prev[tid] = S.assign[tid];
    __syncthreads();
    for (int i = tid; i < KC * D; i += kThreads) {
      const int k = i >> 7, d = i & 127;
      double acc = 0.0;
      int n = 0;
      for (int t = 0; t < P; ++t)
        if (S.assign[t] == k) {
          acc = acc + getx(S, t, d);
          ++n;
        }
      if (n > 0) S.c[k * XS + d] = acc / (double)n;
    }
    __syncthreads();
  }
  // round the centroids to fp16 and assign against what is stored
  uint16_t *cc = (uint16_t *)dst;
  for (int i = tid; i < KC * D; i += kThreads) {
    const int k = i >> 7, d = i & 127;
    const uint16_t h = canon_zero(f64_to_f16(S.c[k * XS + d]));
    S.c[k * XS + d] = f16_to_f64(h);
    cc[tensor == GKV_KEYS ? k * D + d : vcent_index(k, d)] = h;
  }
  __syncthreads();
  kmeans_dist(S);
  if (tid < P / 16) {
    uint32_t w = 0;
    for (int j = 0; j < 16; ++j) w |= (uint32_t)S.assign[tid * 16 + j] << (2 * j);
    ((uint32_t *)(dst + KC * D * 2))[tid] = w;
  }
}

// One-centroid state: the Lloyd iteration with one centroid converges in one
// update to the block mean; the fp64 token-ascending sum of 64 fp16 values (or of
// decoded values) is the same sum the iteration takes, then one fp16 rounding.
__device__ void encode_mean(EncodeShared &S, uint8_t *dst) {
  const int tid = threadIdx.x;
  if (tid < D) {
    double acc = 0.0;
    for (int t = 0; t < P; ++t) acc = acc + getx(S, t, tid);
    const uint16_t h = canon_zero(f64_to_f16(acc / (double)P));
    S.c[tid] = f16_to_f64(h);  // centroid 0, for the certificate
    ((uint16_t *)dst)[tid] = h;
  }
  if (tid < P) S.assign[tid] = 0;
}

__device__ void encode_to(EncodeShared &S, uint8_t *dst, int level, int tensor, bool per_token) {
  if (level == GKV_EXACT) write_exact(S, dst, tensor);
  else if (is_int_level(level)) encode_int(S, dst, level, tensor, per_token);
  else if (level == GKV_MEAN) encode_mean(S, dst);
  else encode_centroid(S, dst, tensor);
}

// Non-negative fp64 -> fp32 rounded towards +inf (the certificate keeps upper
// bounds): one ulp up when the nearest float lies below.
__device__ __forceinline__ float round_up_f32(double x) {
  float f = (float)x;
  if ((double)f < x) f = __builtin_bit_cast(float, __builtin_bit_cast(uint32_t, f) + 1u);
  return f;
}

// Certificate numbers of the block just encoded at `level` from the source in S:
// err = max_t ||x_t - x_hat_t|| and nrm = max_t ||x_t|| over the 64 rows (fp64; x is
// the source, x_hat the new record's reconstruction).  256 threads: 4 per row, 32
// channels each.  Result in S.cert[0..1].
__device__ void block_cert(EncodeShared &S, int level, bool per_token) {
  const int t = threadIdx.x >> 2, j = threadIdx.x & 3;
  double e = 0.0, n = 0.0;
  for (int d = 32 * j; d < 32 * j + 32; ++d) {
    const double x = getx(S, t, d);
    double xh = x;
    if (is_int_level(level)) {
      const int g = per_token ? t : d;
      xh = (double)S.codes[t * D + d] * S.s64[g] + S.z64[g];
    }
    else if (level == GKV_CENTROID || level == GKV_MEAN) xh = S.c[S.assign[t] * XS + d];
    e += (x - xh) * (x - xh);
    n += x * x;
  }
  e += __shfl_xor(e, 1);
  e += __shfl_xor(e, 2);
  n += __shfl_xor(n, 1);
  n += __shfl_xor(n, 2);
  if (j == 0) {
    S.dist[t * KC] = e;  // scratch: the k-means distances are no longer needed
    S.dist[t * KC + 1] = n;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double me = 0.0, mn = 0.0;
    for (int r = 0; r < P; ++r) {
      me = S.dist[r * KC] > me ? S.dist[r * KC] : me;
      mn = S.dist[r * KC + 1] > mn ? S.dist[r * KC + 1] : mn;
    }
    S.cert[0] = __builtin_sqrt(me);
    S.cert[1] = __builtin_sqrt(mn);
  }
  __syncthreads();
}

// Prefill encode: one workgroup per (block, h, b) of one tensor.
__global__ void __launch_bounds__(kThreads) quantize_kernel(const uint16_t *__restrict__ src, int64_t T_src,
                                                            const int8_t *__restrict__ level,
                                                            const int64_t *__restrict__ off, uint8_t *arena,
                                                            int Hkv, int nblk_cap, int blk0, int tensor,
                                                            float *cert, int vtok, const int64_t *seq_len) {
  extern __shared__ __align__(16) unsigned char smem[];
  EncodeShared &S = *reinterpret_cast<EncodeShared *>(smem);
  const int blk = blk0 + blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int64_t u = (int64_t)b * Hkv + h;
  // a sequence's own length bounds its rows; blocks past its end are not encoded
  const int64_t Tb = seq_len ? (seq_len[b] < T_src ? seq_len[b] : T_src) : T_src;
  if ((int64_t)blk * P >= Tb) return;
  const int lv = level[u * nblk_cap + blk];
  const bool per_token = tensor == GKV_VALUES && vtok;
  load_rows(S, src + u * T_src * D, Tb, (int64_t)blk * P);
  __syncthreads();
  encode_to(S, arena + off[u * nblk_cap + blk], lv, tensor, per_token);
  if (cert) {  // error against the exact rows; the value tensor also keeps the row norms
    __syncthreads();
    block_cert(S, lv, per_token);
    if (threadIdx.x == 0) {
      float *cb = cert + (u * nblk_cap + blk) * 4;
      if (tensor == GKV_KEYS) {
        cb[0] = round_up_f32(S.cert[0]);
      } else {
        cb[1] = round_up_f32(S.cert[0]);
        cb[2] = round_up_f32(S.cert[1]);
        cb[3] = 0.f;
      }
    }
  }
}

constexpr int kMaxDemoteJobs = 64;
struct DemoteJobs {
  int32_t b[kMaxDemoteJobs], h[kMaxDemoteJobs], blk[kMaxDemoteJobs];
  int8_t to[kMaxDemoteJobs], cur[kMaxDemoteJobs];  // cur from the host mirror: the key
                                                    // workgroup rewrites the device level
  int64_t koff[kMaxDemoteJobs], voff[kMaxDemoteJobs];
};

// Demotion: grid (jobs, 2 tensors).  Reads the current record through the device
// tables, writes the new record, then points the tables at it.
__global__ void __launch_bounds__(kThreads) demote_kernel(DemoteJobs jobs, int8_t *level, int64_t *koff,
                                                          int64_t *voff, uint8_t *arena, int Hkv, int nblk_cap,
                                                          float *cert, int vtok) {
  extern __shared__ __align__(16) unsigned char smem[];
  EncodeShared &S = *reinterpret_cast<EncodeShared *>(smem);
  const int j = blockIdx.x, tensor = blockIdx.y;
  const int64_t idx = ((int64_t)jobs.b[j] * Hkv + jobs.h[j]) * nblk_cap + jobs.blk[j];
  const int cur = jobs.cur[j];
  int64_t *offt = tensor == GKV_KEYS ? koff : voff;
  const int64_t dst = tensor == GKV_KEYS ? jobs.koff[j] : jobs.voff[j];
  const bool per_token = tensor == GKV_VALUES && vtok;
  load_record(S, arena + offt[idx], cur, tensor, per_token);
  __syncthreads();
  encode_to(S, arena + dst, jobs.to[j], tensor, per_token);
  __syncthreads();
  if (cert) {  // the error grows by at most the change of the reconstruction
    block_cert(S, jobs.to[j], per_token);
    if (threadIdx.x == 0) {
      float *ce = cert + idx * 4 + (tensor == GKV_KEYS ? 0 : 1);
      *ce = round_up_f32((double)*ce + S.cert[0]);
    }
  }
  if (threadIdx.x == 0) {
    offt[idx] = dst;
    if (tensor == GKV_KEYS) level[idx] = jobs.to[j];
  }
}

// Append one token per (b,h); grid (Hkv, B), 128 threads (one per channel).
// The new blocks' slots of the units that open one, and with per-sequence lengths the
// length of every sequence before the token (-1: retired, skipped).
struct NewSlots {
  int64_t k[GKV_MAX_APPEND_UNITS], v[GKV_MAX_APPEND_UNITS];
  int64_t len[GKV_MAX_APPEND_UNITS];
};

// Writes the token of unit u at position T (row tok = T % 64 of the exact block at
// key / value offsets ko / vo, record slot ti): its key and value rows, the value-norm
// bound and, when the token completes a page, that page's box.  128 threads, one per
// channel d.
__device__ __forceinline__ void append_write(const uint16_t *__restrict__ k_new, const uint16_t *__restrict__ v_new,
                                             uint8_t *arena, uint16_t *boxes, int64_t npage_cap, int page,
                                             int64_t u, int64_t T, int64_t ti, int64_t ko, int64_t vo,
                                             bool open_block, float *cert, double *vsq, int d) {
  const int tok = (int)(T % P);
  const uint16_t kv = k_new[u * D + d], vv = v_new[u * D + d];
  if (cert) {  // an exact block: no error; the value norms grow by this row
    const double x = (double)__builtin_bit_cast(_Float16, vv);
    vsq[d] = x * x;
    __syncthreads();
    if (d == 0) {
      double n = 0.0;
      for (int i = 0; i < D; ++i) n += vsq[i];
      float *cb = cert + ti * 4;
      const float vn = round_up_f32(__builtin_sqrt(n));
      if (open_block) {
        cb[0] = 0.f;
        cb[1] = 0.f;
        cb[2] = vn;
        cb[3] = 0.f;
      } else {
        cb[2] = vn > cb[2] ? vn : cb[2];
      }
    }
  }
  // key element (tok, d): page tok>>4, lane ((d>>3)&3)*16 + (tok&15), n = ((d>>5)<<3) | (d&7)
  {
    const int pg = tok >> 4, lane = ((d >> 3) & 3) * 16 + (tok & 15), n = ((d >> 5) << 3) | (d & 7);
    ((uint16_t *)(arena + ko))[(pg * 64 + lane) * 32 + n] = kv;
  }
  // value element (tok, d): page tok>>4, lane ((tok>>2)&3)*16 + (d&15), n = ((d>>4)<<2) | (tok&3)
  {
    const int pg = tok >> 4, lane = ((tok >> 2) & 3) * 16 + (d & 15), n = ((d >> 4) << 2) | (tok & 3);
    ((uint16_t *)(arena + vo))[(pg * 64 + lane) * 32 + n] = vv;
  }
  if (boxes && ((T + 1) % page) == 0) {
    // the page just completed lies in this (exact) block; earlier rows were written
    // by earlier appends, the newest row is still in registers
    const int64_t p = (T + 1) / page - 1;
    const int first = tok + 1 - page;
    _Float16 mn = __builtin_bit_cast(_Float16, kv), mx = mn;
    const uint16_t *rec = (const uint16_t *)(arena + ko);
    for (int t = first; t < tok; ++t) {
      const int pg = t >> 4, lane = ((d >> 3) & 3) * 16 + (t & 15), n = ((d >> 5) << 3) | (d & 7);
      const _Float16 v = __builtin_bit_cast(_Float16, rec[(pg * 64 + lane) * 32 + n]);
      mn = v < mn ? v : mn;
      mx = v > mx ? v : mx;
    }
    uint16_t *bx = boxes + u * npage_cap * 2 * D + box_index(p, d);
    bx[0] = canon_zero(__builtin_bit_cast(uint16_t, mn));
    bx[1] = canon_zero(__builtin_bit_cast(uint16_t, mx));
  }
}

__global__ void __launch_bounds__(128) append_kernel(const uint16_t *__restrict__ k_new,
                                                     const uint16_t *__restrict__ v_new, int8_t *level,
                                                     int64_t *koff, int64_t *voff, uint8_t *arena,
                                                     uint16_t *boxes, int64_t npage_cap, int page, int Hkv,
                                                     int nblk_cap, int64_t T_all, int64_t *seq_len, NewSlots slots,
                                                     float *cert) {
  __shared__ double vsq[D];
  const int h = blockIdx.x, b = blockIdx.y, d = threadIdx.x;
  const int64_t u = (int64_t)b * Hkv + h;
  const int64_t T = seq_len ? slots.len[b] : T_all;
  if (T < 0) return;  // a retired sequence
  if (seq_len && h == 0 && d == 0) seq_len[b] = T + 1;
  const int open_block = (T % P) == 0;
  const int blk = (int)(T / P);
  const int64_t ti = u * nblk_cap + blk;
  int64_t ko, vo;
  if (open_block) {
    ko = slots.k[u];
    vo = slots.v[u];
    if (d == 0) {
      level[ti] = GKV_EXACT;
      koff[ti] = ko;
      voff[ti] = vo;
    }
  } else {
    ko = koff[ti];
    vo = voff[ti];
  }
  if (open_block) {  // a new block's other rows are defined (zero): reads mask them, but 0 * NaN is NaN
    uint4 *kz = (uint4 *)(arena + ko), *vz = (uint4 *)(arena + vo);
    for (int i = d; i < kExactBytes / 16; i += D) {
      kz[i] = make_uint4(0, 0, 0, 0);
      vz[i] = make_uint4(0, 0, 0, 0);
    }
    __syncthreads();
  }
  append_write(k_new, v_new, arena, boxes, npage_cap, page, u, T, ti, ko, vo, open_block, cert, vsq, d);
}

// One decode step's appends for up to kAppendLayers layers of one batch in one launch,
// when no sequence opens a block (the layers share B, Hkv, the block capacity and the
// lengths; the newest block of every unit is exact).  grid (Hkv, B, layers).
constexpr int kAppendLayers = GKV_APPEND_LAYERS;
struct AppendLayer {
  int64_t *koff, *voff;
  uint8_t *arena;
  uint16_t *boxes;
  float *cert;
  int64_t *seq_len;
  int64_t npage_cap;
  int32_t page;
};
struct AppendBatch {
  AppendLayer l[kAppendLayers];
  int64_t len[GKV_MAX_APPEND_UNITS];  // each sequence's length before the step (with per-sequence lengths)
};

__global__ void __launch_bounds__(128) append_layers_kernel(const uint16_t *__restrict__ k_new,
                                                            const uint16_t *__restrict__ v_new, int64_t layer_stride,
                                                            int Hkv, int nblk_cap, int64_t T_all, int ragged,
                                                            AppendBatch ab) {
  __shared__ double vsq[D];
  const int h = blockIdx.x, b = blockIdx.y, l = blockIdx.z, d = threadIdx.x;
  const AppendLayer &L = ab.l[l];
  const int64_t u = (int64_t)b * Hkv + h;
  const int64_t T = ragged ? ab.len[b] : T_all;
  if (T < 0) return;  // a retired sequence
  if (L.seq_len && h == 0 && d == 0) L.seq_len[b] = T + 1;
  const int64_t ti = u * nblk_cap + T / P;
  append_write(k_new + l * layer_stride, v_new + l * layer_stride, L.arena, L.boxes, L.npage_cap, L.page, u, T, ti,
               L.koff[ti], L.voff[ti], false, L.cert, vsq, d);
}

// Page boxes from token-major exact keys; one workgroup per 64 pages of one (b,h).
typedef _Float16 bx8 __attribute__((ext_vector_type(8)));
typedef uint32_t bw4 __attribute__((ext_vector_type(4)));
__global__ void __launch_bounds__(kThreads) boxes_kernel(const uint16_t *__restrict__ k_src, int64_t T_src,
                                                         uint16_t *boxes, int64_t npage_cap, int page, int Hkv,
                                                         int64_t page_begin, int64_t page_end,
                                                         const int64_t *seq_len) {
  __shared__ uint32_t stage[64 * D];  // [channel][page&63] (kmin | kmax << 16)
  const int h = blockIdx.y, b = blockIdx.z;
  const int64_t u = (int64_t)b * Hkv + h;
  const int64_t g0 = (page_begin >> 6) + blockIdx.x;  // box group
  const int64_t p_lo = g0 * 64;
  const uint16_t *src = k_src + u * T_src * D;
  if (seq_len) {  // only the sequence's complete pages
    const int64_t last = seq_len[b] < 0 ? 0 : seq_len[b] / page;
    page_end = page_end < last ? page_end : last;
  }
  // sixteen lanes per page, each with eight channels: sixteen 16-byte streaming row
  // loads in flight per lane, then packed fp16 minima and maxima (exact)
  constexpr int kPagesPerPass = kThreads / 16;
  const int cg = threadIdx.x & 15;
  for (int pi = threadIdx.x >> 4; pi < 64; pi += kPagesPerPass) {
    const int64_t p = p_lo + pi;
    if (p < page_begin || p >= page_end) continue;
    const _Float16 *row = (const _Float16 *)src + p * page * D + 8 * cg;
    bx8 mn, mx;
    for (int t0 = 0; t0 < page; t0 += 16) {
      bx8 v[16];
#pragma unroll
      for (int j = 0; j < 16; ++j) v[j] = __builtin_nontemporal_load((const bx8 *)(row + (int64_t)(t0 + j) * D));
      if (t0 == 0) mn = mx = v[0];
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        mn = __builtin_elementwise_min(mn, v[j]);
        mx = __builtin_elementwise_max(mx, v[j]);
      }
    }
    const bw4 lw = __builtin_bit_cast(bw4, mn), hw = __builtin_bit_cast(bw4, mx);  // channel pairs
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint16_t lo = (uint16_t)(lw[e >> 1] >> (16 * (e & 1))), hi = (uint16_t)(hw[e >> 1] >> (16 * (e & 1)));
      stage[(8 * cg + e) * 64 + pi] = (uint32_t)canon_zero(lo) | ((uint32_t)canon_zero(hi) << 16);
    }
  }
  __syncthreads();
  uint32_t *out = (uint32_t *)(boxes + u * npage_cap * 2 * D + box_index(p_lo, 0));
  for (int i = threadIdx.x; i < 64 * D; i += kThreads) {
    const int pi = i & 63;
    const int64_t p = p_lo + pi;
    if (p < page_begin || p >= page_end) continue;
    out[i] = stage[i];
  }
}

// Rate-distortion token scores (section 3.4, Eq. rdscore):
// s_t = a_t * sum_d fl(fl(v_td - v_hat_td)^2), channel-ascending, written as
// order-preserving 64-bit keys.  One wavefront per block, lane = token: the block's
// value record is staged in the wavefront's LDS (an exact record one half of its
// channels at a time) and each lane runs its token's fp64 chain.  v_hat = code *
// scale + zero and v - v_hat are exact in fp64 (all are multiples of 2^-24 below
// 2^26), so forming v_hat with one fused multiply-add gives the same value as a
// product and a sum; the square and each addition round once.  grid (nblk, Hkv, B),
// 64 threads.
//
// Staged words: chunk ck (32 codes, 4 tokens x 8 channels) holds `wpc` words; the 16
// chunks of one four-token group c = ck >> 4 are contiguous, and group c starts at
// word c * kRdGroup (4 words of padding after each group's 16 * wpc), so that the
// lanes of the 16 groups, which read the same word of their own group, fall in
// different banks.
constexpr int kRdGroup = 16 * 8 + 4;

struct RdShared {
  uint32_t w[16 * kRdGroup];  // staged record words (also the centroids as fp64)
  double2 sz[D];              // per channel: (scale, zero); the one-centroid value in .x
};

__device__ __forceinline__ double h2d(uint32_t bits16) {
  return (double)(float)__builtin_bit_cast(_Float16, (uint16_t)bits16);
}

// Stage the 256 chunks of a record, wpc words of each (chunk ck's at word
// ck * src_wpc + src_off of `src`), into the group layout: wpc 16-byte pieces a lane.
__device__ __forceinline__ void rd_stage(uint32_t *w, const uint8_t *src, int wpc, int src_wpc, int src_off,
                                         int lane) {
  const int gw = 16 * wpc;  // words of one group
  for (int i = 0; i < wpc; ++i) {
    const int w0 = (i * 64 + lane) * 4;  // staged word index without padding
    const int ck = w0 / wpc, k = w0 % wpc;
    const bw4 x = __builtin_nontemporal_load((const bw4 *)(src + ((int64_t)ck * src_wpc + src_off + k) * 4));
    *(bw4 *)(w + (w0 / gw) * kRdGroup + w0 % gw) = x;
  }
}

// This lane's code of channel d = 16 j + m (token t: group c = t >> 2, tq = t & 3):
// code n = 4 j + tq of chunk 16 c + m, at bit pos[j & 3] = code_pos(BITS, n) of its word.
template <int BITS>
__device__ __forceinline__ uint32_t rd_code(const uint32_t *wl, int j, int m, const int (&pos)[4]) {
  const uint32_t word = wl[m * BITS + 4 * j / (32 / BITS)];
  return __builtin_amdgcn_ubfe(word, (uint32_t)pos[j & 3], BITS);
}

// e += (v_d - v_hat(d))^2 over the channels, ascending.
template <class F>
__device__ __forceinline__ void rd_chain(double &e, const uint32_t (&vr)[64], F vhat) {
#pragma unroll
  for (int d = 0; d < D; ++d) {
    const double v = h2d(vr[d >> 1] >> (16 * (d & 1)));
    const double diff = v - vhat(d);
    const double sq = diff * diff;
    e = e + sq;
    // LDS reads are not hoisted past 16 channels (else the unrolled chain keeps the
    // reads of many more channels in registers)
    if ((d & 15) == 15) asm volatile("" ::: "memory");
  }
}

__global__ void __launch_bounds__(64) rd_score_kernel(const uint16_t *__restrict__ v_src,
                                                      const float *__restrict__ mass, int64_t T,
                                                      const int8_t *__restrict__ level,
                                                      const int64_t *__restrict__ voff,
                                                      const uint8_t *__restrict__ arena, int Hkv, int nblk_cap,
                                                      uint64_t *__restrict__ keys, int64_t key_stride, int vtok) {
  __shared__ __align__(16) RdShared S;
  const int blk = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int lane = threadIdx.x, c = lane >> 2, tq = lane & 3;
  const int64_t u = (int64_t)b * Hkv + h;
  const int64_t ti = u * nblk_cap + blk;
  const int64_t tok = (int64_t)blk * P + lane;
  const int64_t tr = tok < T ? tok : T - 1;  // rows past T are read as the last row, not stored
  const int lv = level[ti];
  const uint8_t *rec = arena + voff[ti];

  // this token's source row, 16 bytes at a time (cached loads: the eight loads of
  // one 128-byte line by the same lane find it in the cache)
  uint32_t vr[64];
  const bw4 *row = (const bw4 *)(v_src + (u * T + tr) * D);
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const bw4 x = row[i];
#pragma unroll
    for (int k = 0; k < 4; ++k) vr[4 * i + k] = x[k];
  }
  const double a = (double)mass[u * T + tr];

  double e = 0.0;
  const uint32_t *wl = S.w + c * kRdGroup;
  if (lv == GKV_EXACT) {  // chunk ck: 64 B; channels 16 j + m of token 4 c + tq at half 4 j + tq of chunk 16 c + m
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      if (hf) __syncthreads();
      rd_stage(S.w, rec, 8, 16, 8 * hf, lane);
      __syncthreads();
      const uint32_t *wh = wl + (tq >> 1);
      const int sh = 16 * (tq & 1);
#pragma unroll
      for (int d = 64 * hf; d < 64 * hf + 64; ++d) {
        const int j = (d >> 4) - 4 * hf, m = d & 15;
        const double v = h2d(vr[d >> 1] >> (16 * (d & 1)));
        const double diff = v - h2d(wh[m * 8 + 2 * j] >> sh);
        const double sq = diff * diff;
        e = e + sq;
        if ((d & 15) == 15) asm volatile("" ::: "memory");
      }
    }
  } else if (lv == GKV_MEAN || lv == GKV_CENTROID) {
    const uint16_t *cc = (const uint16_t *)rec;
    if (lv == GKV_MEAN) {
      for (int d = lane; d < D; d += 64) S.sz[d].x = h2d(cc[d]);
      __syncthreads();
      rd_chain(e, vr, [&](int d) { return S.sz[d].x; });
    } else {
      double *cent = (double *)S.w;  // [KC][D + 1]
      for (int i = lane; i < KC * D; i += 64) {
        const int k = i >> 7, d = i & 127;
        cent[k * (D + 1) + d] = h2d(cc[vcent_index(k, d)]);
      }
      const int id = (rec[KC * D * 2 + (lane >> 2)] >> (2 * (lane & 3))) & 3;
      __syncthreads();
      const double *ct = cent + id * (D + 1);
      rd_chain(e, vr, [&](int d) { return ct[d]; });
    }
  } else {  // int8 / int4 / int2: (scale, zero) per channel or per token, then the codes
    const uint16_t *sz = (const uint16_t *)rec;
    double s = 0.0, z = 0.0;
    if (vtok) {
      s = h2d(sz[lane]);
      z = h2d(sz[P + lane]);
    } else {
      for (int e2 = lane; e2 < D; e2 += 64) S.sz[sz_channel(GKV_VALUES, e2)] = make_double2(h2d(sz[e2]), h2d(sz[D + e2]));
    }
    int pos[4];  // bit positions of this lane's codes (the same every four channel groups j)
#pragma unroll
    for (int r = 0; r < 4; ++r) pos[r] = code_pos(lv, 4 * r + tq);
    const uint8_t *codes = rec + kSZBytes;
    if (lv == GKV_INT8) rd_stage(S.w, codes, 8, 8, 0, lane);
    else if (lv == GKV_INT4) rd_stage(S.w, codes, 4, 4, 0, lane);
    else rd_stage(S.w, codes, 2, 2, 0, lane);
    __syncthreads();
#define GKV_RD_INT(BITS)                                                                                   \
  if (vtok)                                                                                                \
    rd_chain(e, vr, [&](int d) { return __builtin_fma((double)rd_code<BITS>(wl, d >> 4, d & 15, pos), s, z); }); \
  else                                                                                                     \
    rd_chain(e, vr, [&](int d) {                                                                           \
      const double2 g = S.sz[d];                                                                           \
      return __builtin_fma((double)rd_code<BITS>(wl, d >> 4, d & 15, pos), g.x, g.y);                       \
    })
    if (lv == GKV_INT8) GKV_RD_INT(8);
    else if (lv == GKV_INT4) GKV_RD_INT(4);
    else GKV_RD_INT(2);
#undef GKV_RD_INT
  }
  if (tok < T) {
    double sc = a * e;
    sc = sc + 0.0;  // -0 -> +0
    uint64_t bits;
    __builtin_memcpy(&bits, &sc, 8);
    keys[u * key_stride + tok] = (bits >> 63) ? ~bits : (bits | 0x8000000000000000ull);
  }
}

}  // namespace

void gkv_launch_rd_score(const gkv_cache *c, const uint16_t *v_src, const float *mass, uint64_t *keys,
                         int64_t key_stride, hipStream_t stream) {
  const int nblk = (int)((c->T + P - 1) / P);
  hipLaunchKernelGGL(rd_score_kernel, dim3(nblk, c->Hkv, c->B), dim3(64), 0, stream, v_src,
                     mass, c->T, c->level, c->voff, c->arena, c->Hkv, c->nblk_cap, keys, key_stride, c->v_per_token);
}

// ---------------------------------------------------------------- C ABI
static gkv_status hip_status() { return hipGetLastError() == hipSuccess ? GKV_OK : GKV_E_HIP; }

__global__ void set_len_kernel(int64_t *seq_len, int b, int64_t v) {
  if (threadIdx.x == 0) seq_len[b] = v;
}

gkv_status gkv_launch_set_len(int64_t *seq_len, int b, int64_t v, hipStream_t stream) {
  hipLaunchKernelGGL(set_len_kernel, dim3(1), dim3(64), 0, stream, seq_len, b, v);
  return hip_status();
}

extern "C" gkv_status gkv_quantize_block(const gkv_cache *c, int32_t which, const uint16_t *src, int64_t T_src,
                                         int32_t blk_begin, int32_t blk_end, void *stream) {
  gkv_status st = gkv_validate_cache(c);
  if (st) return st;
  if (!src || (which != GKV_KEYS && which != GKV_VALUES) || T_src <= 0) return GKV_E_ARG;
  if (blk_begin < 0 || blk_end > c->nblk_cap || blk_begin > blk_end) return GKV_E_SHAPE;
  if (blk_begin == blk_end) return GKV_OK;
  for (int b = 0; b < c->B; ++b) {
    // with per-sequence lengths the sequence's own length bounds its blocks
    const int64_t Tb = c->seq_len_host ? c->seq_len_host[b] : T_src;
    if (Tb > T_src) return GKV_E_SHAPE;
    for (int h = 0; h < c->Hkv; ++h)
      for (int blk = blk_begin; blk < blk_end; ++blk) {
        if (c->seq_len_host && (int64_t)blk * P >= Tb) continue;  // not encoded
        const int lv = c->level_host[((int64_t)b * c->Hkv + h) * c->nblk_cap + blk];
        if (level_rank(lv) < 0) return GKV_E_ARG;
        if ((int64_t)(blk + 1) * P > Tb && lv != GKV_EXACT) return GKV_E_SHAPE;
        if ((int64_t)blk * P >= Tb) return GKV_E_SHAPE;
      }
  }
  dim3 grid(blk_end - blk_begin, c->Hkv, c->B);
  hipLaunchKernelGGL(quantize_kernel, grid, dim3(kThreads), sizeof(EncodeShared), (hipStream_t)stream, src,
                     T_src, c->level, which == GKV_KEYS ? c->koff : c->voff, c->arena, c->Hkv, c->nblk_cap,
                     blk_begin, which, c->cert, c->v_per_token, (const int64_t *)c->seq_len);
  return hip_status();
}

extern "C" gkv_status gkv_demote(gkv_cache *c, int32_t n, const int32_t *jobs, const int8_t *to,
                                 const int64_t *nk, const int64_t *nv, void *stream) {
  gkv_status st = gkv_validate_cache(c);
  if (st) return st;
  if (n < 0) return GKV_E_ARG;
  if (n == 0) return GKV_OK;
  if (!jobs || !to || !nk || !nv) return GKV_E_ARG;
  const int64_t nblk = (c->T + P - 1) / P;
  for (int i = 0; i < n; ++i) {
    const int b = jobs[3 * i], h = jobs[3 * i + 1], blk = jobs[3 * i + 2];
    if (b < 0 || b >= c->B || h < 0 || h >= c->Hkv || blk < 0 || blk >= nblk) return GKV_E_SHAPE;
    const int cur = c->level_host[((int64_t)b * c->Hkv + h) * c->nblk_cap + blk];
    if (level_rank(to[i]) < 0) return GKV_E_ARG;
    if (level_rank(to[i]) >= level_rank(cur)) return GKV_E_NOT_MONOTONE;
    if ((int64_t)(blk + 1) * P > seq_tokens(c, b)) return GKV_E_SHAPE;  // a partial block stays exact
    const int64_t bb = block_bytes(to[i]);
    if (nk[i] < 0 || nv[i] < 0 || nk[i] + bb > c->arena_bytes || nv[i] + bb > c->arena_bytes) return GKV_E_ARG;
    for (int j = 0; j < i; ++j)
      if (jobs[3 * j] == b && jobs[3 * j + 1] == h && jobs[3 * j + 2] == blk) return GKV_E_ARG;
  }
  for (int base = 0; base < n; base += kMaxDemoteJobs) {
    const int cnt = n - base < kMaxDemoteJobs ? n - base : kMaxDemoteJobs;
    DemoteJobs J;
    for (int i = 0; i < cnt; ++i) {
      J.b[i] = jobs[3 * (base + i)];
      J.h[i] = jobs[3 * (base + i) + 1];
      J.blk[i] = jobs[3 * (base + i) + 2];
      J.to[i] = to[base + i];
      J.cur[i] = c->level_host[((int64_t)J.b[i] * c->Hkv + J.h[i]) * c->nblk_cap + J.blk[i]];
      J.koff[i] = nk[base + i];
      J.voff[i] = nv[base + i];
    }
    hipLaunchKernelGGL(demote_kernel, dim3(cnt, 2), dim3(kThreads), sizeof(EncodeShared), (hipStream_t)stream, J,
                       c->level, c->koff, c->voff, c->arena, c->Hkv, c->nblk_cap, c->cert, c->v_per_token);
    if (hipGetLastError() != hipSuccess) return GKV_E_HIP;
  }
  for (int i = 0; i < n; ++i)
    c->level_host[((int64_t)jobs[3 * i] * c->Hkv + jobs[3 * i + 1]) * c->nblk_cap + jobs[3 * i + 2]] = to[i];
  gkv_stamp(c);
  return GKV_OK;
}

extern "C" gkv_status gkv_page_boxes(const gkv_cache *c, const uint16_t *k_src, int64_t T_src,
                                     int64_t page_begin, int64_t page_end, void *stream) {
  gkv_status st = gkv_validate_cache(c);
  if (st) return st;
  if (!c->page || !k_src) return GKV_E_ARG;
  if (page_begin < 0 || page_begin > page_end || page_end > c->npage_cap) return GKV_E_SHAPE;
  if (page_end * c->page > T_src) return GKV_E_SHAPE;
  if (page_begin == page_end) return GKV_OK;
  const int64_t g0 = page_begin >> 6, g1 = (page_end + 63) >> 6;
  dim3 grid((unsigned)(g1 - g0), c->Hkv, c->B);
  hipLaunchKernelGGL(boxes_kernel, grid, dim3(kThreads), 0, (hipStream_t)stream, k_src, T_src, c->boxes,
                     c->npage_cap, c->page, c->Hkv, page_begin, page_end, (const int64_t *)c->seq_len);
  return hip_status();
}

extern "C" gkv_status gkv_append(gkv_cache *c, const uint16_t *k_new, const uint16_t *v_new,
                                 const int64_t *new_koff, const int64_t *new_voff, void *stream) {
  gkv_status st = gkv_validate_cache(c);
  if (st) return st;
  if (!k_new || !v_new) return GKV_E_ARG;
  const int64_t units = (int64_t)c->B * c->Hkv;
  if (c->seq_len_host && c->B > GKV_MAX_APPEND_UNITS) return GKV_E_UNSUPPORTED;
  NewSlots slots;
  bool any_open = false;
  for (int b = 0; b < c->B; ++b) {
    const int64_t T = seq_tokens(c, b);
    if (c->seq_len_host) slots.len[b] = T;
    if (T < 0) continue;  // retired
    const int blk = (int)(T / P);
    if (blk >= c->nblk_cap) return GKV_E_SHAPE;
    if (c->page && (T + 1) / c->page > c->npage_cap) return GKV_E_SHAPE;
    const bool open = (T % P) == 0;
    any_open |= open;
    for (int h = 0; h < c->Hkv; ++h) {
      const int64_t u = (int64_t)b * c->Hkv + h;
      if (open) {
        if (units > GKV_MAX_APPEND_UNITS) return GKV_E_UNSUPPORTED;
        if (!new_koff || !new_voff) return GKV_E_ARG;
        if (new_koff[u] < 0 || new_voff[u] < 0 || new_koff[u] + kExactBytes > c->arena_bytes ||
            new_voff[u] + kExactBytes > c->arena_bytes)
          return GKV_E_ARG;
        slots.k[u] = new_koff[u];
        slots.v[u] = new_voff[u];
      } else if (c->level_host[u * c->nblk_cap + blk] != GKV_EXACT) {
        return GKV_E_ARG;
      }
    }
  }
  hipLaunchKernelGGL(append_kernel, dim3(c->Hkv, c->B), dim3(128), 0, (hipStream_t)stream, k_new, v_new, c->level,
                     c->koff, c->voff, c->arena, c->page ? c->boxes : nullptr, c->npage_cap, c->page ? c->page : 1,
                     c->Hkv, c->nblk_cap, c->T, c->seq_len, slots, c->cert);
  if (hipGetLastError() != hipSuccess) return GKV_E_HIP;
  gkv_append_commit(c, any_open);
  return GKV_OK;
}

// The host side of an enqueued append: the opened blocks' levels, the lengths and T.
void gkv_append_commit(gkv_cache *c, bool any_open) {
  int64_t mx = 0;
  for (int b = 0; b < c->B; ++b) {
    const int64_t T = seq_tokens(c, b);
    if (T < 0) continue;
    if (T % P == 0)
      for (int h = 0; h < c->Hkv; ++h) c->level_host[((int64_t)b * c->Hkv + h) * c->nblk_cap + T / P] = GKV_EXACT;
    if (c->seq_len_host) c->seq_len_host[b] = T + 1;
    mx = T + 1 > mx ? T + 1 : mx;
  }
  c->T = c->seq_len_host ? mx : c->T + 1;
  // the tables change only when a block opens; a dense plan covers whole blocks, and
  // the attention masks a block's tokens past the length at run time
  if (any_open) gkv_stamp(c);
}

// One launch for n <= GKV_APPEND_LAYERS layers of a step that opens no block (k_new,
// v_new: their rows, layer after layer): the caller has checked what gkv_append
// checks (same B, Hkv, capacity and lengths over the layers; every newest block
// exact; page-box capacity).  Nothing of the host state changes.
gkv_status gkv_launch_append_layers(gkv_cache *const *caches, int n, const uint16_t *k_new, const uint16_t *v_new,
                                    hipStream_t stream) {
  const gkv_cache *c0 = caches[0];
  if (n < 1 || n > kAppendLayers) return GKV_E_ARG;
  if (c0->seq_len_host && c0->B > GKV_MAX_APPEND_UNITS) return GKV_E_UNSUPPORTED;
  const int64_t stride = (int64_t)c0->B * c0->Hkv * D;
  AppendBatch ab;
  for (int i = 0; i < n; ++i) {
    const gkv_cache *c = caches[i];
    ab.l[i] = AppendLayer{c->koff, c->voff, c->arena, c->page ? c->boxes : nullptr, c->cert, c->seq_len,
                          c->npage_cap, c->page ? c->page : 1};
  }
  if (c0->seq_len_host)
    for (int b = 0; b < c0->B; ++b) ab.len[b] = c0->seq_len_host[b];
  hipLaunchKernelGGL(append_layers_kernel, dim3(c0->Hkv, c0->B, n), dim3(128), 0, stream, k_new, v_new, stride,
                     c0->Hkv, c0->nblk_cap, c0->T, c0->seq_len_host ? 1 : 0, ab);
  return hipGetLastError() == hipSuccess ? GKV_OK : GKV_E_HIP;
}
