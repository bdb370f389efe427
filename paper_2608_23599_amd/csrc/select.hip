// Compressed-Quest page ranking (section 3.5) and rate-distortion residual
// selection (section 3.4): scoring kernels write order-preserving 64-bit keys, a
// radix-select kernel picks the first k of the order (key descending, index
// ascending) and writes the winners in ascending index order.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gkv_internal.h"

#pragma clang fp contract(off)

using namespace gkv;

void gkv_launch_rd_score(const gkv_cache *c, const uint16_t *v_src, const float *mass, uint64_t *keys,
                         int64_t key_stride, hipStream_t stream);
int64_t gkv_attn_workspace(const gkv_cache *c, int32_t topk);

namespace {

__device__ __forceinline__ uint64_t order_key(double x) {
  x = x + 0.0;  // -0 -> +0
  uint64_t bits;
  __builtin_memcpy(&bits, &x, 8);
  return (bits >> 63) ? ~bits : (bits | 0x8000000000000000ull);
}

// Box upper bound of every ranked page for the G query heads of a KV head:
// UB_g(p) = sum_d q_gd * (q_gd >= 0 ? kmax_pd : kmin_pd), channel-ascending in fp32;
// page score = max_g UB_g.  The product of two fp16 values is exact in fp32 (22
// significant bits, magnitudes from 2^-48 to below 2^32, so neither a denormal nor an
// overflow), so each step rounds once, on the add; v_fma_mix_f32 takes both fp16
// operands as they are, with no conversion instructions.
//
// One wavefront covers 64 pages (lane = page) and G / HG of the heads; a workgroup is
// four wavefronts: 4 / HG page groups times HG head groups, whose bounds meet in LDS.
// The query is read as given (fp16 rows of 128 channels): a wavefront's heads and
// channels are uniform, so its coefficients come through the scalar cache, two
// channels per dword, and each head picks the half of a box word by the sign of its
// coefficient.  grid (ceil(npages / (64 * 4 / HG)), Hkv, B) x 256 threads.
constexpr int kScoreBatch = 32;  // box words in flight per lane
template <int G, int HG>
__global__ void __launch_bounds__(256) quest_score_kernel(const uint16_t *__restrict__ q,
                                                          const uint16_t *__restrict__ boxes, int64_t npage_cap,
                                                          int64_t npages, int Hkv, uint64_t *__restrict__ keys,
                                                          const int64_t *__restrict__ seq_len, int page) {
  constexpr int HPW = G / HG;
  __shared__ float ub[4][64];
  const int h = blockIdx.y, b = blockIdx.z;
  const int64_t u = (int64_t)b * Hkv + h;
  const int w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6)), lane = threadIdx.x & 63;
  const int hg = w % HG;
  const int64_t pg0 = ((int64_t)blockIdx.x * (4 / HG) + w / HG) * 64;
  const int64_t pg = pg0 + lane;
  const bool on = pg < npages;
  float best = 0.0f;
  if (pg0 < npages) {
    // the whole 64-page group lies inside the box capacity (a multiple of 64 pages),
    // so every lane loads; lanes past the ranked pages drop their result
    const uint32_t *bx = (const uint32_t *)(boxes + u * npage_cap * 2 * D) + (box_index(pg0, 0) >> 1) + lane;
    const uint32_t *qw = (const uint32_t *)(q + (u * G + (int64_t)hg * HPW) * D);  // this wavefront's heads
    float acc[HPW];
#pragma unroll
    for (int j = 0; j < HPW; ++j) acc[j] = 0.0f;
    for (int d0 = 0; d0 < D; d0 += kScoreBatch) {
      uint32_t pr[kScoreBatch];
#pragma unroll
      for (int e = 0; e < kScoreBatch; ++e) pr[e] = bx[(d0 + e) * 64];
#pragma unroll
      for (int e = 0; e < kScoreBatch; ++e) {
        const _Float16 lo = __builtin_bit_cast(_Float16, (uint16_t)pr[e]);          // kmin
        const _Float16 hi = __builtin_bit_cast(_Float16, (uint16_t)(pr[e] >> 16));  // kmax
#pragma unroll
        for (int j = 0; j < HPW; ++j) {
          const uint32_t q2 = qw[(j * D + d0 + e) >> 1];  // channels d0+e and its pair (d0 is even)
          const _Float16 qq = __builtin_bit_cast(_Float16, (uint16_t)((e & 1) ? q2 >> 16 : q2));
          acc[j] = __builtin_fmaf((float)qq, (float)(qq >= (_Float16)0.0f ? hi : lo), acc[j]);
        }
      }
    }
    best = acc[0];
#pragma unroll
    for (int j = 1; j < HPW; ++j) best = acc[j] > best ? acc[j] : best;
  }
  if (HG > 1) {
    ub[w][lane] = best;
    __syncthreads();
    if (hg != 0) return;
#pragma unroll
    for (int j = 1; j < HG; ++j) best = ub[w + j][lane] > best ? ub[w + j][lane] : best;
  }
  // with per-sequence lengths, pages past a sequence's own ranked pages get the key 0,
  // below every score: they rank last and the selection turns them into -1
  int64_t nown = npages;
  if (seq_len) nown = seq_len[b] > 0 ? (seq_len[b] - 1) / page : 0;
  if (on) keys[u * npage_cap + pg] = pg < nown ? order_key((double)best) : 0ull;
}

// Select the first k of the order (key desc, index asc) among keys[0..n) of one
// unit and write their indices ascending to out[0..k) (-1 padded).  With a
// per-unit limit (Compressed-Quest pages of sequences of different lengths), the
// last stage writes -1 for indices at or past the unit's limit (their keys are 0,
// so they are the last of the selection).  Optionally
// sets the selected tokens' bits in a per-64 mask.  One workgroup per unit.
//
// Long inputs are reduced in stages: the first k of the whole order all lie among
// the first k of their own slice, so a stage splits the candidates into slices of
// kSelKPT * kSelThreads, keeps the first k of each slice (one workgroup per slice,
// blockIdx.x) and writes their indices slice after slice, ascending in each; the
// candidates' order by position is then still their order by index, which is the
// tie order.  A stage reads its keys through the previous stage's index list
// (`idx`, null for the first), and the last stage, a single slice, writes the
// result.
//
// Radix select of the threshold key (the need-th largest), up to 8 bits per pass,
// with one LDS histogram that every thread adds to (a wavefront's lanes rarely share
// a digit, so its atomics seldom serialise, and the bucket counts need no reduction
// over wavefronts); then an ordered compaction: selected = key > threshold, or key ==
// threshold among the first `eq_take` such keys by index.  With KPT > 0 (n <= KPT *
// threads) thread t holds keys t * KPT + j (j < KPT) in registers; with KPT == 0
// keys are streamed from memory in 1024-key chunks.
constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;

constexpr int kSelKPT = 8;  // keys per thread held in registers (n <= 8192)
constexpr int kSelPad = 2;  // empty 8-byte words after each thread's keys in the LDS staging
constexpr int kSelStream = 8;  // keys in flight per thread in the streamed loops (a clamped index)
constexpr int kSelRank = 16;  // candidates ranked directly instead of another radix pass (<= 64)

struct SelShared {
  uint32_t hist[256];
  uint64_t prefix, pmask;
  int64_t remaining;
  int64_t wsum[kSelWaves][2];
  uint32_t wpre[kSelWaves][2];  // exclusive prefix of the wavefront totals (scan2)
  uint32_t wtot[2];
  int64_t base[2];
};

// Wavefront scans and reductions of 32-bit values by DPP row shifts within each row
// of 16 lanes and row broadcasts between rows (lane 63 ends with the total).
template <int CTRL, int ROWS>
__device__ __forceinline__ uint32_t dpp_add(uint32_t x) {
  return x + (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, ROWS, 0xF, true);
}
__device__ __forceinline__ uint32_t wave_scan(uint32_t x) {  // inclusive, lane order
  x = dpp_add<0x111, 0xF>(x);  // row_shr:1
  x = dpp_add<0x112, 0xF>(x);  // row_shr:2
  x = dpp_add<0x114, 0xF>(x);  // row_shr:4
  x = dpp_add<0x118, 0xF>(x);  // row_shr:8
  x = dpp_add<0x142, 0xA>(x);  // row_bcast:15 into rows 1, 3
  x = dpp_add<0x143, 0xC>(x);  // row_bcast:31 into rows 2, 3
  return x;
}
template <int CTRL, int ROWS>
__device__ __forceinline__ uint32_t dpp_or(uint32_t x) {
  return x | (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, ROWS, 0xF, true);
}
template <int CTRL, int ROWS>
__device__ __forceinline__ uint32_t dpp_and(uint32_t x) {  // lanes without a source keep all ones
  return x & (uint32_t)__builtin_amdgcn_update_dpp(-1, (int)x, CTRL, ROWS, 0xF, false);
}
__device__ __forceinline__ uint32_t wave_or(uint32_t x) {
  x = dpp_or<0x111, 0xF>(x);
  x = dpp_or<0x112, 0xF>(x);
  x = dpp_or<0x114, 0xF>(x);
  x = dpp_or<0x118, 0xF>(x);
  x = dpp_or<0x142, 0xA>(x);
  x = dpp_or<0x143, 0xC>(x);
  return (uint32_t)__builtin_amdgcn_readlane((int)x, 63);
}
__device__ __forceinline__ uint32_t wave_and(uint32_t x) {
  x = dpp_and<0x111, 0xF>(x);
  x = dpp_and<0x112, 0xF>(x);
  x = dpp_and<0x114, 0xF>(x);
  x = dpp_and<0x118, 0xF>(x);
  x = dpp_and<0x142, 0xA>(x);
  x = dpp_and<0x143, 0xC>(x);
  return (uint32_t)__builtin_amdgcn_readlane((int)x, 63);
}

// Exclusive scan of (a, b) over the workgroup in thread order; returns the totals.
// Counts of one pass fit in 32 bits (at most 8192 keys per workgroup pass).
__device__ __forceinline__ void scan2(SelShared &sh, int64_t &a, int64_t &b, int64_t &ta, int64_t &tb) {
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const uint32_t x = wave_scan((uint32_t)a), y = wave_scan((uint32_t)b);
  if (lane == 63) {
    sh.wsum[wv][0] = x;
    sh.wsum[wv][1] = y;
  }
  __syncthreads();
  if (wv == 0) {  // one wavefront scans the wavefront totals
    const uint32_t px = lane < kSelWaves ? (uint32_t)sh.wsum[lane][0] : 0u;
    const uint32_t py = lane < kSelWaves ? (uint32_t)sh.wsum[lane][1] : 0u;
    const uint32_t sx = wave_scan(px), sy = wave_scan(py);
    if (lane < kSelWaves) {
      sh.wpre[lane][0] = sx - px;
      sh.wpre[lane][1] = sy - py;
    }
    if (lane == 63) {
      sh.wtot[0] = sx;
      sh.wtot[1] = sy;
    }
  }
  __syncthreads();
  a = (int64_t)sh.wpre[wv][0] + x - a;
  b = (int64_t)sh.wpre[wv][1] + y - b;
  ta = sh.wtot[0];
  tb = sh.wtot[1];
  __syncthreads();
}

// The keys that match the current prefix (at most kSelRank) are gathered into LDS and
// ranked exactly by (key descending, index ascending) in one wavefront; the key of
// rank remaining - 1 becomes the threshold and `remaining` the number of keys equal
// to it still to take.  Leaves the workgroup synchronised.
template <int KPT>
__device__ __forceinline__ void small_candidates(SelShared &sh, const uint64_t *kr, const uint64_t *key, int64_t n) {
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  uint64_t *ckey = (uint64_t *)&sh.hist[0];
  int32_t *cidx = (int32_t *)(ckey + 64);
  uint32_t *cnt = (uint32_t *)(cidx + 64);
  const uint64_t pre = sh.prefix, pm = sh.pmask;
  const int64_t rem = sh.remaining;
  if (tid == 0) *cnt = 0;
  __syncthreads();
  if (KPT > 0) {
#pragma unroll
    for (int j = 0; j < (KPT > 0 ? KPT : 1); ++j) {
      const int64_t i = (int64_t)tid * KPT + j;
      if (i < n && (kr[j] & pm) == pre) {
        const uint32_t at = atomicAdd(cnt, 1u);
        ckey[at] = kr[j];
        cidx[at] = (int32_t)i;
      }
    }
  } else {
    for (int64_t i0 = tid; i0 < n; i0 += (int64_t)kSelStream * kSelThreads) {
      uint64_t kv[kSelStream];
#pragma unroll
      for (int j = 0; j < kSelStream; ++j) {
        const int64_t i = i0 + (int64_t)j * kSelThreads;
        kv[j] = key[i < n ? i : n - 1];
      }
#pragma unroll
      for (int j = 0; j < kSelStream; ++j) {
        const int64_t i = i0 + (int64_t)j * kSelThreads;
        if (i < n && (kv[j] & pm) == pre) {
          const uint32_t at = atomicAdd(cnt, 1u);
          ckey[at] = kv[j];
          cidx[at] = (int32_t)i;
        }
      }
    }
  }
  __syncthreads();
  if (wv == 0) {
    const int nc = (int)*cnt;
    const bool in = lane < nc;
    const uint64_t mk = in ? ckey[lane] : 0;
    const int32_t mi = in ? cidx[lane] : 0;
    int rank = 0;
    for (int j = 0; j < nc; ++j) {  // j is uniform: lane reads, not shuffles
      const uint64_t kj = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(mk >> 32), j) << 32) |
                          (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)mk, j);
      const int32_t ij = __builtin_amdgcn_readlane(mi, j);
      rank += kj > mk || (kj == mk && ij < mi);
    }
    const bool thr_lane = in && rank == (int)rem - 1;
    const uint64_t thr = __shfl(mk, __builtin_ctzll(__ballot(thr_lane)));
    const int above = __popcll(__ballot(in && mk > thr));
    if (lane == 0) {
      sh.prefix = thr;
      sh.pmask = ~0ull;
      sh.remaining = rem - above;
    }
  }
  __syncthreads();
}

template <int KPT>
__global__ void __launch_bounds__(kSelThreads) select_kernel(const uint64_t *__restrict__ keys, int64_t key_stride,
                                                             const int32_t *__restrict__ idx, int64_t idx_stride,
                                                             int64_t n_all, int64_t slice, int k,
                                                             int32_t *__restrict__ out, int64_t out_stride,
                                                             uint64_t *mask, int64_t mask_stride,
                                                             int64_t mask_words, const int64_t *seq_len, int Hkv,
                                                             int page, uint64_t *okeys, int64_t okey_stride) {
  __shared__ SelShared sh;
  const int64_t u = blockIdx.y, base = (int64_t)blockIdx.x * slice;
  int64_t limit = INT64_MAX;  // the unit's own ranked pages (last stage only)
  if (seq_len && gridDim.x == 1) {
    const int64_t t = seq_len[u / Hkv];
    limit = t > 0 ? (t - 1) / page : 0;
  }
  const int64_t n = n_all - base < slice ? n_all - base : slice;
  const uint64_t *key = keys + u * key_stride;
  const int32_t *ix = idx ? idx + u * idx_stride + base : nullptr;  // KPT > 0 only
  int32_t *o = out + u * out_stride + (int64_t)blockIdx.x * k;
  uint64_t *ok = okeys ? okeys + u * okey_stride + (int64_t)blockIdx.x * k : nullptr;
  uint64_t *mk = mask ? mask + u * mask_stride : nullptr;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  if (mk)
    for (int64_t i = tid; i < mask_words; i += kSelThreads) mk[i] = 0;
  const int64_t need = n < k ? n : k;
  if (gridDim.x == 1)
    for (int64_t i = need + tid; i < k; i += kSelThreads) o[i] = -1;
  if (need == 0) return;
  uint64_t kr[KPT > 0 ? KPT : 1];
  // bits that differ between keys: bytes above the highest differing byte are the
  // same in every key, so their digits are known without a pass.  Each wavefront's
  // AND and OR of its keys go to LDS before the barrier that the loads need anyway
  // (a clamped load repeats a real key, which changes neither).
  uint64_t kand = ~0ull, kor = 0;
  const auto wave_andor = [&]() {
    kand = ((uint64_t)wave_and((uint32_t)(kand >> 32)) << 32) | wave_and((uint32_t)kand);
    kor = ((uint64_t)wave_or((uint32_t)(kor >> 32)) << 32) | wave_or((uint32_t)kor);
    if (lane == 0) {
      sh.wsum[wv][0] = (int64_t)kand;
      sh.wsum[wv][1] = (int64_t)kor;
    }
  };
  for (int i = tid; i < 256; i += kSelThreads) sh.hist[i] = 0;
  int32_t tix[KPT > 0 ? KPT : 1];  // a later stage: the candidates' original indices
  if (KPT > 0) {
    // a contiguous slice (the first stage's keys, or the previous stage's winners' keys
    // in candidate order): staged through LDS with lane-contiguous loads, then each
    // thread takes its KPT consecutive keys (loads that each touch 64 scattered
    // 8-byte words took three times as long).  Each thread's KPT keys are followed by
    // kSelPad empty words, so that the 16-byte reads of eight neighbouring lanes fall
    // on distinct banks (unpadded, the lanes' 64-byte stride put a wavefront's reads
    // on two 8-byte bank pairs, and the reads took about 2 us)
    extern __shared__ uint64_t stage[];  // kSelThreads * (KPT + kSelPad) words (dynamic)
    const uint64_t *src = key + base;
    uint64_t t[KPT > 0 ? KPT : 1];
#pragma unroll
    for (int j = 0; j < KPT; ++j) {  // unconditional loads (a clamped index): all in flight at once
      const int64_t i = (int64_t)j * kSelThreads + tid;
      t[j] = src[i < n ? i : n - 1];
    }
    if (ix) {
#pragma unroll
      for (int j = 0; j < KPT; ++j) {  // this thread's candidates' indices, for the output
        const int64_t i = (int64_t)tid * KPT + j;
        tix[j] = ix[i < n ? i : n - 1];
      }
    }
#pragma unroll
    for (int j = 0; j < KPT; ++j) {
      const int i = j * kSelThreads + tid;
      stage[(i / KPT) * (KPT + kSelPad) + i % KPT] = i < n ? t[j] : 0;
      kand &= t[j];
      kor |= t[j];
    }
    wave_andor();
    __syncthreads();
#pragma unroll
    for (int j = 0; j < KPT; ++j) kr[j] = stage[tid * (KPT + kSelPad) + j];
  } else {
    for (int64_t i0 = tid; i0 < n; i0 += (int64_t)kSelStream * kSelThreads) {
#pragma unroll
      for (int j = 0; j < kSelStream; ++j) {  // a clamped load repeats a real key
        const int64_t i = i0 + (int64_t)j * kSelThreads;
        const uint64_t kv = key[i < n ? i : n - 1];
        kand &= kv;
        kor |= kv;
      }
    }
    wave_andor();
    __syncthreads();
  }
  if (wv == 0) {  // the wavefront values are combined by one wavefront (lane q reads wavefront q's)
    const uint64_t la = lane < kSelWaves ? (uint64_t)sh.wsum[lane][0] : ~0ull;
    const uint64_t lo = lane < kSelWaves ? (uint64_t)sh.wsum[lane][1] : 0ull;
    const uint64_t a = ((uint64_t)wave_and((uint32_t)(la >> 32)) << 32) | wave_and((uint32_t)la);
    const uint64_t b = ((uint64_t)wave_or((uint32_t)(lo >> 32)) << 32) | wave_or((uint32_t)lo);
    const uint64_t diff = a ^ b;
    const int hb = diff ? 63 - __builtin_clzll(diff) : -1;  // highest differing bit
    const uint64_t known = hb >= 63 ? 0ull : (~0ull << (hb + 1));
    if (lane == 0) {
      sh.prefix = a & known;
      sh.pmask = known;
      sh.remaining = need;
      sh.base[0] = hb;
    }
  }
  __syncthreads();
  // digits of up to 8 bits from the highest differing bit down (the first digit
  // spreads the keys over all its buckets)
  for (int top = (int)sh.base[0]; top >= 0; top -= 8) {
    const int shift = top >= 7 ? top - 7 : 0;
    const uint64_t dmask = (2ull << (top - shift)) - 1;
    const uint64_t pre = sh.prefix, pm = sh.pmask;
    if (KPT > 0) {
#pragma unroll
      for (int j = 0; j < KPT; ++j) {
        const int64_t i = (int64_t)tid * KPT + j;
        if (i < n && (kr[j] & pm) == pre) atomicAdd(&sh.hist[(kr[j] >> shift) & dmask], 1u);
      }
    } else {
      for (int64_t i0 = tid; i0 < n; i0 += (int64_t)kSelStream * kSelThreads) {
        uint64_t kv[kSelStream];
#pragma unroll
        for (int j = 0; j < kSelStream; ++j) {
          const int64_t i = i0 + (int64_t)j * kSelThreads;
          kv[j] = key[i < n ? i : n - 1];
        }
#pragma unroll
        for (int j = 0; j < kSelStream; ++j)
          if (i0 + (int64_t)j * kSelThreads < n && (kv[j] & pm) == pre)
            atomicAdd(&sh.hist[(kv[j] >> shift) & dmask], 1u);
      }
    }
    __syncthreads();
    // wavefront 0: suffix sums over digits (digit d counts keys with digit >= d;
    // lane l holds digits 4l..4l+3), then the digit whose suffix first reaches the
    // remaining count
    if (wv == 0) {
      uint32_t c[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        c[e] = sh.hist[4 * lane + e];
        sh.hist[4 * lane + e] = 0;  // cleared for the next pass
      }
      const uint32_t mine = c[0] + c[1] + c[2] + c[3];
      const uint32_t pref = wave_scan(mine);  // sum over lanes <= this lane
      const uint32_t incl = (uint32_t)__builtin_amdgcn_readlane((int)pref, 63) - pref + mine;  // lanes >= this one
      const int64_t rem = sh.remaining;
      uint32_t suf[5];  // suffix at digits 4l .. 4l+4
      suf[4] = incl - mine;
#pragma unroll
      for (int e = 3; e >= 0; --e) suf[e] = suf[e + 1] + c[e];
      int hit = -1;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if ((int64_t)suf[e] >= rem && (int64_t)suf[e + 1] < rem) hit = e;
      if (hit >= 0) {
        const int dig = 4 * lane + hit;
        sh.remaining = rem - suf[hit + 1];
        sh.prefix = pre | ((uint64_t)dig << shift);
        sh.pmask = pm | (dmask << shift);
        sh.base[1] = c[hit];  // keys in the chosen digit's bucket
      }
    }
    __syncthreads();
    if (shift > 0 && sh.base[1] <= kSelRank) {  // few candidates left: rank them in one wavefront
      small_candidates<KPT>(sh, kr, key, n);
      break;
    }
  }
  const uint64_t thr = sh.prefix;
  const int64_t eq_take = sh.remaining;  // keys equal to thr to take, lowest index first
  if (KPT > 0) {
    int64_t gt = 0, eq = 0;
#pragma unroll
    for (int j = 0; j < KPT; ++j) {
      if ((int64_t)tid * KPT + j < n) {
        gt += kr[j] > thr;
        eq += kr[j] == thr;
      }
    }
    int64_t tg, te;
    scan2(sh, gt, eq, tg, te);  // gt, eq: counts in the threads before this one
    int64_t pos = gt + (eq < eq_take ? eq : eq_take);
#pragma unroll
    for (int j = 0; j < KPT; ++j) {
      const int64_t i = (int64_t)tid * KPT + j;
      if (i < n) {
        const bool sel = kr[j] > thr || (kr[j] == thr && eq++ < eq_take);
        if (sel) {
          const int64_t t = ix ? (int64_t)tix[j] : base + i;
          if (ok) ok[pos] = kr[j];
          o[pos++] = t < limit ? (int32_t)t : -1;
          if (mk) atomicOr((unsigned long long *)&mk[t >> 6], 1ull << (t & 63));
        }
      }
    }
    return;
  }
  // streamed: chunks of kSelStream * kSelThreads keys, kSelStream consecutive keys per
  // thread; b0 (selected so far) and b1 (keys equal to thr so far) follow from the
  // chunks' totals, the same in every thread
  int64_t b0 = 0, b1 = 0;
  const int64_t chunk = (int64_t)kSelStream * kSelThreads;
  for (int64_t c0 = 0; c0 < n; c0 += chunk) {
    const int64_t t0 = c0 + (int64_t)tid * kSelStream;
    uint64_t kv[kSelStream];
#pragma unroll
    for (int j = 0; j < kSelStream; ++j) kv[j] = key[t0 + j < n ? t0 + j : n - 1];
    int64_t g = 0, e = 0;
#pragma unroll
    for (int j = 0; j < kSelStream; ++j)
      if (t0 + j < n) {
        g += kv[j] > thr;
        e += kv[j] == thr;
      }
    int64_t tg, te;
    scan2(sh, g, e, tg, te);  // g, e: counts in the chunk's threads before this one
    const int64_t left = eq_take - b1 > 0 ? eq_take - b1 : 0;  // equal keys still to take
    int64_t pos = b0 + g + (e < left ? e : left);
#pragma unroll
    for (int j = 0; j < kSelStream; ++j) {
      const int64_t i = t0 + j;
      if (i < n) {
        const bool sel = kv[j] > thr || (kv[j] == thr && e++ < left);
        if (sel) {
          o[pos++] = i < limit ? (int32_t)i : -1;
          if (mk) atomicOr((unsigned long long *)&mk[i >> 6], 1ull << (i & 63));
        }
      }
    }
    b0 += tg + (te < left ? te : left);
    b1 += te;
  }
}

constexpr int64_t kSelSlice = (int64_t)kSelKPT * kSelThreads;
constexpr size_t kSelStageBytes = (size_t)kSelThreads * (kSelKPT + kSelPad) * 8;  // the LDS staging of one slice
// Entries per unit of a stage's winners' key list: a stage keeps at most k of every
// slice with 2k <= kSelSlice, so at most n / 2 + kSelSlice / 2 of n candidates.
static int64_t sel_ckey_stride(int64_t key_stride) { return key_stride / 2 + kSelSlice / 2; }

// idx_ws: two index lists of `key_stride` entries per unit (the stages' candidates),
// then two key lists of sel_ckey_stride(key_stride) entries per unit (their keys).
// seq_len, Hkv, page: the per-unit limit of Compressed-Quest pages (seq_len null: none).
void launch_select(const uint64_t *keys, int64_t key_stride, int64_t n, int k, int32_t *out, int64_t out_stride,
                   uint64_t *mask, int64_t mask_stride, int64_t mask_words, int units, int32_t *idx_ws,
                   hipStream_t s, const int64_t *seq_len = nullptr, int Hkv = 1, int page = 1) {
  if (n > kSelSlice && 2 * (int64_t)k > kSelSlice) {  // too few candidates dropped per stage: one streamed pass
    hipLaunchKernelGGL(select_kernel<0>, dim3(1, units), dim3(kSelThreads), 0, s, keys, key_stride,
                       (const int32_t *)nullptr, (int64_t)0, n, n, k, out, out_stride, mask, mask_stride, mask_words,
                       seq_len, Hkv, page, (uint64_t *)nullptr, (int64_t)0);
    return;
  }
  const int32_t *idx = nullptr;
  const uint64_t *kin = keys;
  int64_t kin_stride = key_stride, cur = n;
  const int64_t cks = sel_ckey_stride(key_stride);
  uint64_t *ckeys = (uint64_t *)(idx_ws + 2 * (int64_t)units * key_stride);
  for (int buf = 0; cur > kSelSlice; buf ^= 1) {
    const int64_t S = (cur + kSelSlice - 1) / kSelSlice;
    int32_t *dst = idx_ws + (int64_t)buf * units * key_stride;
    uint64_t *kdst = ckeys + (int64_t)buf * units * cks;
    hipLaunchKernelGGL(select_kernel<kSelKPT>, dim3((unsigned)S, units), dim3(kSelThreads), kSelStageBytes, s, kin,
                       kin_stride, idx, key_stride, cur, kSelSlice, k, dst, key_stride, (uint64_t *)nullptr,
                       (int64_t)0, (int64_t)0, seq_len, Hkv, page, kdst, cks);
    const int64_t last = cur - (S - 1) * kSelSlice;
    cur = (S - 1) * k + (last < k ? last : k);
    idx = dst;
    kin = kdst;
    kin_stride = cks;
  }
  hipLaunchKernelGGL(select_kernel<kSelKPT>, dim3(1, units), dim3(kSelThreads), kSelStageBytes, s, kin, kin_stride,
                     idx, key_stride, cur, cur, k, out, out_stride, mask, mask_stride, mask_words, seq_len, Hkv, page,
                     (uint64_t *)nullptr, (int64_t)0);
}

// Copy the exact key/value rows of the selected residual tokens into exact-format
// pseudo-blocks.  grid (ceil(nkeep/64), Hkv, B), 256 threads.  Rows are read 16 bytes
// (8 channels) at a time; a key record takes 8 consecutive channels of a row as one
// 16-byte piece of a chunk, so keys are written straight from the loads; a value chunk
// holds 4 rows x 8 channels 16 apart, so the value rows are staged in LDS and every
// thread writes one whole 64-byte chunk.
__global__ void __launch_bounds__(256) res_gather_kernel(const uint16_t *__restrict__ k_src,
                                                         const uint16_t *__restrict__ v_src, int64_t T,
                                                         const int32_t *__restrict__ res_idx, int nres_cap,
                                                         int nkeep, uint8_t *res_rows, int Hkv) {
  constexpr int kRow = D + 8;  // padded LDS row (halves)
  __shared__ __align__(16) uint16_t sv[P * kRow];
  const int rb = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int64_t u = (int64_t)b * Hkv + h;
  const int nrb = (nres_cap + P - 1) / P;
  uint16_t *kr = (uint16_t *)(res_rows + (u * nrb + rb) * (2 * kExactBytes));
  uint16_t *vr = kr + kExactBytes / 2;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int pc = threadIdx.x + 256 * k, slot = pc >> 4, a = pc & 15;  // channels 8a .. 8a+7 of row slot
    const int r = rb * P + slot;
    uint4 kv = make_uint4(0, 0, 0, 0), vv = kv;
    if (r < nkeep) {
      const int64_t row = (u * T + res_idx[u * nres_cap + r]) * D + 8 * a;
      kv = *(const uint4 *)(k_src + row);
      vv = *(const uint4 *)(v_src + row);
    }
    // key chunk (page slot >> 4, lane (a & 3) * 16 + (slot & 15)), codes 8 (a >> 2) ..
    const int lane = (a & 3) * 16 + (slot & 15);
    *(uint4 *)(kr + ((slot >> 4) * 64 + lane) * 32 + 8 * (a >> 2)) = kv;
    *(uint4 *)(sv + slot * kRow + 8 * a) = vv;
  }
  __syncthreads();
  // value chunk ck = (page, lane kg * 16 + m): element n is row 16 page + 4 kg + (n & 3),
  // channel 16 (n >> 2) + m
  const int ck = threadIdx.x, pg = ck >> 6, kg = (ck >> 4) & 3, m = ck & 15;
  const uint16_t *s0 = sv + (16 * pg + 4 * kg) * kRow + m;
  uint32_t w[16];
#pragma unroll
  for (int n = 0; n < 32; n += 2)
    w[n >> 1] = (uint32_t)s0[(n & 3) * kRow + 16 * (n >> 2)] | ((uint32_t)s0[((n + 1) & 3) * kRow + 16 * ((n + 1) >> 2)] << 16);
  uint4 *o = (uint4 *)(vr + ck * 32);
#pragma unroll
  for (int q = 0; q < 4; ++q) o[q] = make_uint4(w[4 * q], w[4 * q + 1], w[4 * q + 2], w[4 * q + 3]);
}

// Residual rows before every block (res_off[blk] = sum over blocks < blk of the
// mask's population count), for blocks 0 .. nblk_cap: a read that finds token t of
// block blk in the mask finds its row at res_off[blk] + popcount(mask below t).
// One workgroup per (b, KV head).
__global__ void __launch_bounds__(256) res_off_kernel(const uint64_t *__restrict__ res_mask, int nblk_cap,
                                                      int32_t *__restrict__ res_off) {
  __shared__ int32_t part[256];
  const int64_t u = blockIdx.x;
  const uint64_t *m = res_mask + u * nblk_cap;
  int32_t *o = res_off + u * (nblk_cap + 1);
  const int per = (nblk_cap + 255) / 256;
  const int b0 = threadIdx.x * per, b1 = b0 + per < nblk_cap ? b0 + per : nblk_cap;
  int32_t c = 0;
  for (int b = b0; b < b1; ++b) c += __popcll(m[b]);
  part[threadIdx.x] = c;
  __syncthreads();
  if (threadIdx.x == 0) {  // exclusive scan of the 256 partial counts
    int32_t run = 0;
    for (int i = 0; i < 256; ++i) {
      const int32_t x = part[i];
      part[i] = run;
      run += x;
    }
    o[nblk_cap] = run;
  }
  __syncthreads();
  int32_t run = part[threadIdx.x];
  for (int b = b0; b < b1; ++b) {
    o[b] = run;
    run += __popcll(m[b]);
  }
}

}  // namespace

// ---------------------------------------------------------------- C ABI
// keys (8 bytes) and two candidate index lists (4 bytes each) per ranked item, then the
// two key lists of the selection stages
static int64_t quest_ws(const gkv_cache *c) {
  return (int64_t)c->B * c->Hkv * (c->npage_cap * 16 + 2 * sel_ckey_stride(c->npage_cap) * 8);
}
// the residual selection's keys and lists are strided by the block capacity in tokens,
// so that one workspace serves the cache at any length
static int64_t rd_stride(const gkv_cache *c) { return (int64_t)c->nblk_cap * P; }
static int64_t rd_ws(const gkv_cache *c) {
  return (int64_t)c->B * c->Hkv * (rd_stride(c) * 16 + 2 * sel_ckey_stride(rd_stride(c)) * 8);
}

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
  if ((uintptr_t)q & 3) return GKV_E_ARG;  // read two channels per dword
  if (!c->page) return GKV_E_ARG;
  if (c->T <= 0) return GKV_E_SHAPE;
  if (ws_bytes < quest_ws(c)) return GKV_E_WORKSPACE;
  const int G = c->Hq / c->Hkv;
  const int64_t ncur = (c->T - 1) / c->page;  // ranked pages
  if (ncur > c->npage_cap) return GKV_E_SHAPE;
  hipStream_t s = (hipStream_t)stream;
  uint64_t *keys = (uint64_t *)ws;
  if (ncur > 0) {
    // two head groups per page group (a wavefront then does half the arithmetic and the
    // box words its sibling also reads come from the cache), four when that still
    // leaves fewer than four wavefronts per compute unit
    const int64_t groups = (int64_t)c->B * c->Hkv * ((ncur + 63) / 64);
    int HG = G % 2 == 0 ? 2 : 1;
    if (G % 4 == 0 && groups * 2 < 4 * (int64_t)gkv_device_cus()) HG = 4;
    const int per = 4 / HG;  // page groups per workgroup
    dim3 grid((unsigned)(((ncur + 63) / 64 + per - 1) / per), c->Hkv, c->B);
    switch (G * 4 + HG - 1) {
#define GKV_SCORE(g, hg)                                                                                          \
  case g * 4 + hg - 1:                                                                                            \
    hipLaunchKernelGGL((quest_score_kernel<g, hg>), grid, dim3(256), 0, s, q, c->boxes, c->npage_cap, ncur, c->Hkv, \
                       keys, (const int64_t *)c->seq_len, c->page);                                               \
    break;
      GKV_SCORE(1, 1) GKV_SCORE(3, 1) GKV_SCORE(5, 1) GKV_SCORE(7, 1) GKV_SCORE(9, 1) GKV_SCORE(11, 1)
      GKV_SCORE(13, 1) GKV_SCORE(15, 1)
      GKV_SCORE(2, 2) GKV_SCORE(4, 2) GKV_SCORE(6, 2) GKV_SCORE(8, 2) GKV_SCORE(10, 2) GKV_SCORE(12, 2)
      GKV_SCORE(14, 2) GKV_SCORE(16, 2)
      GKV_SCORE(4, 4) GKV_SCORE(8, 4) GKV_SCORE(12, 4) GKV_SCORE(16, 4)
#undef GKV_SCORE
      default: return GKV_E_SHAPE;
    }
  }
  int32_t *idx_ws = (int32_t *)(keys + (int64_t)c->B * c->Hkv * c->npage_cap);
  launch_select((const uint64_t *)keys, c->npage_cap, ncur, topk, pages, (int64_t)topk, nullptr, 0, 0, c->B * c->Hkv,
                idx_ws, s, (const int64_t *)c->seq_len, c->Hkv, c->page);
  return hipGetLastError() == hipSuccess ? GKV_OK : GKV_E_HIP;
}

extern "C" gkv_status gkv_rd_residual_select(gkv_cache *c, const uint16_t *k_src, const uint16_t *v_src,
                                             const float *mass, int32_t nkeep, void *ws, int64_t ws_bytes,
                                             void *stream) {
  gkv_status st = gkv_validate_cache(c);
  if (st) return st;
  if (!k_src || !v_src || !mass || !ws || nkeep < 0) return GKV_E_ARG;
  if (((uintptr_t)k_src | (uintptr_t)v_src) & 15) return GKV_E_ARG;  // 16-byte row loads
  if (c->seq_len_host) return GKV_E_UNSUPPORTED;  // prefill-time selection on one length
  if (c->T <= 0) return GKV_E_SHAPE;
  if (nkeep > c->nres_cap || nkeep > c->T) return GKV_E_SHAPE;
  if (ws_bytes < rd_ws(c)) return GKV_E_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  uint64_t *keys = (uint64_t *)ws;
  const int64_t stride = rd_stride(c);
  if (nkeep > 0) gkv_launch_rd_score(c, v_src, mass, keys, stride, s);
  int32_t *idx_ws = (int32_t *)(keys + (int64_t)c->B * c->Hkv * stride);
  launch_select((const uint64_t *)keys, stride, c->T, nkeep, c->res_idx, (int64_t)c->nres_cap, c->res_mask,
                (int64_t)c->nblk_cap, (int64_t)c->nblk_cap, c->B * c->Hkv, idx_ws, s);
  if (nkeep > 0) {
    dim3 g2((unsigned)((nkeep + P - 1) / P), c->Hkv, c->B);
    hipLaunchKernelGGL(res_gather_kernel, g2, dim3(256), 0, s, k_src, v_src, c->T, (const int32_t *)c->res_idx,
                       c->nres_cap, nkeep, c->res_rows, c->Hkv);
  }
  if (c->nres_cap > 0)
    hipLaunchKernelGGL(res_off_kernel, dim3(c->B * c->Hkv), dim3(256), 0, s, (const uint64_t *)c->res_mask,
                       c->nblk_cap, c->res_off);
  if (hipGetLastError() != hipSuccess) return GKV_E_HIP;
  c->nres = nkeep;
  gkv_stamp(c);
  return GKV_OK;
}
