// Host-only parts of libgkv: status strings, ladder profiles, the slab arena pool,
// rate accounting, the record decoder and argument validation.
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <vector>

#include "gkv_internal.h"

using namespace gkv;

extern "C" const char *gkv_strerror(gkv_status s) {
  switch (s) {
    case GKV_OK: return "ok";
    case GKV_E_ARG: return "invalid argument";
    case GKV_E_SHAPE: return "shape mismatch";
    case GKV_E_NOT_MONOTONE: return "demotion is not strictly downwards";
    case GKV_E_WORKSPACE: return "workspace too small";
    case GKV_E_HIP: return "HIP runtime error";
    case GKV_E_UNSUPPORTED: return "unsupported combination";
    case GKV_E_POOL: return "a slab pool has no free slot";
  }
  return "unknown status";
}

extern "C" int64_t gkv_block_bytes(int32_t level) { return block_bytes(level); }

// ---------------------------------------------------------------- table versions
static std::atomic<uint64_t> g_version{0};

void gkv_stamp(gkv_cache *c) { c->version = g_version.fetch_add(1, std::memory_order_relaxed) + 1; }

extern "C" void gkv_cache_changed(gkv_cache *c) {
  if (c) gkv_stamp(c);
}

extern "C" uint16_t gkv_f64_to_f16(double x) { return f64_to_f16(x); }

// ---------------------------------------------------------------- ladder (section 3.2)
extern "C" gkv_status gkv_ladder_levels(int32_t profile, int64_t T, int8_t *lv, int32_t nblk) {
  if (!lv || T < 0 || nblk < 0) return GKV_E_ARG;
  if ((T + P - 1) / P != nblk) return GKV_E_SHAPE;
  if (profile == 0) {
    for (int32_t i = 0; i < nblk; ++i) {
      const int32_t r = nblk - 1 - i;
      lv[i] = r < 4 ? GKV_EXACT : r < 12 ? GKV_INT8 : r < 24 ? GKV_INT4 : GKV_INT2;
    }
    return GKV_OK;
  }
  if (profile == 1) {
    // block i has age r = nblk - 1 - i; each level is a contiguous range of i, and
    // the ranges are written in increasing precedence (int2 < int4 < int8 <
    // centroid < exact) so that a later one overrides an earlier one
    const int64_t E = 16;
    const int64_t R = nblk > E ? nblk - E : 0;
    const int64_t b8 = E + (25 * R) / 100, b4 = E + (60 * R) / 100, nc = (10 * (int64_t)nblk) / 100;
    auto fill = [&](int64_t lo, int64_t hi, int8_t v) {
      lo = lo < 0 ? 0 : lo;
      hi = hi > nblk ? nblk : hi;
      if (hi > lo) memset(lv + lo, v, (size_t)(hi - lo));
    };
    fill(0, nblk, GKV_INT2);
    fill(nblk - b4, nblk, GKV_INT4);   // r < b4
    fill(nblk - b8, nblk, GKV_INT8);   // r < b8
    fill(0, nc, GKV_CENTROID);         // i < nc
    fill(nblk - E, nblk, GKV_EXACT);   // r < E
    return GKV_OK;
  }
  if (profile == 2) {
    for (int32_t i = 0; i < nblk; ++i) lv[i] = GKV_EXACT;
    return GKV_OK;
  }
  if (profile == 3) {  // RD-V2 base: newest 16 exact, the rest one-centroid
    for (int32_t i = 0; i < nblk; ++i) lv[i] = nblk - 1 - i < 16 ? GKV_EXACT : GKV_MEAN;
    return GKV_OK;
  }
  return GKV_E_ARG;
}

extern "C" int32_t gkv_ladder_crossings(const gkv_cache *c, int32_t profile, int64_t T_new, int32_t *jobs,
                                       int8_t *to, int32_t max_jobs) {
  gkv_status st = gkv_validate_cache(c);
  if (st) return st;
  if (!jobs || !to || max_jobs < 0 || T_new < c->T) return GKV_E_ARG;
  const int64_t grow = T_new - c->T;
  if ((c->T + grow + P - 1) / P > c->nblk_cap) return GKV_E_SHAPE;
  std::vector<int8_t> lv;
  int64_t lv_T = -1;  // the length whose ladder lv holds
  int32_t n = 0;
  for (int b = 0; b < c->B; ++b) {
    const int64_t Tb = seq_tokens(c, b);
    if (Tb < 0) continue;  // retired
    const int64_t Tb_new = Tb + grow;
    if (Tb_new != lv_T) {
      const int32_t nb_new = (int32_t)((Tb_new + P - 1) / P);
      lv.assign((size_t)nb_new + 1, 0);
      st = gkv_ladder_levels(profile, Tb_new, lv.data(), nb_new);
      if (st) return st;
      lv_T = Tb_new;
    }
    const int64_t nb_old = (Tb + P - 1) / P;
    for (int h = 0; h < c->Hkv; ++h) {
      const int8_t *cl = c->level_host + ((int64_t)b * c->Hkv + h) * c->nblk_cap;
      if (memcmp(cl, lv.data(), (size_t)nb_old) == 0) continue;  // the common case: nothing crosses
      for (int64_t i = 0; i < nb_old; ++i) {
        if ((i & 63) == 0 && i + 64 <= nb_old && memcmp(cl + i, lv.data() + i, 64) == 0) {
          i += 63;  // 64 equal levels
          continue;
        }
        const int cur = cl[i];
        if (lv[i] == cur) continue;
        if (level_rank(lv[i]) > level_rank(cur)) return GKV_E_NOT_MONOTONE;
        if (n < max_jobs) {
          jobs[3 * n] = b;
          jobs[3 * n + 1] = h;
          jobs[3 * n + 2] = (int32_t)i;
          to[n] = lv[i];
        }
        ++n;
      }
    }
  }
  return n;
}

// ---------------------------------------------------------------- slab pool
constexpr int kNLevels = 6;
static const int kLevels[kNLevels] = {GKV_EXACT, GKV_INT8, GKV_INT4, GKV_INT2, GKV_CENTROID, GKV_MEAN};
static int level_slot(int level) {
  for (int i = 0; i < kNLevels; ++i)
    if (kLevels[i] == level) return i;
  return -1;
}

struct gkv_pool {
  int64_t base[kNLevels], cap[kNLevels], bytes;
  std::vector<int64_t> free_list[kNLevels];  // slot indices, popped from the back
  std::vector<uint8_t> used[kNLevels];
  int64_t nused[kNLevels];
};

extern "C" gkv_pool *gkv_pool_create(const int64_t cap[kNLevels]) {
  if (!cap) return nullptr;
  gkv_pool *p = new gkv_pool();
  int64_t off = 0;
  for (int i = 0; i < kNLevels; ++i) {
    if (cap[i] < 0) {
      delete p;
      return nullptr;
    }
    p->base[i] = off;
    p->cap[i] = cap[i];
    off += cap[i] * block_bytes(kLevels[i]);
    off = (off + 255) & ~(int64_t)255;
    p->free_list[i].resize(cap[i]);
    for (int64_t s = 0; s < cap[i]; ++s) p->free_list[i][s] = cap[i] - 1 - s;  // lowest slot first
    p->used[i].assign(cap[i], 0);
    p->nused[i] = 0;
  }
  p->bytes = off;
  return p;
}

extern "C" int64_t gkv_pool_bytes(const gkv_pool *p) { return p ? p->bytes : -1; }

extern "C" int64_t gkv_pool_alloc(gkv_pool *p, int32_t level) {
  const int i = level_slot(level);
  if (!p || i < 0 || p->free_list[i].empty()) return -1;
  const int64_t s = p->free_list[i].back();
  p->free_list[i].pop_back();
  p->used[i][s] = 1;
  p->nused[i]++;
  return p->base[i] + s * block_bytes(level);
}

extern "C" gkv_status gkv_pool_free(gkv_pool *p, int32_t level, int64_t off) {
  const int i = level_slot(level);
  if (!p || i < 0) return GKV_E_ARG;
  const int64_t bb = block_bytes(level);
  const int64_t rel = off - p->base[i];
  if (rel < 0 || rel % bb != 0 || rel / bb >= p->cap[i]) return GKV_E_ARG;
  const int64_t s = rel / bb;
  if (!p->used[i][s]) return GKV_E_ARG;
  p->used[i][s] = 0;
  p->nused[i]--;
  p->free_list[i].push_back(s);
  return GKV_OK;
}

extern "C" int64_t gkv_pool_used(const gkv_pool *p, int32_t level) {
  const int i = level_slot(level);
  if (!p || i < 0) return -1;
  return p->nused[i];
}

extern "C" void gkv_pool_destroy(gkv_pool *p) { delete p; }

// ---------------------------------------------------------------- sequence lifecycle
extern "C" gkv_status gkv_retire_sequence(gkv_cache *c, gkv_pool *pool, const int64_t *koff_host,
                                          const int64_t *voff_host, int32_t b, void *stream) {
  gkv_status st = gkv_validate_cache(c);
  if (st) return st;
  if (!c->seq_len_host || !pool || !koff_host || !voff_host) return GKV_E_ARG;
  if (b < 0 || b >= c->B) return GKV_E_SHAPE;
  const int64_t Tb = c->seq_len_host[b];
  if (Tb < 0) return GKV_E_ARG;
  const int64_t nblk = (Tb + P - 1) / P;
  // every slot must be a used slot of its level, each listed once: checked before
  // anything changes
  std::vector<std::pair<int, int64_t>> slots;  // (level index, slot)
  for (int h = 0; h < c->Hkv; ++h)
    for (int64_t i = 0; i < nblk; ++i) {
      const int64_t e = ((int64_t)b * c->Hkv + h) * c->nblk_cap + i;
      const int li = level_slot(c->level_host[e]);
      if (li < 0) return GKV_E_ARG;
      const int64_t bb = block_bytes(kLevels[li]);
      for (const int64_t off : {koff_host[e], voff_host[e]}) {
        const int64_t rel = off - pool->base[li];
        if (rel < 0 || rel % bb != 0 || rel / bb >= pool->cap[li] || !pool->used[li][rel / bb]) return GKV_E_ARG;
        slots.emplace_back(li, rel / bb);
      }
    }
  std::vector<std::pair<int, int64_t>> sorted = slots;
  std::sort(sorted.begin(), sorted.end());
  if (std::adjacent_find(sorted.begin(), sorted.end()) != sorted.end()) return GKV_E_ARG;
  if (gkv_launch_set_len(c->seq_len, b, -1, (hipStream_t)stream) != GKV_OK) return GKV_E_HIP;
  for (const auto &sl : slots) {
    pool->used[sl.first][sl.second] = 0;
    pool->nused[sl.first]--;
    pool->free_list[sl.first].push_back(sl.second);
  }
  c->seq_len_host[b] = -1;
  int64_t mx = 0;
  for (int i = 0; i < c->B; ++i) mx = c->seq_len_host[i] > mx ? c->seq_len_host[i] : mx;
  c->T = mx;
  gkv_stamp(c);
  return GKV_OK;
}

extern "C" gkv_status gkv_admit_sequence(gkv_cache *c, int32_t b, void *stream) {
  gkv_status st = gkv_validate_cache(c);
  if (st) return st;
  if (!c->seq_len_host) return GKV_E_ARG;
  if (b < 0 || b >= c->B) return GKV_E_SHAPE;
  if (c->seq_len_host[b] != -1) return GKV_E_ARG;
  if (gkv_launch_set_len(c->seq_len, b, 0, (hipStream_t)stream) != GKV_OK) return GKV_E_HIP;
  c->seq_len_host[b] = 0;
  gkv_stamp(c);
  return GKV_OK;
}

// ---------------------------------------------------------------- validation
gkv_status gkv_validate_cache(const gkv_cache *c) {
  if (!c) return GKV_E_ARG;
  if (c->D != D) return GKV_E_SHAPE;
  if (c->B <= 0 || c->Hkv <= 0 || c->Hq <= 0 || c->Hq % c->Hkv) return GKV_E_SHAPE;
  const int G = c->Hq / c->Hkv;
  if (G < 1 || G > 16) return GKV_E_SHAPE;
  if (c->T < 0 || c->nblk_cap <= 0) return GKV_E_SHAPE;
  if ((c->T + P - 1) / P > c->nblk_cap) return GKV_E_SHAPE;
  if (!c->level || !c->koff || !c->voff || !c->arena || !c->level_host) return GKV_E_ARG;
  if (c->page) {
    if (c->page != 16 && c->page != 32 && c->page != 64) return GKV_E_SHAPE;
    if (!c->boxes || c->npage_cap <= 0 || c->npage_cap % 64) return GKV_E_ARG;
    if (c->T / c->page > c->npage_cap) return GKV_E_SHAPE;
  }
  if (!c->seq_len != !c->seq_len_host) return GKV_E_ARG;
  if (c->seq_len_host) {  // every length in [-1, T]; T the largest
    int64_t mx = 0;
    for (int b = 0; b < c->B; ++b) {
      const int64_t t = c->seq_len_host[b];
      if (t < -1 || t > c->T) return GKV_E_SHAPE;
      mx = t > mx ? t : mx;
    }
    if (mx != c->T) return GKV_E_SHAPE;
  }
  if (c->nres < 0 || c->nres > c->nres_cap) return GKV_E_SHAPE;
  if (c->nres_cap > 0 && (!c->res_idx || !c->res_rows || !c->res_mask || !c->res_off)) return GKV_E_ARG;
  if (c->v_per_token != 0 && c->v_per_token != 1) return GKV_E_ARG;
  return GKV_OK;
}

// ---------------------------------------------------------------- accounting
static int64_t row_bits(int level) {
  if (level == GKV_EXACT) return D * 16;
  if (is_int_level(level)) return (int64_t)D * level;
  if (level == GKV_CENTROID) return 2;
  return 0;
}
static int64_t overhead_bits(int level) {
  if (is_int_level(level)) return D * 2 * 16;
  if (level == GKV_CENTROID) return KC * D * 16;
  if (level == GKV_MEAN) return D * 16;
  return 0;
}

extern "C" gkv_status gkv_account(const gkv_cache *c, const int32_t *pages, int32_t topk, const int32_t *res_idx,
                                  gkv_rates *out) {
  gkv_status st = gkv_validate_cache(c);
  if (st) return st;
  if (!out) return GKV_E_ARG;
  if (pages && (!c->page || topk <= 0)) return GKV_E_ARG;
  if (pages && c->nres && !res_idx) return GKV_E_ARG;
  const int64_t box_bits = 2 * D * 16;
  int64_t resident = 0, read = 0, values = 0;
  std::vector<uint8_t> touched;
  for (int b = 0; b < c->B; ++b) {
    const int64_t T = seq_tokens(c, b);
    if (T <= 0) continue;  // retired or empty
    const int64_t nblk = (T + P - 1) / P;
    values += (int64_t)c->Hkv * T * 2 * D;
    for (int h = 0; h < c->Hkv; ++h) {
      const int8_t *lv = c->level_host + ((int64_t)b * c->Hkv + h) * c->nblk_cap;
      int64_t graded = 0;
      for (int64_t i = 0; i < nblk; ++i) graded += 2 * block_bytes(lv[i]) * 8;
      const int64_t boxes = c->page ? (T / c->page) * box_bits : 0;
      const int64_t res = c->nres ? (int64_t)c->nres * (2 * D * 16 + 32) + nblk * 64 : 0;
      resident += graded + boxes + res;
      if (!pages) {
        read += graded + res;
        continue;
      }
      const int64_t cur = (T - 1) / c->page;
      int64_t r = boxes;
      touched.assign(nblk, 0);
      const int32_t *pg = pages + ((int64_t)b * c->Hkv + h) * topk;
      std::vector<int64_t> list;
      for (int k = 0; k < topk; ++k)
        if (pg[k] >= 0 && pg[k] != cur) list.push_back(pg[k]);
      list.push_back(cur);
      std::sort(list.begin(), list.end());  // a page listed twice is read once
      list.erase(std::unique(list.begin(), list.end()), list.end());
      for (int64_t p : list) {
        const int64_t t0 = p * c->page, t1 = t0 + c->page < T ? t0 + c->page : T;
        for (int64_t t = t0; t < t1; ++t) {
          r += 2 * row_bits(lv[t / P]);
          touched[t / P] = 1;
        }
      }
      int64_t ntouched = 0;
      for (int64_t i = 0; i < nblk; ++i)
        if (touched[i]) {
          r += 2 * overhead_bits(lv[i]);
          ++ntouched;
        }
      if (c->nres) {  // the residual rows of the read tokens and the touched blocks' masks
        std::vector<uint8_t> in_read((size_t)T, 0);
        for (int64_t p : list) {
          const int64_t t0 = p * c->page, t1 = t0 + c->page < T ? t0 + c->page : T;
          for (int64_t t = t0; t < t1; ++t) in_read[t] = 1;
        }
        const int32_t *ri = res_idx + ((int64_t)b * c->Hkv + h) * c->nres_cap;
        for (int32_t k = 0; k < c->nres; ++k)
          if (ri[k] >= 0 && ri[k] < T && in_read[ri[k]]) r += 2 * D * 16 + 32;
        r += ntouched * 64;
      }
      read += r;
    }
  }
  out->resident_bits = resident;
  out->read_bits = read;
  out->values = values;
  return GKV_OK;
}

// ---------------------------------------------------------------- record decoder
extern "C" gkv_status gkv_decode_record(int32_t level, int32_t tensor, const uint8_t *rec, double *vals,
                                       int32_t *codes, uint16_t *scale, uint16_t *zero, int32_t *ids,
                                       uint16_t *cent) {
  if (!rec || !vals || (tensor != GKV_KEYS && tensor != GKV_VALUES && tensor != GKV_VALUES_PER_TOKEN))
    return GKV_E_ARG;
  if (tensor == GKV_VALUES_PER_TOKEN && is_int_level(level)) {  // scale/zero per token
    const int bits = level;
    const uint16_t *sz = (const uint16_t *)rec;
    const uint32_t *w = (const uint32_t *)(rec + kSZBytes);
    for (int pg = 0; pg < 4; ++pg)
      for (int l = 0; l < 64; ++l)
        for (int n = 0; n < 32; ++n) {
          int t, ch;
          chunk_coord(GKV_VALUES, pg, l, n, t, ch);
          const uint32_t word = w[(pg * 64 + l) * bits + code_word(bits, n)];
          const int c = (int)((word >> code_pos(bits, n)) & ((1u << bits) - 1));
          if (codes) codes[t * D + ch] = c;
          vals[t * D + ch] = (double)c * f16_to_f64(sz[t]) + f16_to_f64(sz[P + t]);
        }
    if (scale) memcpy(scale, sz, P * sizeof(uint16_t));
    if (zero) memcpy(zero, sz + P, P * sizeof(uint16_t));
    return GKV_OK;
  }
  if (tensor == GKV_VALUES_PER_TOKEN) tensor = GKV_VALUES;
  if (level == GKV_EXACT) {
    const uint16_t *h = (const uint16_t *)rec;
    for (int pg = 0; pg < 4; ++pg)
      for (int l = 0; l < 64; ++l)
        for (int n = 0; n < 32; ++n) {
          int t, ch;
          chunk_coord(tensor, pg, l, n, t, ch);
          vals[t * D + ch] = f16_to_f64(h[(pg * 64 + l) * 32 + n]);
        }
    return GKV_OK;
  }
  if (is_int_level(level)) {
    const int bits = level;
    const uint16_t *sz = (const uint16_t *)rec;
    uint16_t s[D], z[D];
    for (int e = 0; e < D; ++e) {
      const int ch = sz_channel(tensor, e);
      s[ch] = sz[e];
      z[ch] = sz[D + e];
    }
    const uint32_t *w = (const uint32_t *)(rec + kSZBytes);
    const int wpc = bits;  // 32 codes * bits / 32 bits per word
    for (int pg = 0; pg < 4; ++pg)
      for (int l = 0; l < 64; ++l)
        for (int n = 0; n < 32; ++n) {
          int t, ch;
          chunk_coord(tensor, pg, l, n, t, ch);
          const uint32_t word = w[(pg * 64 + l) * wpc + code_word(bits, n)];
          const int c = (int)((word >> code_pos(bits, n)) & ((1u << bits) - 1));
          if (codes) codes[t * D + ch] = c;
          vals[t * D + ch] = (double)c * f16_to_f64(s[ch]) + f16_to_f64(z[ch]);
        }
    if (scale) memcpy(scale, s, sizeof s);
    if (zero) memcpy(zero, z, sizeof z);
    return GKV_OK;
  }
  if (level == GKV_CENTROID) {
    const uint16_t *cc = (const uint16_t *)rec;
    uint16_t cen[KC][D];
    for (int k = 0; k < KC; ++k)
      for (int d = 0; d < D; ++d) cen[k][d] = tensor == GKV_KEYS ? cc[k * D + d] : cc[vcent_index(k, d)];
    const uint8_t *idb = rec + KC * D * 2;
    for (int t = 0; t < P; ++t) {
      const int id = (idb[t >> 2] >> (2 * (t & 3))) & 3;
      if (ids) ids[t] = id;
      for (int d = 0; d < D; ++d) vals[t * D + d] = f16_to_f64(cen[id][d]);
    }
    if (cent) memcpy(cent, cen, sizeof cen);
    return GKV_OK;
  }
  if (level == GKV_MEAN) {
    const uint16_t *cc = (const uint16_t *)rec;
    for (int t = 0; t < P; ++t) {
      if (ids) ids[t] = 0;
      for (int d = 0; d < D; ++d) vals[t * D + d] = f16_to_f64(cc[d]);
    }
    if (cent) memcpy(cent, cc, D * sizeof(uint16_t));
    return GKV_OK;
  }
  return GKV_E_ARG;
}
