// Multi-layer decode-step maintenance: the paged append service around the cache
// calls (section 3.2 incremental append and monotone demotion, run for every layer
// of a model by one host call, as a serving block manager does).
//
// The layers share B, Hkv and T; each layer's ladder crossings are computed from its
// own levels (layers laid out by the section 3.3 allocator hold different levels).
// Every slot the step needs (new exact blocks, demotion targets) is taken from the
// layers' pools, and checked against each layer's arena, before anything is
// enqueued, so a full pool or a bad arena fails the call without side effects.
#include <string.h>

#include <vector>

#include "gkv_internal.h"

using namespace gkv;

namespace {

struct Taken {  // slots taken for one layer, released again on failure
  gkv_pool *pool;
  std::vector<std::pair<int32_t, int64_t>> slots;
  bool take(int32_t level, int64_t &off) {
    off = gkv_pool_alloc(pool, level);
    if (off < 0) return false;
    slots.emplace_back(level, off);
    return true;
  }
  void give_back() {
    for (auto &s : slots) gkv_pool_free(pool, s.first, s.second);
    slots.clear();
  }
  // every slot lies inside an arena of `bytes`
  bool fits(int64_t bytes) const {
    for (auto &s : slots)
      if (s.second < 0 || s.second + block_bytes(s.first) > bytes) return false;
    return true;
  }
};

struct Crossings {  // one layer's demotions at T + 1
  std::vector<int32_t> jobs;
  std::vector<int8_t> to;
  int32_t n = 0;
};

}  // namespace

extern "C" int32_t gkv_layers_step(gkv_cache *const *caches, gkv_pool *const *pools, int64_t *const *koff_host,
                                   int64_t *const *voff_host, int32_t L, int32_t profile, const uint16_t *k_new,
                                   const uint16_t *v_new, void *stream) {
  if (!caches || !pools || !koff_host || !voff_host || L < 1 || !k_new || !v_new) return GKV_E_ARG;
  for (int l = 0; l < L; ++l) {
    if (!caches[l] || !pools[l] || !koff_host[l] || !voff_host[l]) return GKV_E_ARG;
    const gkv_status st = gkv_validate_cache(caches[l]);
    if (st) return st;
    const gkv_cache *c0 = caches[0], *c = caches[l];
    if (c->B != c0->B || c->Hkv != c0->Hkv || c->T != c0->T || c->nblk_cap != c0->nblk_cap) return GKV_E_SHAPE;
    if (!c->seq_len_host != !c0->seq_len_host) return GKV_E_SHAPE;
    if (c->seq_len_host)  // the layers of one batch hold the same sequences
      for (int b = 0; b < c->B; ++b)
        if (c->seq_len_host[b] != c0->seq_len_host[b]) return GKV_E_SHAPE;
  }
  const gkv_cache *c0 = caches[0];
  const int64_t units = (int64_t)c0->B * c0->Hkv, cap = c0->nblk_cap;
  // the block each unit writes into, and whether the token opens it (per sequence)
  std::vector<int64_t> ublk(units, -1);
  std::vector<char> uopen(units, 0);
  bool any_open = false;
  for (int b = 0; b < c0->B; ++b) {
    const int64_t Tb = seq_tokens(c0, b);
    if (Tb < 0) continue;  // retired
    if (Tb / P >= cap) return GKV_E_SHAPE;
    for (int h = 0; h < c0->Hkv; ++h) {
      ublk[(int64_t)b * c0->Hkv + h] = Tb / P;
      uopen[(int64_t)b * c0->Hkv + h] = Tb % P == 0;
    }
    any_open |= Tb % P == 0;
  }
  // what gkv_append would reject, rejected here before any slot is taken
  if (any_open && units > GKV_MAX_APPEND_UNITS) return GKV_E_UNSUPPORTED;
  if (c0->seq_len_host && c0->B > GKV_MAX_APPEND_UNITS) return GKV_E_UNSUPPORTED;
  for (int l = 0; l < L; ++l) {
    const gkv_cache *c = caches[l];
    for (int b = 0; b < c->B; ++b) {
      const int64_t Tb = seq_tokens(c, b);
      if (Tb >= 0 && c->page && (Tb + 1) / c->page > c->npage_cap) return GKV_E_SHAPE;
    }
    for (int64_t u = 0; u < units; ++u)
      if (ublk[u] >= 0 && !uopen[u] && c->level_host[u * cap + ublk[u]] != GKV_EXACT) return GKV_E_ARG;
  }
  const int64_t T = c0->T;
  // every layer's crossings of T + 1 (the block the token opens never crosses); a
  // layer whose levels the profile would raise fails the call here
  std::vector<Crossings> cr(L);
  for (int l = 0; l < L; ++l) {
    int32_t none_j[3];
    int8_t none_t[1];
    const int32_t n = gkv_ladder_crossings(caches[l], profile, T + 1, none_j, none_t, 0);  // the count only
    if (n < 0) return n;
    cr[l].n = n;
    cr[l].jobs.resize(3 * (size_t)n + 3);
    cr[l].to.resize((size_t)n + 1);
    if (n) {
      const int32_t m = gkv_ladder_crossings(caches[l], profile, T + 1, cr[l].jobs.data(), cr[l].to.data(), n);
      if (m != n) return m < 0 ? m : GKV_E_ARG;
    }
  }
  // every slot of the step, before anything is enqueued
  std::vector<Taken> taken(L);
  std::vector<std::vector<int64_t>> nk(L), nv(L), dk(L), dv(L);
  auto give_back_from = [&](int l0) {
    for (int j = l0; j < L; ++j) taken[j].give_back();
  };
  for (int l = 0; l < L; ++l) {
    taken[l].pool = pools[l];
    bool ok = true;
    if (any_open) {
      nk[l].assign(units, -1);
      nv[l].assign(units, -1);
      for (int64_t u = 0; u < units && ok; ++u)
        if (uopen[u]) ok = taken[l].take(GKV_EXACT, nk[l][u]) && taken[l].take(GKV_EXACT, nv[l][u]);
    }
    const int32_t n = cr[l].n;
    dk[l].resize(n);
    dv[l].resize(n);
    for (int32_t i = 0; i < n && ok; ++i)
      ok = taken[l].take(cr[l].to[i], dk[l][i]) && taken[l].take(cr[l].to[i], dv[l][i]);
    if (!ok) {
      give_back_from(0);
      return GKV_E_POOL;
    }
    if (!taken[l].fits(caches[l]->arena_bytes)) {  // a pool larger than the layer's arena
      give_back_from(0);
      return GKV_E_ARG;
    }
  }
  if (!any_open) {  // no block opens: one launch appends the token of up to 16 layers
    const size_t row = (size_t)units * D;
    for (int l0 = 0; l0 < L; l0 += GKV_APPEND_LAYERS) {
      const int n = L - l0 < GKV_APPEND_LAYERS ? L - l0 : GKV_APPEND_LAYERS;
      const gkv_status st =
          gkv_launch_append_layers(caches + l0, n, k_new + l0 * row, v_new + l0 * row, (hipStream_t)stream);
      if (st) {  // the layers before l0 are appended (not yet demoted); the others are not
        for (int l = 0; l < l0; ++l) gkv_append_commit(caches[l], false);
        give_back_from(0);
        return st;
      }
    }
    for (int l = 0; l < L; ++l) gkv_append_commit(caches[l], false);
  }
  int32_t total = 0;
  for (int l = 0; l < L; ++l) {
    gkv_cache *c = caches[l];
    const size_t row = (size_t)units * D;
    const int32_t n = cr[l].n;
    const int32_t *jobs = cr[l].jobs.data();
    const int8_t *to = cr[l].to.data();
    gkv_status st = any_open ? gkv_append(c, k_new + l * row, v_new + l * row, nk[l].data(), nv[l].data(), stream)
                             : GKV_OK;
    if (st) {  // layers before l are stepped; nothing of layer l or later is
      give_back_from(l);
      return st;
    }
    for (int64_t u = 0; u < units; ++u)
      if (uopen[u]) {
        koff_host[l][u * cap + ublk[u]] = nk[l][u];
        voff_host[l][u * cap + ublk[u]] = nv[l][u];
      }
    total += n;
    if (!n) continue;
    // the current slots of the crossing blocks are free once the stream has passed
    // the demotion (later work on this stream that reuses them is ordered after it)
    std::vector<int8_t> from(n);
    std::vector<int64_t> ok_(n), ov_(n);
    for (int32_t i = 0; i < n; ++i) {
      const int64_t idx = ((int64_t)jobs[3 * i] * c->Hkv + jobs[3 * i + 1]) * cap + jobs[3 * i + 2];
      from[i] = c->level_host[idx];
      ok_[i] = koff_host[l][idx];
      ov_[i] = voff_host[l][idx];
    }
    st = gkv_demote(c, n, jobs, to, dk[l].data(), dv[l].data(), stream);
    if (st) {  // layer l is appended but not demoted: its demotion slots go back too
      for (int32_t i = 0; i < n; ++i) {
        gkv_pool_free(pools[l], to[i], dk[l][i]);
        gkv_pool_free(pools[l], to[i], dv[l][i]);
      }
      give_back_from(l + 1);
      return st;
    }
    for (int32_t i = 0; i < n; ++i) {
      const int64_t idx = ((int64_t)jobs[3 * i] * c->Hkv + jobs[3 * i + 1]) * cap + jobs[3 * i + 2];
      koff_host[l][idx] = dk[l][i];
      voff_host[l][idx] = dv[l][i];
      gkv_pool_free(pools[l], from[i], ok_[i]);
      gkv_pool_free(pools[l], from[i], ov_[i]);
    }
  }
  return total;
}
