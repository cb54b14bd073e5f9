// Mixed-precision expert cache manager (Section 3.4, "Cache Manager design",
// Eq. 3): separate caches for high- and low-precision expert copies; per
// sequence, the last-use time R, use count F and high-precision use count H
// of every expert; on a miss the incoming copy replaces the resident of the
// same cache with the lowest Eq. 3 priority
//   p_t = w_lru R_t/T + w_lfu F_t/T + w_lhu H_t/T + w_fld (1 - ((l_t - l_i + l_n) mod l_n)/l_n)
// (ties to the smaller expert key), residents masked by the predictor
// excepted.  A high-precision miss costs C, a low-precision miss
// C * B_l / B_h (Section 3.4, "Cache replacement policies").
//
// Host code: one manager is driven by the host loop that decides which copy
// of each routed expert is streamed; layer_tags() turns its state into the
// per-expert tags of moe_set_expert_precision.
#include <algorithm>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <mutex>
#include <new>
#include <set>
#include <string>
#include <vector>

#include "moe.h"

namespace moe {
void set_last_error(const char* msg);  // moe_api.cpp: the text moe_last_error returns
}

struct moe_cache {
  moe_cache_desc d;
  int64_t T = 0;
  std::vector<int64_t> R;
  std::vector<int64_t> F, H;
  std::vector<uint8_t> in_hi, in_lo, masked;
  std::vector<int32_t> hi, lo;  // resident keys
  double penalty = 0.0;
  int64_t hi_misses = 0, lo_misses = 0, hits = 0;
};

namespace {

std::mutex g_cache_mu;
std::set<moe_cache*> g_cache_live;

moe_status cfail(moe_status st, const char* fmt, ...) {
  char buf[256];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  moe::set_last_error(buf);
  return st;
}

bool live(moe_cache* c) {
  std::lock_guard<std::mutex> g(g_cache_mu);
  return c && g_cache_live.count(c) != 0;
}

// Eq. 3 for expert key t relative to layer li, in the order written.
double priority(const moe_cache* c, int32_t t, int32_t li) {
  const int32_t L = c->d.n_layers;
  const int32_t lt = t / c->d.n_experts;
  double p_lru = 0.0, p_lfu = 0.0, p_lhu = 0.0;
  if (c->T > 0) {
    const double T = (double)c->T;
    p_lru = (double)c->R[t] / T;
    p_lfu = (double)c->F[t] / T;
    p_lhu = (double)c->H[t] / T;
  }
  const double p_fld = 1.0 - (double)((lt - li + L) % L) / (double)L;
  return c->d.w_lru * p_lru + c->d.w_lfu * p_lfu + c->d.w_lhu * p_lhu + c->d.w_fld * p_fld;
}

// Index in `res` of the lowest-priority resident (unmasked ones first).
size_t victim(const moe_cache* c, const std::vector<int32_t>& res, int32_t li) {
  bool any_unmasked = false;
  for (int32_t t : res) any_unmasked |= !c->masked[t];
  size_t best = res.size();
  double bp = 0.0;
  for (size_t i = 0; i < res.size(); ++i) {
    const int32_t t = res[i];
    if (any_unmasked && c->masked[t]) continue;
    const double p = priority(c, t, li);
    if (best == res.size() || p < bp || (p == bp && t < res[best])) {
      best = i;
      bp = p;
    }
  }
  return best;
}

void use(moe_cache* c, int32_t layer, int32_t expert, bool high, int32_t* hit,
         int32_t* ev_layer, int32_t* ev_expert) {
  const int32_t t = layer * c->d.n_experts + expert;
  c->R[t] = c->T;
  c->F[t] += 1;
  if (high) c->H[t] += 1;
  std::vector<uint8_t>& in = high ? c->in_hi : c->in_lo;
  std::vector<int32_t>& res = high ? c->hi : c->lo;
  const int32_t cap = high ? c->d.hi_capacity : c->d.lo_capacity;
  if (ev_layer) *ev_layer = -1;
  if (ev_expert) *ev_expert = -1;
  if (in[t]) {
    ++c->hits;
    if (hit) *hit = 1;
    return;
  }
  if (hit) *hit = 0;
  if (high) {
    ++c->hi_misses;
    c->penalty += c->d.miss_cost;
  } else {
    ++c->lo_misses;
    c->penalty += c->d.miss_cost * (double)c->d.bits_lo / (double)c->d.bits_hi;
  }
  if (cap <= 0) return;
  if ((int32_t)res.size() >= cap) {
    const size_t v = victim(c, res, layer);
    const int32_t ev = res[v];
    in[ev] = 0;
    res[v] = res.back();
    res.pop_back();
    if (ev_layer) *ev_layer = ev / c->d.n_experts;
    if (ev_expert) *ev_expert = ev % c->d.n_experts;
  }
  res.push_back(t);
  in[t] = 1;
}

moe_status check_ix(moe_cache* c, int32_t layer, int32_t expert) {
  if (!live(c)) return cfail(MOE_ESTATE, "invalid or destroyed cache handle");
  if (layer < 0 || layer >= c->d.n_layers || expert < 0 || expert >= c->d.n_experts)
    return cfail(MOE_EINVAL, "(layer %d, expert %d) out of range", layer, expert);
  return MOE_OK;
}

}  // namespace

extern "C" {

moe_status moe_cache_create(const moe_cache_desc* desc, moe_cache_t* out) {
  moe::set_last_error("");
  if (!out) return cfail(MOE_EINVAL, "out is NULL");
  *out = nullptr;
  if (!desc) return cfail(MOE_EINVAL, "desc is NULL");
  const moe_cache_desc& d = *desc;
  if (d.n_layers < 1 || d.n_experts < 1 || (int64_t)d.n_layers * d.n_experts > (1 << 24))
    return cfail(MOE_EINVAL, "need n_layers, n_experts >= 1 and at most 2^24 experts");
  if (d.hi_capacity < 0 || d.lo_capacity < 0)
    return cfail(MOE_EINVAL, "capacities must be >= 0");
  if (d.bits_hi < 1 || d.bits_lo < 1 || d.bits_lo > d.bits_hi)
    return cfail(MOE_EINVAL, "need 1 <= bits_lo <= bits_hi");
  const double w[4] = {d.w_lru, d.w_lfu, d.w_lhu, d.w_fld};
  double sum = 0.0;
  for (double v : w) {
    if (!(v >= 0.0)) return cfail(MOE_EINVAL, "policy weights must be >= 0");
    sum += v;
  }
  if (!(sum > 0.999999 && sum < 1.000001)) return cfail(MOE_EINVAL, "policy weights must sum to 1");
  if (!(d.miss_cost >= 0.0)) return cfail(MOE_EINVAL, "miss_cost must be >= 0");
  moe_cache* c = new (std::nothrow) moe_cache();
  if (!c) return cfail(MOE_ENOMEM, "host allocation failed");
  c->d = d;
  const size_t n = (size_t)d.n_layers * d.n_experts;
  try {
    c->R.assign(n, 0);
    c->F.assign(n, 0);
    c->H.assign(n, 0);
    c->in_hi.assign(n, 0);
    c->in_lo.assign(n, 0);
    c->masked.assign(n, 0);
    c->hi.reserve(d.hi_capacity);
    c->lo.reserve(d.lo_capacity);
  } catch (...) {
    delete c;
    return cfail(MOE_ENOMEM, "host allocation failed");
  }
  {
    std::lock_guard<std::mutex> g(g_cache_mu);
    g_cache_live.insert(c);
  }
  *out = c;
  return MOE_OK;
}

moe_status moe_cache_begin_sequence(moe_cache_t c) {
  moe::set_last_error("");
  if (!live(c)) return cfail(MOE_ESTATE, "invalid or destroyed cache handle");
  c->T = 0;
  std::fill(c->R.begin(), c->R.end(), 0);
  std::fill(c->F.begin(), c->F.end(), 0);
  std::fill(c->H.begin(), c->H.end(), 0);
  return MOE_OK;
}

moe_status moe_cache_begin_token(moe_cache_t c) {
  moe::set_last_error("");
  if (!live(c)) return cfail(MOE_ESTATE, "invalid or destroyed cache handle");
  ++c->T;
  return MOE_OK;
}

moe_status moe_cache_access(moe_cache_t c, int32_t layer, int32_t expert, int32_t high,
                            int32_t* hit, int32_t* evicted_layer, int32_t* evicted_expert) {
  moe::set_last_error("");
  moe_status st = check_ix(c, layer, expert);
  if (st != MOE_OK) return st;
  use(c, layer, expert, high != 0, hit, evicted_layer, evicted_expert);
  return MOE_OK;
}

moe_status moe_cache_contains(moe_cache_t c, int32_t layer, int32_t expert, int32_t high,
                              int32_t* present) {
  moe::set_last_error("");
  moe_status st = check_ix(c, layer, expert);
  if (st != MOE_OK) return st;
  if (!present) return cfail(MOE_EINVAL, "present is NULL");
  const int32_t t = layer * c->d.n_experts + expert;
  *present = high ? c->in_hi[t] : c->in_lo[t];
  return MOE_OK;
}

moe_status moe_cache_set_mask(moe_cache_t c, int32_t layer, int32_t expert, int32_t masked) {
  moe::set_last_error("");
  moe_status st = check_ix(c, layer, expert);
  if (st != MOE_OK) return st;
  c->masked[layer * c->d.n_experts + expert] = masked ? 1 : 0;
  return MOE_OK;
}

moe_status moe_cache_clear_masks(moe_cache_t c) {
  moe::set_last_error("");
  if (!live(c)) return cfail(MOE_ESTATE, "invalid or destroyed cache handle");
  std::fill(c->masked.begin(), c->masked.end(), 0);
  return MOE_OK;
}

moe_status moe_cache_replay(moe_cache_t c, int64_t n, const int32_t* tokens,
                            const int32_t* layers, const int32_t* experts, const int32_t* highs,
                            const uint8_t* new_sequence, int32_t* hits, int32_t* evicted) {
  moe::set_last_error("");
  if (!live(c)) return cfail(MOE_ESTATE, "invalid or destroyed cache handle");
  if (n < 0) return cfail(MOE_EINVAL, "n must be >= 0");
  if (n > 0 && (!tokens || !layers || !experts || !highs))
    return cfail(MOE_EINVAL, "tokens, layers, experts and highs must not be NULL");
  for (int64_t i = 0; i < n; ++i)
    if (layers[i] < 0 || layers[i] >= c->d.n_layers || experts[i] < 0 ||
        experts[i] >= c->d.n_experts)
      return cfail(MOE_EINVAL, "use %lld: (layer %d, expert %d) out of range", (long long)i,
                   layers[i], experts[i]);
  bool have_last = false;
  int32_t last = 0;
  for (int64_t i = 0; i < n; ++i) {
    if (new_sequence && new_sequence[i]) {
      moe_cache_begin_sequence(c);
      have_last = false;
    }
    if (!have_last || tokens[i] != last) {
      ++c->T;
      last = tokens[i];
      have_last = true;
    }
    int32_t h = 0, el = -1, ee = -1;
    use(c, layers[i], experts[i], highs[i] != 0, &h, &el, &ee);
    if (hits) hits[i] = h;
    if (evicted) evicted[i] = el < 0 ? -1 : el * c->d.n_experts + ee;
  }
  return MOE_OK;
}

moe_status moe_cache_layer_tags(moe_cache_t c, int32_t layer, int32_t* tags) {
  moe::set_last_error("");
  moe_status st = check_ix(c, layer, 0);
  if (st != MOE_OK) return st;
  if (!tags) return cfail(MOE_EINVAL, "tags is NULL");
  // fp16 models pair with int4 or int2 copies, int8 models with int2
  // (Section 4.1)
  const int hi = c->d.bits_hi, lo = c->d.bits_lo;
  if (!((hi == 16 && (lo == 4 || lo == 2)) || (hi == 8 && lo == 2)))
    return cfail(MOE_EUNSUPPORTED, "layer tags need bits 16/4, 16/2 or 8/2 (got %d/%d)", hi, lo);
  const int32_t hit = hi == 8 ? MOE_TAG_INT8 : MOE_TAG_FP16;
  const int32_t miss = hi == 8 ? MOE_TAG_MISS_INT8_INT2 : lo == 4 ? MOE_TAG_MISS_INT4 : MOE_TAG_MISS_INT2;
  for (int32_t e = 0; e < c->d.n_experts; ++e)
    tags[e] = c->in_hi[layer * c->d.n_experts + e] ? hit : miss;
  return MOE_OK;
}

moe_status moe_cache_stats(moe_cache_t c, double* penalty, int64_t* hi_misses,
                           int64_t* lo_misses, int64_t* hits) {
  moe::set_last_error("");
  if (!live(c)) return cfail(MOE_ESTATE, "invalid or destroyed cache handle");
  if (penalty) *penalty = c->penalty;
  if (hi_misses) *hi_misses = c->hi_misses;
  if (lo_misses) *lo_misses = c->lo_misses;
  if (hits) *hits = c->hits;
  return MOE_OK;
}

moe_status moe_cache_destroy(moe_cache_t c) {
  moe::set_last_error("");
  if (!c) return cfail(MOE_EINVAL, "cache is NULL");
  {
    std::lock_guard<std::mutex> g(g_cache_mu);
    if (!g_cache_live.erase(c)) return cfail(MOE_ESTATE, "invalid or destroyed cache handle");
  }
  delete c;
  return MOE_OK;
}

}  // extern "C"
