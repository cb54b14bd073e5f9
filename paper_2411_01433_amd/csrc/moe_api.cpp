// Host runtime behind include/moe.h: argument validation, handle registry,
// workspace, expert table and the launch sequence of one layer call.
#include "moe.h"

#include <hip/hip_runtime.h>

#include <array>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <set>
#include <string>
#include <vector>

#include "moe_internal.h"

using namespace moe;

namespace {

thread_local std::string g_err;

moe_status fail(moe_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

moe_status hip_fail(hipError_t e, const char* what) {
  return fail(MOE_EHIP, "%s: %s", what, hipGetErrorString(e));
}

#define HIP_TRY(expr, what)                    \
  do {                                         \
    hipError_t e_ = (expr);                    \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Copy slot of a quantised bit width: 4, 2 (low copies), 8 (int8 high copy).
int slot_of_bits(int bits) { return bits == 4 ? 0 : bits == 2 ? 1 : 2; }

// Bit widths a tag's copies need: the low copy (4, 2 or 0) and the high
// copy (16: the borrowed fp16 weights, 8: an int8 copy, 0: none).
int low_bits_of(int tag) {
  return (tag == MOE_TAG_INT4 || tag == MOE_TAG_MISS_INT4) ? 4
         : (tag == MOE_TAG_INT2 || tag == MOE_TAG_MISS_INT2 || tag == MOE_TAG_MISS_INT8_INT2) ? 2
                                                                                             : 0;
}
int high_bits_of(int tag) {
  if (tag == MOE_TAG_INT8 || tag == MOE_TAG_MISS_INT8_INT2) return 8;
  return (tag == MOE_TAG_FP16 || tag == MOE_TAG_MISS_INT4 || tag == MOE_TAG_MISS_INT2) ? 16 : 0;
}

}  // namespace

struct moe_layer {
  moe_layer_desc desc;
  int device = -1;
  const f16* w_router = nullptr;
  std::vector<ExpertEntry> host_table;
  // library-owned quantised copies: [expert][slot_of_bits(bits)][matrix]
  std::vector<void*> owned;
  std::vector<std::array<std::array<uint8_t*, 3>, 3>> low_q;
  std::vector<std::array<std::array<f16*, 3>, 3>> low_s;
  // the fp16 matrix each copy was quantised from (an expert re-bound to
  // other fp16 weights gets its copies rebuilt)
  std::vector<std::array<std::array<const f16*, 3>, 3>> low_src;
  // device memory
  ExpertEntry* d_table = nullptr;
  Workspace ws;             // carved from the arena, sized for max_tokens
  void* arena = nullptr;    // the table and, unless shared, the workspace
  // workspace sharing (stacks): the layer whose workspace this one runs on,
  // and how many layers run on this one's
  moe_layer* ws_owner = nullptr;
  int ws_sharers = 0;
  // stage timing (measurement only): 5 events per recorded call
  bool timing = false;
  std::vector<hipEvent_t> ev_pool;
  size_t ev_used = 0;
};

namespace {

std::mutex g_mu;
std::set<moe_layer*> g_live;

bool live(moe_layer* l) {
  std::lock_guard<std::mutex> g(g_mu);
  return g_live.count(l) != 0;
}

moe_status check_desc(const moe_layer_desc* d) {
  if (!d) return fail(MOE_EINVAL, "desc is NULL");
  if (d->group_size != kGroup) return fail(MOE_EINVAL, "group_size must be 32 (got %d)", d->group_size);
  if (d->d_model <= 0 || d->d_model % 64 || d->d_model > 16384)
    return fail(MOE_EINVAL, "d_model must be a positive multiple of 64, <= 16384 (got %d)", d->d_model);
  if (d->d_ff <= 0 || d->d_ff % 64 || d->d_ff > 65536)
    return fail(MOE_EINVAL, "d_ff must be a positive multiple of 64, <= 65536 (got %d)", d->d_ff);
  if (d->n_experts < 1 || d->n_experts > kMaxExperts)
    return fail(MOE_EINVAL, "n_experts must be in [1, 64] (got %d)", d->n_experts);
  if (d->top_k < 1 || d->top_k > kMaxTopK || d->top_k > d->n_experts)
    return fail(MOE_EINVAL, "top_k must be in [1, min(8, n_experts)] (got %d)", d->top_k);
  if (d->max_tokens < 1 || d->max_tokens > 8192)
    return fail(MOE_EINVAL, "max_tokens must be in [1, 8192] (got %d)", d->max_tokens);
  if (!(d->t1 == d->t1) || !(d->t2 == d->t2) || !(d->rms_eps >= 0.0f))
    return fail(MOE_EINVAL, "t1, t2 must be numbers and rms_eps >= 0");
  if (d->flags != 0) return fail(MOE_EINVAL, "flags must be 0");
  return MOE_OK;
}

moe_status check_call(moe_layer* l, int32_t n_tokens, int32_t limit,
                      const void* x, const void* out0, const void* out1) {
  if (!l || !live(l)) return fail(MOE_ESTATE, "invalid or destroyed layer handle");
  if (n_tokens < 1 || n_tokens > limit)
    return fail(MOE_EINVAL, "n_tokens must be in [1, %d] (got %d)", limit, n_tokens);
  if (!x || !out0) return fail(MOE_EINVAL, "x and the output must not be NULL");
  if (!aligned16(x) || !aligned16(out0) || (out1 && !aligned16(out1)))
    return fail(MOE_EINVAL, "x and outputs must be 16-byte aligned");
  return MOE_OK;
}

moe_status set_device(moe_layer* l) {
  HIP_TRY(hipSetDevice(l->device), "hipSetDevice");
  return MOE_OK;
}

RouteParams route_params(moe_layer* l, int T, const void* x) {
  RouteParams p;
  p.x = static_cast<const f16*>(x);
  p.wg = l->w_router;
  p.table = l->d_table;
  p.T = T;
  p.d = l->desc.d_model;
  p.E = l->desc.n_experts;
  p.K = l->desc.top_k;
  p.t1 = l->desc.t1;
  p.t2 = l->desc.t2;
  return p;
}

RouteOut route_out(const Workspace& ws, int32_t* idx, float* w, int8_t* prec) {
  RouteOut o;
  o.idx = ws.idx;
  o.w = ws.w;
  o.prec = ws.prec;
  o.user_idx = idx;
  o.user_w = w;
  o.user_prec = prec;
  return o;
}

int max_groups_of(moe_layer* l, int T) {
  const int a = T * l->desc.top_k, b = 2 * l->desc.n_experts;
  return a < b ? a : b;
}

// Record event number `slot` (0..4) of the current call when timing is on.
hipError_t mark(moe_layer* l, int slot, hipStream_t s) {
  if (!l->timing) return hipSuccess;
  if (slot == 0 && l->ev_used + 5 > l->ev_pool.size()) {
    for (int i = 0; i < 5; ++i) {
      hipEvent_t e;
      hipError_t he = hipEventCreate(&e);
      if (he != hipSuccess) return he;
      l->ev_pool.push_back(e);
    }
  }
  const size_t at = l->ev_used + slot;
  if (slot == 4) l->ev_used += 5;
  return hipEventRecord(l->ev_pool[at], s);
}

// Which decode kernels a step takes.  The dot2 kernels stream each expert
// copy once per two tokens of its group, the matrix-core kernels once per
// 16; with at most about one token per expert copy (T*K <= E) the dot2
// kernels' smaller blocks win (Phi-shaped layer, 4 tokens: 148 -> 134 us per
// step), with more they lose (Mixtral-shaped, 8 tokens: 313 -> 393 us).
bool decode_on_matrix_cores(int T, int K, int E) {
  if (T <= 2) return false;
  return T > kDecodeDot2MaxTokens || T * K > E;
}

// The launch sequence of a decode step with the workspace `ws` (the layer's
// arena, or the static scratch of the allocation-free entry point).
// With prenorm, h_res is the residual stream on entry and x an output: the
// step forms x = fp16(rmsnorm(h_res)) first (inside the router when its
// activations fit in its LDS, else with the norm kernel), then
// h_res += MoE(x); x_next is not formed.
moe_status decode_launch(moe_layer* l, const Workspace& ws, int32_t T, const void* x, float* y,
                         float* h_res, void* x_next, int32_t* idx, float* w, int8_t* prec,
                         hipStream_t s, bool prenorm = false) {
  const int d = l->desc.d_model, f = l->desc.d_ff, K = l->desc.top_k;
  const int mg = max_groups_of(l, T);
  HIP_TRY(mark(l, 0, s), "timing event");
  RouteParams rp = route_params(l, T, x);
  if (prenorm) {
    if (route_decode_fuses_norm(T, d)) {
      rp.h_res = h_res;
      rp.x_out = static_cast<f16*>(const_cast<void*>(x));
      rp.eps = l->desc.rms_eps;
    } else {
      HIP_TRY(launch_rmsnorm(h_res, static_cast<f16*>(const_cast<void*>(x)), T, d,
                             l->desc.rms_eps, s), "rmsnorm kernel launch");
    }
  }
  HIP_TRY(launch_route_decode(rp, route_out(ws, idx, w, prec), ws.wl, ws.perm, ws.pos, s),
          "route kernel launch");
  HIP_TRY(mark(l, 1, s), "timing event");
  if (decode_on_matrix_cores(T, K, l->desc.n_experts)) {
    // several tokens per expert copy: matrix-core kernels, per-pair down
    // rows and the fused combine (+ residual rmsnorm) of the prefill path
    HIP_TRY(launch_decode_up_mfma(l->d_table, ws.wl, ws.perm, static_cast<const f16*>(x),
                                  ws.h, d, f, K, mg, s), "up kernel launch");
    HIP_TRY(mark(l, 2, s), "timing event");
    HIP_TRY(launch_decode_down_mfma(l->d_table, ws.wl, ws.perm, ws.h, ws.eperm,
                                    d, f, mg, s), "down kernel launch");
    HIP_TRY(launch_combine_prefill(ws.eperm, ws.pos, ws.w, ws.prec, T, d, K, y, h_res,
                                   static_cast<f16*>(x_next), l->desc.rms_eps, s),
            "combine kernel launch");
    HIP_TRY(mark(l, 3, s), "timing event");
  } else {
    HIP_TRY(launch_decode_up(l->d_table, ws.wl, ws.perm, static_cast<const f16*>(x),
                             ws.h, T, d, f, K, mg, s), "up kernel launch");
    HIP_TRY(mark(l, 2, s), "timing event");
    HIP_TRY(launch_decode_down(l->d_table, ws.wl, ws.perm, ws.w, ws.h, y, h_res,
                               T, d, f, K, s), "down kernel launch");
    HIP_TRY(mark(l, 3, s), "timing event");
    if (h_res && x_next)
      HIP_TRY(launch_rmsnorm(h_res, static_cast<f16*>(x_next), T, d, l->desc.rms_eps, s),
              "rmsnorm kernel launch");
  }
  HIP_TRY(mark(l, 4, s), "timing event");
  return MOE_OK;
}

moe_status decode_impl(moe_layer* l, int32_t T, const void* x, float* y,
                       float* h_res, void* x_next, int32_t* idx, float* w,
                       int8_t* prec, void* stream) {
  if (!l || !live(l)) return fail(MOE_ESTATE, "invalid or destroyed layer handle");
  const int lim = l->desc.max_tokens < kDecodeMaxTokens ? l->desc.max_tokens : kDecodeMaxTokens;
  moe_status st = check_call(l, T, lim, x, h_res ? (const void*)h_res : (const void*)y, x_next);
  if (st != MOE_OK) return st;
  if (h_res && !x_next) return fail(MOE_EINVAL, "x_next must not be NULL");
  if ((st = set_device(l)) != MOE_OK) return st;
  return decode_launch(l, l->ws, T, x, y, h_res, x_next, idx, w, prec,
                       static_cast<hipStream_t>(stream));
}

moe_status prefill_impl(moe_layer* l, int32_t T, const void* x, float* y,
                        float* h_res, void* x_next, int32_t* idx, float* w,
                        int8_t* prec, void* stream) {
  if (!l || !live(l)) return fail(MOE_ESTATE, "invalid or destroyed layer handle");
  moe_status st = check_call(l, T, l->desc.max_tokens, x,
                             h_res ? (const void*)h_res : (const void*)y, x_next);
  if (st != MOE_OK) return st;
  if (h_res && !x_next) return fail(MOE_EINVAL, "x_next must not be NULL");
  if ((st = set_device(l)) != MOE_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int d = l->desc.d_model, f = l->desc.d_ff, K = l->desc.top_k;
  const int mg = max_groups_of(l, T);
  HIP_TRY(mark(l, 0, s), "timing event");
  const Workspace& ws = l->ws;
  HIP_TRY(launch_route_prefill(route_params(l, T, x), route_out(ws, idx, w, prec),
                               ws.wl, ws.perm, ws.pos, s), "route kernel launch");
  HIP_TRY(mark(l, 1, s), "timing event");
  HIP_TRY(launch_prefill_up(l->d_table, ws.wl, ws.perm, static_cast<const f16*>(x),
                            ws.h, T, d, f, K, mg, s), "prefill up launch");
  HIP_TRY(mark(l, 2, s), "timing event");
  HIP_TRY(launch_prefill_down(l->d_table, ws.wl, ws.h, ws.eperm, T, d, f, K, mg, s),
          "prefill down launch");
  HIP_TRY(mark(l, 3, s), "timing event");
  HIP_TRY(launch_combine_prefill(ws.eperm, ws.pos, ws.w, ws.prec, T, d, K, y,
                                 h_res, static_cast<f16*>(x_next), l->desc.rms_eps, s),
          "combine kernel launch");
  HIP_TRY(mark(l, 4, s), "timing event");
  return MOE_OK;
}

void free_layer(moe_layer* l) {
  for (hipEvent_t e : l->ev_pool) (void)hipEventDestroy(e);
  for (void* p : l->owned) (void)hipFree(p);
  if (l->arena) (void)hipFree(l->arena);
  delete l;
}

}  // namespace

// Stacking Computer handle: the stacked gates of the next p layers and the
// workspace of one prediction.
struct moe_predictor {
  int device = -1;
  int32_t d = 0, E = 0, K = 0, p = 0, max_tokens = 0;
  void* arena = nullptr;
  f16* d_stack = nullptr;        // [p*E, d]
  float* d_logits = nullptr;     // [max_tokens, p*E]
  unsigned* d_counter = nullptr; // finished blocks of the running launch
};

namespace {

std::set<moe_predictor*> g_live_pred;

bool live_pred(moe_predictor* q) {
  std::lock_guard<std::mutex> g(g_mu);
  return g_live_pred.count(q) != 0;
}

}  // namespace

namespace moe {
void set_last_error(const char* msg) { g_err = msg; }
}  // namespace moe

extern "C" {

const char* moe_last_error(void) { return g_err.c_str(); }

moe_status moe_predictor_init(int32_t d_model, int32_t n_experts, int32_t top_k,
                              int32_t n_ahead, int32_t max_tokens,
                              const void* const* w_router_next, void* stream,
                              moe_predictor_t* out) {
  g_err.clear();
  if (!out) return fail(MOE_EINVAL, "out is NULL");
  *out = nullptr;
  if (d_model <= 0 || d_model % 64 || d_model > 16384)
    return fail(MOE_EINVAL, "d_model must be a positive multiple of 64, <= 16384 (got %d)", d_model);
  if (n_experts < 1 || n_experts > kMaxExperts)
    return fail(MOE_EINVAL, "n_experts must be in [1, 64] (got %d)", n_experts);
  if (top_k < 1 || top_k > kMaxTopK || top_k > n_experts)
    return fail(MOE_EINVAL, "top_k must be in [1, min(8, n_experts)] (got %d)", top_k);
  if (n_ahead < 1 || n_ahead > kMaxPredLayers)
    return fail(MOE_EINVAL, "n_ahead must be in [1, %d] (got %d)", kMaxPredLayers, n_ahead);
  if (max_tokens < 1 || max_tokens > 8192)
    return fail(MOE_EINVAL, "max_tokens must be in [1, 8192] (got %d)", max_tokens);
  if (!w_router_next) return fail(MOE_EINVAL, "w_router_next is NULL");
  for (int j = 0; j < n_ahead; ++j) {
    if (!w_router_next[j]) return fail(MOE_EINVAL, "gate %d is NULL", j);
    if (!aligned16(w_router_next[j])) return fail(MOE_EINVAL, "gate %d must be 16-byte aligned", j);
  }
  moe_predictor* q = new (std::nothrow) moe_predictor();
  if (!q) return fail(MOE_ENOMEM, "host allocation failed");
  q->d = d_model;
  q->E = n_experts;
  q->K = top_k;
  q->p = n_ahead;
  q->max_tokens = max_tokens;
  hipError_t he = hipGetDevice(&q->device);
  if (he != hipSuccess) { delete q; return hip_fail(he, "hipGetDevice"); }
  auto al = [](size_t b) { return (b + 255) & ~(size_t)255; };
  const size_t rows = (size_t)n_ahead * n_experts;
  const size_t gate_bytes = (size_t)n_experts * d_model * sizeof(f16);
  const size_t o_stack = 0;
  const size_t o_logits = o_stack + al(rows * d_model * sizeof(f16));
  const size_t o_counter = o_logits + al((size_t)max_tokens * rows * sizeof(float));
  const size_t total = o_counter + al(sizeof(unsigned));
  he = hipMalloc(&q->arena, total);
  if (he != hipSuccess) {
    delete q;
    return fail(MOE_ENOMEM, "hipMalloc of %zu predictor bytes failed: %s", total, hipGetErrorString(he));
  }
  char* base = static_cast<char*>(q->arena);
  q->d_stack = reinterpret_cast<f16*>(base + o_stack);
  q->d_logits = reinterpret_cast<float*>(base + o_logits);
  q->d_counter = reinterpret_cast<unsigned*>(base + o_counter);
  hipStream_t s = static_cast<hipStream_t>(stream);
  // the stacking: gate j occupies rows [j*E, (j+1)*E)
  for (int j = 0; j < n_ahead && he == hipSuccess; ++j)
    he = hipMemcpyAsync(reinterpret_cast<char*>(q->d_stack) + j * gate_bytes, w_router_next[j],
                        gate_bytes, hipMemcpyDeviceToDevice, s);
  if (he == hipSuccess) he = hipMemsetAsync(q->d_counter, 0, sizeof(unsigned), s);
  if (he == hipSuccess) he = hipStreamSynchronize(s);
  if (he != hipSuccess) {
    (void)hipFree(q->arena);
    delete q;
    return hip_fail(he, "predictor init copy");
  }
  {
    std::lock_guard<std::mutex> g(g_mu);
    g_live_pred.insert(q);
  }
  *out = q;
  return MOE_OK;
}

moe_status moe_predict(moe_predictor_t q, int32_t n_tokens, const void* x,
                       const uint64_t* cached, int32_t* pred_idx, float* pred_w,
                       int32_t* first_miss, uint64_t* preload, void* stream) {
  g_err.clear();
  if (!q || !live_pred(q)) return fail(MOE_ESTATE, "invalid or destroyed predictor handle");
  if (n_tokens < 1 || n_tokens > q->max_tokens)
    return fail(MOE_EINVAL, "n_tokens must be in [1, %d] (got %d)", q->max_tokens, n_tokens);
  if (!x || !cached || !pred_idx || !first_miss || !preload)
    return fail(MOE_EINVAL, "x, cached, pred_idx, first_miss and preload must not be NULL");
  if (!aligned16(x)) return fail(MOE_EINVAL, "x must be 16-byte aligned");
  if (((uintptr_t)cached & 7u) || ((uintptr_t)preload & 7u))
    return fail(MOE_EINVAL, "cached and preload must be 8-byte aligned");
  HIP_TRY(hipSetDevice(q->device), "hipSetDevice");
  PredictParams pp;
  pp.x = static_cast<const f16*>(x);
  pp.wstack = q->d_stack;
  pp.cached = cached;
  pp.logits = q->d_logits;
  pp.counter = q->d_counter;
  pp.idx = pred_idx;
  pp.w = pred_w;
  pp.first_miss = first_miss;
  pp.preload = preload;
  pp.T = n_tokens;
  pp.d = q->d;
  pp.E = q->E;
  pp.K = q->K;
  pp.p = q->p;
  HIP_TRY(launch_predict(pp, static_cast<hipStream_t>(stream)), "predict kernel launch");
  return MOE_OK;
}

moe_status moe_predictor_destroy(moe_predictor_t q) {
  g_err.clear();
  if (!q) return fail(MOE_EINVAL, "predictor is NULL");
  {
    std::lock_guard<std::mutex> g(g_mu);
    if (!g_live_pred.erase(q)) return fail(MOE_ESTATE, "invalid or destroyed predictor handle");
  }
  hipError_t he = hipSetDevice(q->device);
  if (he == hipSuccess) he = hipDeviceSynchronize();
  (void)hipFree(q->arena);
  delete q;
  if (he != hipSuccess) return hip_fail(he, "destroy synchronize");
  return MOE_OK;
}

moe_status moe_layer_init(const moe_layer_desc* desc, const void* w_router,
                          const void* const* w1, const void* const* w3,
                          const void* const* w2, void* stream, moe_layer_t* out) {
  g_err.clear();
  if (!out) return fail(MOE_EINVAL, "out is NULL");
  *out = nullptr;
  moe_status st = check_desc(desc);
  if (st != MOE_OK) return st;
  if (!w_router || !w1 || !w3 || !w2) return fail(MOE_EINVAL, "weight pointers must not be NULL");
  if (!aligned16(w_router)) return fail(MOE_EINVAL, "w_router must be 16-byte aligned");
  for (int e = 0; e < desc->n_experts; ++e) {
    if (!w1[e] || !w3[e] || !w2[e]) return fail(MOE_EINVAL, "expert %d has a NULL weight pointer", e);
    if (!aligned16(w1[e]) || !aligned16(w3[e]) || !aligned16(w2[e]))
      return fail(MOE_EINVAL, "expert %d weights must be 16-byte aligned", e);
  }
  moe_layer* l = new (std::nothrow) moe_layer();
  if (!l) return fail(MOE_ENOMEM, "host allocation failed");
  l->desc = *desc;
  hipError_t he = hipGetDevice(&l->device);
  if (he != hipSuccess) { delete l; return hip_fail(he, "hipGetDevice"); }
  // the static scratch of moe_decode_step_noalloc: its address on this
  // device is looked up here, once per device, with the device current
  he = scratch_setup(l->device, nullptr);
  if (he != hipSuccess) { delete l; return hip_fail(he, "scratch address lookup"); }
  l->w_router = static_cast<const f16*>(w_router);
  const int E = desc->n_experts, K = desc->top_k, d = desc->d_model, f = desc->d_ff;
  const int64_t M = desc->max_tokens;
  l->host_table.resize(E);
  l->low_q.resize(E);
  l->low_s.resize(E);
  l->low_src.resize(E);
  for (int e = 0; e < E; ++e) {
    ExpertEntry& x = l->host_table[e];
    std::memset(&x, 0, sizeof x);
    x.w[0] = static_cast<const f16*>(w1[e]);
    x.w[1] = static_cast<const f16*>(w3[e]);
    x.w[2] = static_cast<const f16*>(w2[e]);
    x.tag = TAG_FP16;
    x.hi_bits = 16;
    for (auto& a : l->low_q[e]) a.fill(nullptr);
    for (auto& a : l->low_s[e]) a.fill(nullptr);
    for (auto& a : l->low_src[e]) a.fill(nullptr);
  }
  // one arena: every region 256-byte aligned
  auto al = [](size_t b) { return (b + 255) & ~(size_t)255; };
  size_t off = 0;
  const size_t o_table = off; off += al(sizeof(ExpertEntry) * E);
  const size_t o_wl = off;    off += al(sizeof(WorkList));
  const size_t o_perm = off;  off += al(sizeof(int32_t) * M * K);
  const size_t o_pos = off;   off += al(sizeof(int32_t) * M * K);
  const size_t o_idx = off;   off += al(sizeof(int32_t) * M * K);
  const size_t o_w = off;     off += al(sizeof(float) * M * K);
  const size_t o_prec = off;  off += al(sizeof(int8_t) * M * K);
  const size_t o_h = off;     off += al(sizeof(f16) * M * K * f);
  const size_t o_ep = off;    off += al(sizeof(float) * M * K * d);
  he = hipMalloc(&l->arena, off);
  if (he != hipSuccess) {
    delete l;
    return fail(MOE_ENOMEM, "hipMalloc of %zu workspace bytes failed: %s", off, hipGetErrorString(he));
  }
  char* base = static_cast<char*>(l->arena);
  l->d_table = reinterpret_cast<ExpertEntry*>(base + o_table);
  l->ws.wl = reinterpret_cast<WorkList*>(base + o_wl);
  l->ws.perm = reinterpret_cast<int32_t*>(base + o_perm);
  l->ws.pos = reinterpret_cast<int32_t*>(base + o_pos);
  l->ws.idx = reinterpret_cast<int32_t*>(base + o_idx);
  l->ws.w = reinterpret_cast<float*>(base + o_w);
  l->ws.prec = reinterpret_cast<int8_t*>(base + o_prec);
  l->ws.h = reinterpret_cast<f16*>(base + o_h);
  l->ws.eperm = reinterpret_cast<float*>(base + o_ep);
  hipStream_t s = static_cast<hipStream_t>(stream);
  he = hipMemcpyAsync(l->d_table, l->host_table.data(), sizeof(ExpertEntry) * E,
                      hipMemcpyHostToDevice, s);
  if (he == hipSuccess) he = hipMemsetAsync(l->ws.wl, 0, sizeof(WorkList), s);
  if (he == hipSuccess) he = hipStreamSynchronize(s);
  if (he != hipSuccess) {
    free_layer(l);
    return hip_fail(he, "layer init copy");
  }
  {
    std::lock_guard<std::mutex> g(g_mu);
    g_live.insert(l);
  }
  *out = l;
  return MOE_OK;
}

moe_status moe_set_expert_precision(moe_layer_t l, int32_t expert, int32_t tag,
                                    void* stream) {
  g_err.clear();
  if (!l || !live(l)) return fail(MOE_ESTATE, "invalid or destroyed layer handle");
  if (expert < 0 || expert >= l->desc.n_experts)
    return fail(MOE_EINVAL, "expert %d out of range [0, %d)", expert, l->desc.n_experts);
  if (tag < MOE_TAG_FP16 || tag > MOE_TAG_MISS_INT8_INT2) return fail(MOE_EINVAL, "unknown tag %d", tag);
  moe_status st = set_device(l);
  if (st != MOE_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  ExpertEntry v = l->host_table[expert];
  if (!v.w[0] || !v.w[1] || !v.w[2])
    return fail(MOE_ESTATE, "expert %d is bound without fp16 weights: bind it again instead", expert);
  v.tag = tag;
  // quantised copies this tag needs, built once from the fp16 weights (and
  // rebuilt in place, in stream order, when the expert has been re-bound to
  // other fp16 weights since)
  const int d = l->desc.d_model, f = l->desc.d_ff;
  auto ensure = [&](int bits, const uint8_t* (&q_out)[3], const f16* (&s_out)[3]) -> moe_status {
    const int slot = slot_of_bits(bits);
    for (int m = 0; m < 3; ++m) {
      const int64_t rows = m < 2 ? f : d, cols = m < 2 ? d : f;
      uint8_t* q = l->low_q[expert][slot][m];
      f16* sc = l->low_s[expert][slot][m];
      const bool fresh = q == nullptr;
      if (fresh) {
        void *qv = nullptr, *sv = nullptr;
        hipError_t he = hipMalloc(&qv, (size_t)rows * cols * bits / 8);
        if (he == hipSuccess) he = hipMalloc(&sv, (size_t)rows * (cols / kGroup) * sizeof(f16));
        if (he != hipSuccess) {
          if (qv) (void)hipFree(qv);
          return fail(MOE_ENOMEM, "allocation of the int%d copy failed: %s", bits, hipGetErrorString(he));
        }
        q = static_cast<uint8_t*>(qv);
        sc = static_cast<f16*>(sv);
      }
      if (fresh || l->low_src[expert][slot][m] != v.w[m]) {
        const hipError_t he = launch_quantize(v.w[m], rows, cols, bits, q, sc, s);
        if (he != hipSuccess) {
          if (fresh) {
            (void)hipFree(q);
            (void)hipFree(sc);
          } else {
            // the old contents may be partly overwritten: never reuse them
            l->low_src[expert][slot][m] = nullptr;
          }
          return hip_fail(he, "quantize kernel launch");
        }
        if (fresh) {
          l->owned.push_back(q);
          l->owned.push_back(sc);
          l->low_q[expert][slot][m] = q;
          l->low_s[expert][slot][m] = sc;
        }
        l->low_src[expert][slot][m] = v.w[m];
      }
      q_out[m] = q;
      s_out[m] = sc;
    }
    return MOE_OK;
  };
  const int lb = low_bits_of(tag), hb = high_bits_of(tag);
  for (int m = 0; m < 3; ++m) { v.q[m] = nullptr; v.s[m] = nullptr; v.hq[m] = nullptr; v.hs[m] = nullptr; }
  if (lb) {
    st = ensure(lb, v.q, v.s);
    if (st != MOE_OK) return st;
  }
  if (hb == 8) {
    st = ensure(8, v.hq, v.hs);
    if (st != MOE_OK) return st;
  }
  v.low_bits = lb;
  v.hi_bits = hb == 8 ? 8 : 16;
  l->host_table[expert] = v;
  HIP_TRY(launch_set_entry(l->d_table, expert, v, s), "table update launch");
  return MOE_OK;
}

moe_status moe_layer_bind_expert(moe_layer_t l, int32_t expert, int32_t tag,
                                 const void* const* w, const void* const* q,
                                 const void* const* sc, int32_t low_bits, void* stream) {
  g_err.clear();
  if (!l || !live(l)) return fail(MOE_ESTATE, "invalid or destroyed layer handle");
  if (expert < 0 || expert >= l->desc.n_experts)
    return fail(MOE_EINVAL, "expert %d out of range [0, %d)", expert, l->desc.n_experts);
  if (tag == MOE_TAG_INT8 || tag == MOE_TAG_MISS_INT8_INT2)
    return fail(MOE_EUNSUPPORTED, "int8-model tags are set with moe_set_expert_precision, not bound");
  if (tag < MOE_TAG_FP16 || tag > MOE_TAG_MISS_INT2) return fail(MOE_EINVAL, "unknown tag %d", tag);
  const bool need_w = tag == MOE_TAG_FP16 || tag == MOE_TAG_MISS_INT4 || tag == MOE_TAG_MISS_INT2;
  const int bits = (tag == MOE_TAG_INT4 || tag == MOE_TAG_MISS_INT4) ? 4
                   : (tag == MOE_TAG_INT2 || tag == MOE_TAG_MISS_INT2) ? 2 : 0;
  if (bits && low_bits != bits)
    return fail(MOE_EINVAL, "tag %d needs a %d-bit copy (low_bits %d)", tag, bits, low_bits);
  for (int m = 0; m < 3; ++m) {
    if (need_w && (!w || !w[m] || !aligned16(w[m])))
      return fail(MOE_EINVAL, "tag %d needs three 16-byte aligned fp16 matrices", tag);
    if (bits && (!q || !sc || !q[m] || !sc[m] || !aligned16(q[m]) || !aligned16(sc[m])))
      return fail(MOE_EINVAL, "tag %d needs three 16-byte aligned code and scale arrays", tag);
  }
  moe_status st = set_device(l);
  if (st != MOE_OK) return st;
  ExpertEntry v;
  std::memset(&v, 0, sizeof v);
  for (int m = 0; m < 3; ++m) {
    v.w[m] = need_w ? static_cast<const f16*>(w[m]) : nullptr;
    v.q[m] = bits ? static_cast<const uint8_t*>(q[m]) : nullptr;
    v.s[m] = bits ? static_cast<const f16*>(sc[m]) : nullptr;
  }
  v.tag = tag;
  v.low_bits = bits;
  v.hi_bits = 16;
  l->host_table[expert] = v;
  HIP_TRY(launch_set_entry(l->d_table, expert, v, static_cast<hipStream_t>(stream)),
          "table update launch");
  return MOE_OK;
}

moe_status moe_decode_step(moe_layer_t l, int32_t n_tokens, const void* x, float* y,
                           int32_t* topk_idx, float* topk_w, int8_t* prec_used,
                           void* stream) {
  g_err.clear();
  return decode_impl(l, n_tokens, x, y, nullptr, nullptr, topk_idx, topk_w, prec_used, stream);
}

moe_status moe_decode_step_noalloc(moe_layer_t l, int32_t T, const void* x, float* y,
                                   int32_t* topk_idx, float* topk_w, int8_t* prec_used,
                                   void* stream) {
  g_err.clear();
  if (!l || !live(l)) return fail(MOE_ESTATE, "invalid or destroyed layer handle");
  const int lim = l->desc.max_tokens < kDecodeMaxTokens ? l->desc.max_tokens : kDecodeMaxTokens;
  moe_status st = check_call(l, T, lim, x, y, nullptr);
  if (st != MOE_OK) return st;
  // the layout of the layer's arena, sized for T tokens
  auto al = [](size_t b) { return (b + 255) & ~(size_t)255; };
  const size_t P = (size_t)T * l->desc.top_k;
  size_t off = 0;
  const size_t o_wl = off;   off += al(sizeof(WorkList));
  const size_t o_perm = off; off += al(sizeof(int32_t) * P);
  const size_t o_pos = off;  off += al(sizeof(int32_t) * P);
  const size_t o_idx = off;  off += al(sizeof(int32_t) * P);
  const size_t o_w = off;    off += al(sizeof(float) * P);
  const size_t o_prec = off; off += al(sizeof(int8_t) * P);
  const size_t o_h = off;    off += al(sizeof(f16) * P * l->desc.d_ff);
  const size_t o_ep = off;
  const bool mc = decode_on_matrix_cores(T, l->desc.top_k, l->desc.n_experts);
  if (mc) off += al(sizeof(float) * P * l->desc.d_model);
  if (off > scratch_bytes())
    return fail(MOE_EINVAL,
                "a %d-token step of this layer needs %zu bytes of scratch; the static scratch "
                "holds %zu (use fewer tokens per call, or moe_decode_step)",
                T, off, scratch_bytes());
  if ((st = set_device(l)) != MOE_OK) return st;
  void* base_v = nullptr;
  HIP_TRY(scratch_setup(l->device, &base_v), "scratch address lookup");
  char* base = static_cast<char*>(base_v);
  Workspace ws;
  ws.wl = reinterpret_cast<WorkList*>(base + o_wl);
  ws.perm = reinterpret_cast<int32_t*>(base + o_perm);
  ws.pos = reinterpret_cast<int32_t*>(base + o_pos);
  ws.idx = reinterpret_cast<int32_t*>(base + o_idx);
  ws.w = reinterpret_cast<float*>(base + o_w);
  ws.prec = reinterpret_cast<int8_t*>(base + o_prec);
  ws.h = reinterpret_cast<f16*>(base + o_h);
  ws.eperm = mc ? reinterpret_cast<float*>(base + o_ep) : nullptr;
  return decode_launch(l, ws, T, x, y, nullptr, nullptr, topk_idx, topk_w, prec_used,
                       static_cast<hipStream_t>(stream));
}

moe_status moe_decode_step_residual(moe_layer_t l, int32_t n_tokens, const void* x,
                                    float* h, void* x_next, int32_t* topk_idx,
                                    float* topk_w, int8_t* prec_used, void* stream) {
  g_err.clear();
  return decode_impl(l, n_tokens, x, nullptr, h, x_next, topk_idx, topk_w, prec_used, stream);
}

moe_status moe_decode_step_prenorm(moe_layer_t l, int32_t T, float* h, void* x,
                                   int32_t* topk_idx, float* topk_w, int8_t* prec_used,
                                   void* stream) {
  g_err.clear();
  if (!l || !live(l)) return fail(MOE_ESTATE, "invalid or destroyed layer handle");
  const int lim = l->desc.max_tokens < kDecodeMaxTokens ? l->desc.max_tokens : kDecodeMaxTokens;
  moe_status st = check_call(l, T, lim, h, x, nullptr);
  if (st != MOE_OK) return st;
  if ((st = set_device(l)) != MOE_OK) return st;
  return decode_launch(l, l->ws, T, x, nullptr, h, nullptr, topk_idx, topk_w, prec_used,
                       static_cast<hipStream_t>(stream), true);
}

moe_status moe_prefill(moe_layer_t l, int32_t n_tokens, const void* x, float* y,
                       int32_t* topk_idx, float* topk_w, int8_t* prec_used, void* stream) {
  g_err.clear();
  return prefill_impl(l, n_tokens, x, y, nullptr, nullptr, topk_idx, topk_w, prec_used, stream);
}

moe_status moe_prefill_residual(moe_layer_t l, int32_t n_tokens, const void* x, float* h,
                                void* x_next, int32_t* topk_idx, float* topk_w,
                                int8_t* prec_used, void* stream) {
  g_err.clear();
  return prefill_impl(l, n_tokens, x, nullptr, h, x_next, topk_idx, topk_w, prec_used, stream);
}

moe_status moe_export_packed(moe_layer_t l, int32_t expert, int32_t matrix, int32_t bits,
                             void* codes, void* scales, void* stream) {
  g_err.clear();
  if (!l || !live(l)) return fail(MOE_ESTATE, "invalid or destroyed layer handle");
  if (expert < 0 || expert >= l->desc.n_experts) return fail(MOE_EINVAL, "expert out of range");
  if (matrix < 0 || matrix > 2) return fail(MOE_EINVAL, "matrix must be 0, 1 or 2");
  if (bits != 8 && bits != 4 && bits != 2) return fail(MOE_EINVAL, "bits must be 8, 4 or 2");
  if (!codes || !scales) return fail(MOE_EINVAL, "codes and scales must not be NULL");
  const int slot = slot_of_bits(bits);
  const uint8_t* q = l->low_q[expert][slot][matrix];
  const f16* sc = l->low_s[expert][slot][matrix];
  if (!q) return fail(MOE_ESTATE, "expert %d has no int%d copy", expert, bits);
  moe_status st = set_device(l);
  if (st != MOE_OK) return st;
  const int d = l->desc.d_model, f = l->desc.d_ff;
  const int64_t rows = matrix < 2 ? f : d, cols = matrix < 2 ? d : f;
  hipStream_t s = static_cast<hipStream_t>(stream);
  HIP_TRY(hipMemcpyAsync(codes, q, (size_t)rows * cols * bits / 8, hipMemcpyDeviceToDevice, s),
          "export codes");
  HIP_TRY(hipMemcpyAsync(scales, sc, (size_t)rows * (cols / kGroup) * sizeof(f16),
                         hipMemcpyDeviceToDevice, s), "export scales");
  return MOE_OK;
}

moe_status moe_quantize(const void* w, int64_t rows, int64_t cols, int32_t bits,
                        void* codes, void* scales, void* stream) {
  g_err.clear();
  if (!w || !codes || !scales) return fail(MOE_EINVAL, "pointers must not be NULL");
  if (rows < 0 || cols < 0 || cols % kGroup) return fail(MOE_EINVAL, "cols must be a multiple of 32");
  if (bits != 8 && bits != 4 && bits != 2) return fail(MOE_EINVAL, "bits must be 8, 4 or 2");
  if (rows > 0 && cols / kGroup > (((int64_t)1 << 38) / rows)) return fail(MOE_EINVAL, "matrix too large");
  if (!aligned16(w) || ((uintptr_t)codes & 7u) || ((uintptr_t)scales & 1u))
    return fail(MOE_EINVAL, "w must be 16-byte aligned, codes 8-byte, scales 2-byte");
  if (bits >= 4 && ((uintptr_t)codes & 15u))
    return fail(MOE_EINVAL, "int4 and int8 codes must be 16-byte aligned");
  HIP_TRY(launch_quantize(static_cast<const f16*>(w), rows, cols, bits,
                          static_cast<uint8_t*>(codes), static_cast<f16*>(scales),
                          static_cast<hipStream_t>(stream)), "quantize kernel launch");
  return MOE_OK;
}

moe_status moe_rmsnorm(const float* h, void* x, int32_t n_tokens, int32_t d_model, float eps,
                       void* stream) {
  g_err.clear();
  if (!h || !x) return fail(MOE_EINVAL, "h and x must not be NULL");
  if (n_tokens < 1) return fail(MOE_EINVAL, "n_tokens must be >= 1 (got %d)", n_tokens);
  if (d_model <= 0 || d_model % 64 || d_model > 16384)
    return fail(MOE_EINVAL, "d_model must be a positive multiple of 64, <= 16384 (got %d)", d_model);
  if (!(eps >= 0.0f)) return fail(MOE_EINVAL, "eps must be >= 0");
  if (!aligned16(h) || !aligned16(x)) return fail(MOE_EINVAL, "h and x must be 16-byte aligned");
  HIP_TRY(launch_rmsnorm(h, static_cast<f16*>(x), n_tokens, d_model, eps,
                         static_cast<hipStream_t>(stream)), "rmsnorm kernel launch");
  return MOE_OK;
}

moe_status moe_layer_enable_timing(moe_layer_t l, int32_t enable) {
  g_err.clear();
  if (!l || !live(l)) return fail(MOE_ESTATE, "invalid or destroyed layer handle");
  l->timing = enable != 0;
  l->ev_used = 0;
  return MOE_OK;
}

moe_status moe_layer_stage_times(moe_layer_t l, double* ms, int32_t* n_calls) {
  g_err.clear();
  if (!l || !live(l)) return fail(MOE_ESTATE, "invalid or destroyed layer handle");
  if (!ms || !n_calls) return fail(MOE_EINVAL, "ms and n_calls must not be NULL");
  for (int i = 0; i < 4; ++i) ms[i] = 0.0;
  const size_t calls = l->ev_used / 5;
  if (calls) {
    moe_status st = set_device(l);
    if (st != MOE_OK) return st;
    HIP_TRY(hipEventSynchronize(l->ev_pool[l->ev_used - 1]), "timing synchronize");
  }
  for (size_t c = 0; c < calls; ++c)
    for (int i = 0; i < 4; ++i) {
      float t = 0.0f;
      HIP_TRY(hipEventElapsedTime(&t, l->ev_pool[5 * c + i], l->ev_pool[5 * c + i + 1]),
              "timing elapsed");
      ms[i] += t;
    }
  *n_calls = (int32_t)calls;
  l->ev_used = 0;
  return MOE_OK;
}

moe_status moe_layer_share_workspace(moe_layer_t l, moe_layer_t owner, void* stream) {
  g_err.clear();
  if (!l || !owner) return fail(MOE_EINVAL, "layer and owner must be non-NULL");
  if (l == owner) return fail(MOE_EINVAL, "a layer cannot share its own workspace");
  moe_layer* o = nullptr;
  {
    std::lock_guard<std::mutex> g(g_mu);
    if (!g_live.count(l) || !g_live.count(owner))
      return fail(MOE_ESTATE, "invalid or destroyed layer handle");
    o = owner->ws_owner ? owner->ws_owner : owner;  // the workspace's owner
    if (l->ws_owner == o) return MOE_OK;             // already shared
    if (l->ws_owner) return fail(MOE_ESTATE, "the layer already runs on another layer's workspace");
    if (l->ws_sharers > 0)
      return fail(MOE_ESTATE, "%d layer(s) run on this layer's workspace", l->ws_sharers);
  }
  const moe_layer_desc &a = l->desc, &b = o->desc;
  if (a.d_model != b.d_model || a.d_ff != b.d_ff || a.top_k != b.top_k ||
      a.max_tokens != b.max_tokens)
    return fail(MOE_EINVAL, "shared workspaces need equal d_model, d_ff, top_k and max_tokens");
  if (l->device != o->device) return fail(MOE_EINVAL, "the layers live on different devices");
  moe_status st = set_device(l);
  if (st != MOE_OK) return st;
  // a table-only arena replaces the layer's own (table + workspace)
  hipStream_t s = static_cast<hipStream_t>(stream);
  const size_t tb = sizeof(ExpertEntry) * a.n_experts;
  void* t = nullptr;
  hipError_t he = hipMalloc(&t, tb);
  if (he != hipSuccess) return fail(MOE_ENOMEM, "hipMalloc of %zu table bytes failed", tb);
  he = hipMemcpyAsync(t, l->d_table, tb, hipMemcpyDeviceToDevice, s);
  if (he == hipSuccess) he = hipStreamSynchronize(s);
  if (he == hipSuccess) he = hipDeviceSynchronize();  // nothing may still use the old arena
  if (he != hipSuccess) {
    (void)hipFree(t);
    return hip_fail(he, "share workspace copy");
  }
  (void)hipFree(l->arena);
  l->arena = t;
  l->d_table = static_cast<ExpertEntry*>(t);
  l->ws = o->ws;
  std::lock_guard<std::mutex> g(g_mu);
  l->ws_owner = o;
  ++o->ws_sharers;
  return MOE_OK;
}

moe_status moe_layer_destroy(moe_layer_t l) {
  g_err.clear();
  if (!l) return fail(MOE_EINVAL, "layer is NULL");
  {
    std::lock_guard<std::mutex> g(g_mu);
    if (!g_live.count(l)) return fail(MOE_ESTATE, "invalid or destroyed layer handle");
    if (l->ws_sharers > 0)
      return fail(MOE_ESTATE, "%d layer(s) still run on this layer's workspace; destroy them first",
                  l->ws_sharers);
    g_live.erase(l);
    if (l->ws_owner) --l->ws_owner->ws_sharers;
  }
  hipError_t he = hipSetDevice(l->device);
  if (he == hipSuccess) he = hipDeviceSynchronize();
  free_layer(l);
  if (he != hipSuccess) return hip_fail(he, "destroy synchronize");
  return MOE_OK;
}

}  // extern "C"
