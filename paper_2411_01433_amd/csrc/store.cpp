// Expert storage in pinned host memory and the expert loads of the Dynamic
// Expert Loader (Section 3.2, Fig. 6: expert copies live in host Expert
// Storage and a cache miss loads the copy of the precision the Eq. 2 rule
// chose into the GPU expert cache; Section 2.2: an int4 copy moves about a
// quarter of the fp16 bytes, so it loads about four times faster).
//
// One store holds one layer's experts: for each, the fp16 W1, W3 [d_ff,
// d_model] and W2 [d_model, d_ff] and their low-precision copy (codes
// [rows, cols*b/8], fp16 scales [rows, cols/32], the layer's quantiser),
// all in hipHostMalloc memory so that hipMemcpyAsync transfers run on the
// DMA engines, asynchronously on the caller's stream.
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <new>
#include <set>
#include <vector>

#include "moe.h"
#include "moe_internal.h"

namespace moe {
void set_last_error(const char* msg);  // moe_api.cpp
}

struct moe_store {
  int device = -1;
  int32_t d = 0, f = 0, E = 0, bits = 0;
  size_t fp16_bytes = 0, code_bytes = 0, scale_bytes = 0, per_expert = 0;
  char* host = nullptr;
  std::vector<uint8_t> filled;
  char* w(int e, int m) { return host + (size_t)e * per_expert + m * fp16_bytes; }
  char* q(int e, int m) { return host + (size_t)e * per_expert + 3 * fp16_bytes + m * code_bytes; }
  char* s(int e, int m) {
    return host + (size_t)e * per_expert + 3 * (fp16_bytes + code_bytes) + m * scale_bytes;
  }
};

namespace {

std::mutex g_store_mu;
std::set<moe_store*> g_store_live;

moe_status sfail(moe_status st, const char* fmt, ...) {
  char buf[256];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  moe::set_last_error(buf);
  return st;
}

moe_status shfail(hipError_t e, const char* what) {
  return sfail(MOE_EHIP, "%s: %s", what, hipGetErrorString(e));
}

bool live(moe_store* st) {
  std::lock_guard<std::mutex> g(g_store_mu);
  return st && g_store_live.count(st) != 0;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

}  // namespace

extern "C" {

moe_status moe_store_create(int32_t d_model, int32_t d_ff, int32_t n_experts, int32_t low_bits,
                            moe_store_t* out) {
  moe::set_last_error("");
  if (!out) return sfail(MOE_EINVAL, "out is NULL");
  *out = nullptr;
  if (d_model <= 0 || d_model % 64 || d_model > 16384)
    return sfail(MOE_EINVAL, "d_model must be a positive multiple of 64, <= 16384 (got %d)", d_model);
  if (d_ff <= 0 || d_ff % 64 || d_ff > 65536)
    return sfail(MOE_EINVAL, "d_ff must be a positive multiple of 64, <= 65536 (got %d)", d_ff);
  if (n_experts < 1 || n_experts > moe::kMaxExperts)
    return sfail(MOE_EINVAL, "n_experts must be in [1, 64] (got %d)", n_experts);
  if (low_bits != 4 && low_bits != 2) return sfail(MOE_EINVAL, "low_bits must be 4 or 2");
  moe_store* st = new (std::nothrow) moe_store();
  if (!st) return sfail(MOE_ENOMEM, "host allocation failed");
  hipError_t he = hipGetDevice(&st->device);
  if (he != hipSuccess) { delete st; return shfail(he, "hipGetDevice"); }
  st->d = d_model;
  st->f = d_ff;
  st->E = n_experts;
  st->bits = low_bits;
  const size_t n = (size_t)d_model * d_ff;
  st->fp16_bytes = n * 2;
  st->code_bytes = n * low_bits / 8;
  st->scale_bytes = n / moe::kGroup * 2;
  st->per_expert = 3 * (st->fp16_bytes + st->code_bytes + st->scale_bytes);
  he = hipHostMalloc(reinterpret_cast<void**>(&st->host), st->per_expert * n_experts,
                     hipHostMallocDefault);
  if (he != hipSuccess) {
    delete st;
    return sfail(MOE_ENOMEM, "hipHostMalloc of %zu bytes failed: %s",
                 st->per_expert * (size_t)n_experts, hipGetErrorString(he));
  }
  st->filled.assign(n_experts, 0);
  {
    std::lock_guard<std::mutex> g(g_store_mu);
    g_store_live.insert(st);
  }
  *out = st;
  return MOE_OK;
}

moe_status moe_store_sizes(moe_store_t st, int64_t* fp16_bytes, int64_t* code_bytes,
                           int64_t* scale_bytes) {
  moe::set_last_error("");
  if (!live(st)) return sfail(MOE_ESTATE, "invalid or destroyed store handle");
  if (fp16_bytes) *fp16_bytes = (int64_t)st->fp16_bytes;
  if (code_bytes) *code_bytes = (int64_t)st->code_bytes;
  if (scale_bytes) *scale_bytes = (int64_t)st->scale_bytes;
  return MOE_OK;
}

moe_status moe_store_put(moe_store_t st, int32_t expert, const void* w1, const void* w3,
                         const void* w2, void* stream) {
  moe::set_last_error("");
  if (!live(st)) return sfail(MOE_ESTATE, "invalid or destroyed store handle");
  if (expert < 0 || expert >= st->E) return sfail(MOE_EINVAL, "expert %d out of range", expert);
  const void* w[3] = {w1, w3, w2};
  for (int m = 0; m < 3; ++m) {
    if (!w[m]) return sfail(MOE_EINVAL, "weight %d is NULL", m);
    if (!aligned16(w[m])) return sfail(MOE_EINVAL, "weights must be 16-byte aligned");
  }
  hipError_t he = hipSetDevice(st->device);
  if (he != hipSuccess) return shfail(he, "hipSetDevice");
  hipStream_t s = static_cast<hipStream_t>(stream);
  void *tq = nullptr, *ts = nullptr;
  he = hipMalloc(&tq, st->code_bytes);
  if (he == hipSuccess) he = hipMalloc(&ts, st->scale_bytes);
  if (he != hipSuccess) {
    if (tq) (void)hipFree(tq);
    return sfail(MOE_ENOMEM, "device staging for the low copy failed: %s", hipGetErrorString(he));
  }
  for (int m = 0; m < 3 && he == hipSuccess; ++m) {
    const int64_t rows = m < 2 ? st->f : st->d, cols = m < 2 ? st->d : st->f;
    he = hipMemcpyAsync(st->w(expert, m), w[m], st->fp16_bytes, hipMemcpyDeviceToHost, s);
    if (he == hipSuccess)
      he = moe::launch_quantize(static_cast<const moe::f16*>(w[m]), rows, cols, st->bits,
                                static_cast<uint8_t*>(tq), static_cast<moe::f16*>(ts), s);
    if (he == hipSuccess)
      he = hipMemcpyAsync(st->q(expert, m), tq, st->code_bytes, hipMemcpyDeviceToHost, s);
    if (he == hipSuccess)
      he = hipMemcpyAsync(st->s(expert, m), ts, st->scale_bytes, hipMemcpyDeviceToHost, s);
    // the staging buffers are reused by the next matrix
    if (he == hipSuccess) he = hipStreamSynchronize(s);
  }
  (void)hipFree(tq);
  (void)hipFree(ts);
  if (he != hipSuccess) return shfail(he, "store put");
  st->filled[expert] = 1;
  return MOE_OK;
}

moe_status moe_store_load(moe_store_t st, int32_t expert, int32_t high, void* const* dst_w,
                          void* const* dst_q, void* const* dst_s, void* stream) {
  moe::set_last_error("");
  if (!live(st)) return sfail(MOE_ESTATE, "invalid or destroyed store handle");
  if (expert < 0 || expert >= st->E) return sfail(MOE_EINVAL, "expert %d out of range", expert);
  if (!st->filled[expert]) return sfail(MOE_ESTATE, "expert %d was never put", expert);
  if (high ? !dst_w : (!dst_q || !dst_s))
    return sfail(MOE_EINVAL, "destination array is NULL");
  for (int m = 0; m < 3; ++m) {
    if (high ? !dst_w[m] : (!dst_q[m] || !dst_s[m]))
      return sfail(MOE_EINVAL, "destination %d is NULL", m);
  }
  hipError_t he = hipSetDevice(st->device);
  if (he != hipSuccess) return shfail(he, "hipSetDevice");
  hipStream_t s = static_cast<hipStream_t>(stream);
  for (int m = 0; m < 3 && he == hipSuccess; ++m) {
    if (high) {
      he = hipMemcpyAsync(dst_w[m], st->w(expert, m), st->fp16_bytes, hipMemcpyHostToDevice, s);
    } else {
      he = hipMemcpyAsync(dst_q[m], st->q(expert, m), st->code_bytes, hipMemcpyHostToDevice, s);
      if (he == hipSuccess)
        he = hipMemcpyAsync(dst_s[m], st->s(expert, m), st->scale_bytes, hipMemcpyHostToDevice, s);
    }
  }
  if (he != hipSuccess) return shfail(he, "store load copy");
  return MOE_OK;
}

moe_status moe_store_destroy(moe_store_t st) {
  moe::set_last_error("");
  if (!st) return sfail(MOE_EINVAL, "store is NULL");
  {
    std::lock_guard<std::mutex> g(g_store_mu);
    if (!g_store_live.erase(st)) return sfail(MOE_ESTATE, "invalid or destroyed store handle");
  }
  hipError_t he = hipSetDevice(st->device);
  if (he == hipSuccess) he = hipDeviceSynchronize();  // no copy still reads the pages
  (void)hipHostFree(st->host);
  delete st;
  if (he != hipSuccess) return shfail(he, "store destroy synchronize");
  return MOE_OK;
}

}  // extern "C"
