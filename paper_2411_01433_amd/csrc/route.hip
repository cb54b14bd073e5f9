// Gating and the token-level precision decision.
//
//   logits l[t, e] = sum_d x[t, d] Wg[e, d]           (Eq. 1 gate, fp32 acc)
//   top-k by (l desc, index asc); w = softmax over the K selected logits
//   (Section 3.2: the gate values are normalised)
//   Eq. 2: with slots already in descending gate order, s_0 = 0 and
//   s_j = sum_{i<j} w_i; miss-tagged experts run high if s <= t1, low if
//   t1 < s <= t2, are skipped if s > t2; slot 0 is always high.
//
// Then a work list groups the (token, slot) pairs by (expert, precision):
// a stable counting sort over pair ids p = t*K + k, so pair order inside a
// group follows token order and the result is deterministic.
#include "moe_internal.h"

namespace moe {

namespace {

constexpr int kRouteThreads = 1024;
static_assert(kMaxExperts <= kRouteThreads, "one thread per expert stages the table");
constexpr int kPrefillTokPerBlock = 1;
constexpr int kPrefillThreads = 256;

// fp16-pair dot product with fp32 accumulation.  The operands are taken
// as scalars on purpose: clang's __builtin_bit_cast applied directly to a
// vector component expression (v.y) reads component 0.
__device__ inline float dot2(uint32_t a, uint32_t b, float acc) {
  return __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2, a),
                                __builtin_bit_cast(f16x2, b), acc, false);
}

// Wave sums use wave_sum_dpp (moe_internal.h): the decode and prefill
// routers sum their logits with it, so their logits stay bit-identical.

// Dot products of tokens [t0, t1) against all E gate rows.  One wave per
// (expert, batch of up to TB tokens): the gate row chunk is loaded once and
// used for every token of the batch; KB chunks of 512 columns (8 fp16 per
// lane) of the gate row and of each token are loaded before any arithmetic
// so that the loads overlap (one memory latency per KB chunks).  Results go
// to lg[t-t0][e].
template <int TB, int KB>
__device__ void gate_logits(const RouteParams& p, int t0, int t1, float* lg) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int n_waves = blockDim.x >> 6;
  const int n_tb = (t1 - t0 + TB - 1) / TB;
  const int n_items = n_tb * p.E;
  for (int q = wave; q < n_items; q += n_waves) {
    const int e = q % p.E;
    const int tb0 = t0 + (q / p.E) * TB;
    const int nt = min(TB, t1 - tb0);
    const f16* gr = p.wg + (int64_t)e * p.d;
    float acc[TB];
#pragma unroll
    for (int i = 0; i < TB; ++i) acc[i] = 0.0f;
    for (int c0 = 0; c0 < p.d; c0 += KB * 512) {
      u32x4 b[KB], a[TB][KB];
#pragma unroll
      for (int j = 0; j < KB; ++j) {
        const int c = c0 + j * 512 + lane * 8;
        b[j] = c < p.d ? *reinterpret_cast<const u32x4*>(gr + c) : u32x4{0, 0, 0, 0};
#pragma unroll
        for (int i = 0; i < TB; ++i)
          a[i][j] = (i < nt && c < p.d)
                        ? *reinterpret_cast<const u32x4*>(p.x + (int64_t)(tb0 + i) * p.d + c)
                        : u32x4{0, 0, 0, 0};
      }
#pragma unroll
      for (int i = 0; i < TB; ++i)
#pragma unroll
        for (int j = 0; j < KB; ++j) {
          acc[i] = dot2(a[i][j].x, b[j].x, acc[i]);
          acc[i] = dot2(a[i][j].y, b[j].y, acc[i]);
          acc[i] = dot2(a[i][j].z, b[j].z, acc[i]);
          acc[i] = dot2(a[i][j].w, b[j].w, acc[i]);
        }
    }
#pragma unroll
    for (int i = 0; i < TB; ++i) {
      const float v = wave_sum_dpp(acc[i]);
      if (lane == 0 && i < nt) lg[(tb0 - t0 + i) * p.E + e] = v;
    }
  }
}

// top-k, softmax over the selected logits and the Eq. 2 rule for one token;
// tags[e] is the expert table's tag column staged in LDS.
__device__ void decide_token(const RouteParams& p, int t, const float* lrow,
                             const int* tags, RouteOut o, int32_t* s_idx = nullptr,
                             int8_t* s_prec = nullptr) {
  int sel[kMaxTopK];
  float ls[kMaxTopK];
  uint64_t taken = 0;  // E <= 64
  for (int k = 0; k < p.K; ++k) {
    int best = -1;
    float bv = 0.0f;
    for (int e = 0; e < p.E; ++e) {
      if (taken >> e & 1ull) continue;
      const float v = lrow[e];
      if (best < 0 || v > bv) {  // strict: exact ties keep the lower index
        best = e;
        bv = v;
      }
    }
    taken |= 1ull << best;
    sel[k] = best;
    ls[k] = bv;
  }
  float ex[kMaxTopK];
  float z = 0.0f;
  for (int k = 0; k < p.K; ++k) {
    ex[k] = expf(ls[k] - ls[0]);
    z += ex[k];
  }
  float above = 0.0f;  // Eq. 2 running score
  for (int k = 0; k < p.K; ++k) {
    const float w = ex[k] / z;
    const int e = sel[k];
    const int tag = tags[e];
    int prec;
    if (tag == TAG_FP16 || tag == TAG_INT8) {
      prec = PREC_HIGH;
    } else if (tag == TAG_INT4 || tag == TAG_INT2) {
      prec = PREC_LOW;
    } else {
      const float s = (k == 0) ? 0.0f : above;
      prec = (k == 0 || s <= p.t1) ? PREC_HIGH
                                   : (s <= p.t2 ? PREC_LOW : PREC_SKIP);
    }
    above += w;
    const int pi = t * p.K + k;
    o.idx[pi] = e;
    o.w[pi] = w;
    o.prec[pi] = (int8_t)prec;
    if (s_idx) {
      s_idx[pi] = e;
      s_prec[pi] = (int8_t)prec;
    }
    if (o.user_idx) o.user_idx[pi] = e;
    if (o.user_w) o.user_w[pi] = w;
    if (o.user_prec) o.user_prec[pi] = (int8_t)prec;
  }
}

// Stable counting sort of all T*K pairs by key = expert*2 + (low ? 1 : 0)
// (skipped pairs get no key).  Run by one whole block of kRouteThreads.
// Copy widths of one expert packed in one int: low copy (4, 2 or 0) in
// bits 0-7, high copy (16 or 8) in bits 8-15.
__device__ inline int pack_widths(const ExpertEntry& x) { return x.low_bits | (x.hi_bits << 8); }
__device__ inline int copy_bits(int widths, int low) { return low ? (widths & 0xFF) : (widths >> 8); }

// Pairs are taken one block-wide chunk at a time; inside a wave, lanes with
// equal keys are found with one ballot per distinct key, and a lane's rank
// among them is the number of lower lanes in that ballot; per-wave counts
// are then scanned across waves, so pair order inside a group is the pair
// index order.
__device__ void build_worklist(const RouteParams& p, const int32_t* idx,
                               const int8_t* prec, const int* widths,
                               WorkList* wl, int32_t* perm, int32_t* pos) {
  constexpr int kW = kRouteThreads / 64;
  __shared__ int cnt[kMaxKeys];
  __shared__ int base[kMaxKeys];
  __shared__ int wcnt[kW][kMaxKeys];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int N = p.T * p.K;
  const int n_keys = 2 * p.E;
  for (int k = tid; k < n_keys; k += blockDim.x) cnt[k] = 0;
  __syncthreads();
  for (int i = tid; i < N; i += blockDim.x) {
    const int pr = prec[i];
    if (pr != PREC_SKIP) atomicAdd(&cnt[idx[i] * 2 + (pr == PREC_LOW)], 1);
    else pos[i] = -1;
  }
  __syncthreads();
  if (tid == 0) {
    int off = 0, ng = 0, mx = 0;
    for (int k = 0; k < n_keys; ++k) {
      base[k] = off;
      const int c = cnt[k];
      if (c > 0) {
        const int e = k >> 1;
        Group g;
        g.expert = e;
        g.bits = copy_bits(widths[e], k & 1);
        g.offset = off;
        g.count = c;
        wl->groups[ng++] = g;
        mx = c > mx ? c : mx;
      }
      off += c;
    }
    wl->n_groups = ng;
    wl->max_count = mx;
  }
  const uint64_t lower = (1ull << lane) - 1ull;
  for (int c0 = 0; c0 < N; c0 += blockDim.x) {
    for (int v = tid; v < kW * n_keys; v += blockDim.x) wcnt[v / n_keys][v % n_keys] = 0;
    __syncthreads();
    const int i = c0 + tid;
    int key = -1;
    if (i < N && prec[i] != PREC_SKIP) key = idx[i] * 2 + (prec[i] == PREC_LOW);
    int rank = 0;
    uint64_t todo = __ballot(key >= 0);
    while (todo) {
      const int leader = __ffsll((unsigned long long)todo) - 1;
      const int k = __builtin_amdgcn_readlane(key, leader);
      const uint64_t m = __ballot(key == k);
      if (key == k) rank = __popcll(m & lower);
      if (lane == leader) wcnt[wave][k] = __popcll(m);
      todo &= ~m;
    }
    __syncthreads();
    // exclusive scan of the per-wave counts, per key
    if (tid < n_keys) {
      int run = base[tid];
      for (int w = 0; w < kW; ++w) {
        const int c = wcnt[w][tid];
        wcnt[w][tid] = run;
        run += c;
      }
      base[tid] = run;
    }
    __syncthreads();
    if (key >= 0) {
      const int at = wcnt[wave][key] + rank;
      perm[at] = i;
      pos[i] = at;
    }
    __syncthreads();
  }
}

// Expert tags and copy widths into LDS.
__device__ inline void stage_table(const RouteParams& p, int* tags, int* widths) {
  for (int e = threadIdx.x; e < p.E; e += blockDim.x) {
    tags[e] = p.table[e].tag;
    widths[e] = pack_widths(p.table[e]);
  }
}

// The same in two halves: the loads are issued before the gate loads and
// the LDS stores after them, so the two memory round trips overlap (E is at
// most 64, below the block size).
struct TableRow {
  int tag, widths;
  __device__ inline void load(const RouteParams& p) {
    const int e = threadIdx.x;
    tag = e < p.E ? p.table[e].tag : 0;
    widths = e < p.E ? pack_widths(p.table[e]) : 0;
  }
  __device__ inline void store(const RouteParams& p, int* tags, int* wd) const {
    if ((int)threadIdx.x < p.E) {
      tags[threadIdx.x] = tag;
      wd[threadIdx.x] = widths;
    }
  }
};

// ---- decode fast path ------------------------------------------------------
// When the step's activations fit in LDS (T*d*2 <= 64 KiB) and d <= 4096
// (8 chunks of 512 columns per lane in registers), the gate takes
// one memory round trip: each wave issues the loads of its expert row (lane
// l holds columns 512j + 8l .. +7 of chunk j), the block stages x in LDS,
// and every token's logit is summed over the chunks in the same order as
// gate_logits, so the logits are bit-identical to the other routers'.
constexpr int kFastXBytes = 64 * 1024;
constexpr int kFastChunks = 8;  // 512-column chunks held in registers at once
constexpr int kNormBatch = 4;   // tokens per round of the fused RMSNorm
static_assert(kRouteThreads == kNormThreads, "the fused RMSNorm runs on the whole router block");

__host__ __device__ inline bool fast_gate(int T, int d) { return (int64_t)T * d * 2 <= kFastXBytes && d <= kFastChunks * 512; }

__device__ void gate_fast(const RouteParams& p, f16* xs, float* lg) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  constexpr int kW = kRouteThreads / 64;
  const int nch = (p.d + 511) / 512;
  const int e0 = wave;
  // first group of chunks of this wave's first expert row, before staging
  u32x4 b[kFastChunks];
#pragma unroll
  for (int j = 0; j < kFastChunks; ++j) {
    const int c = j * 512 + lane * 8;
    b[j] = (e0 < p.E && j < nch && c < p.d)
               ? *reinterpret_cast<const u32x4*>(p.wg + (int64_t)e0 * p.d + c)
               : u32x4{0, 0, 0, 0};
  }
  if (p.h_res) {
    // x = fp16(rmsnorm(h_res)), formed here as the residual glue's norm
    // kernel forms it (same sums, same order: bit-identical), written to
    // x_out for the expert kernels and staged in LDS for the gate
    __shared__ float red[kNormBatch * (kNormThreads / 64)];
    for (int t0 = 0; t0 < p.T; t0 += kNormBatch)
      rmsnorm_rows<kNormBatch, 1>(p.h_res, p.d, p.eps, t0, min(kNormBatch, p.T - t0), red,
                                  [&](int t, int q, uint32_t lo, uint32_t hi) {
                                    const int64_t o = (int64_t)t * p.d + 4 * q;
                                    *reinterpret_cast<u32x2*>(p.x_out + o) = u32x2{lo, hi};
                                    *reinterpret_cast<u32x2*>(xs + o) = u32x2{lo, hi};
                                  });
  } else {
    // stage x [T, d] in LDS
    const int nvec = p.T * p.d / 8;
    for (int v = threadIdx.x; v < nvec; v += kRouteThreads)
      reinterpret_cast<u32x4*>(xs)[v] = reinterpret_cast<const u32x4*>(p.x)[v];
  }
  __syncthreads();
  for (int e = e0; e < p.E; e += kW) {
    if (e != e0) {
#pragma unroll
      for (int j = 0; j < kFastChunks; ++j) {
        const int c = j * 512 + lane * 8;
        b[j] = (j < nch && c < p.d) ? *reinterpret_cast<const u32x4*>(p.wg + (int64_t)e * p.d + c)
                                    : u32x4{0, 0, 0, 0};
      }
    }
    for (int t = 0; t < p.T; ++t) {
      float acc = 0.0f;
#pragma unroll
      for (int j = 0; j < kFastChunks; ++j) {
        const int c = j * 512 + lane * 8;
        if (j < nch && c < p.d) {
          const u32x4 xv = *reinterpret_cast<const u32x4*>(xs + (int64_t)t * p.d + c);
          acc = dot2(xv.x, b[j].x, acc);
          acc = dot2(xv.y, b[j].y, acc);
          acc = dot2(xv.z, b[j].z, acc);
          acc = dot2(xv.w, b[j].w, acc);
        }
      }
      const float v = wave_sum_dpp(acc);
      if (lane == 0) lg[t * p.E + e] = v;
    }
  }
}

// Order-preserving key of a float (larger float, larger key).
__device__ inline uint32_t float_key(float v) {
  const uint32_t u = __builtin_bit_cast(uint32_t, v);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// top-k, softmax over the selected logits and the Eq. 2 rule for tokens
// wave, wave + 16, ...: lanes are experts; slot k is the wave maximum of
// (logit, -index) over the experts not yet taken, so exact ties keep the
// lower index.  The softmax and the running Eq. 2 score are evaluated in
// the same order as decide_token.
__device__ void decide_wave(const RouteParams& p, const float* lg, const int* tags,
                            RouteOut o, int32_t* s_idx, int8_t* s_prec) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  constexpr int kW = kRouteThreads / 64;
  for (int t = wave; t < p.T; t += kW) {
    float v = lane < p.E ? lg[t * p.E + lane] : -__builtin_inff();
    int sel[kMaxTopK];
    float ls[kMaxTopK];
#pragma unroll
    for (int k = 0; k < kMaxTopK; ++k) {
      if (k >= p.K) break;
      uint64_t key = ((uint64_t)float_key(v) << 32) | (uint32_t)(63 - lane);
      if (lane >= p.E) key = 0;  // never selected (E >= K experts remain)
#pragma unroll
      for (int o_ = 32; o_ > 0; o_ >>= 1) {
        const uint64_t other = __shfl_xor(key, o_, 64);
        key = other > key ? other : key;
      }
      const int e = 63 - (int)(key & 63u);
      sel[k] = e;
      ls[k] = __shfl(v, e, 64);
      if (lane == e) v = -__builtin_inff();
    }
    float ex[kMaxTopK];
    float z = 0.0f;
#pragma unroll
    for (int k = 0; k < kMaxTopK; ++k) {
      if (k < p.K) {
        ex[k] = expf(ls[k] - ls[0]);
        z += ex[k];
      }
    }
    float above = 0.0f;  // Eq. 2 running score
#pragma unroll
    for (int k = 0; k < kMaxTopK; ++k) {
      if (k >= p.K) break;
      const float w = ex[k] / z;
      const int e = sel[k];
      const int tag = tags[e];
      int prec;
      if (tag == TAG_FP16 || tag == TAG_INT8) {
        prec = PREC_HIGH;
      } else if (tag == TAG_INT4 || tag == TAG_INT2) {
        prec = PREC_LOW;
      } else {
        const float sc = (k == 0) ? 0.0f : above;
        prec = (k == 0 || sc <= p.t1) ? PREC_HIGH : (sc <= p.t2 ? PREC_LOW : PREC_SKIP);
      }
      above += w;
      if (lane == k) {
        const int pi = t * p.K + k;
        o.idx[pi] = e;
        o.w[pi] = w;
        o.prec[pi] = (int8_t)prec;
        s_idx[pi] = e;
        s_prec[pi] = (int8_t)prec;
        if (o.user_idx) o.user_idx[pi] = e;
        if (o.user_w) o.user_w[pi] = w;
        if (o.user_prec) o.user_prec[pi] = (int8_t)prec;
      }
    }
  }
}

// The stable counting sort of build_worklist for at most 64 pairs, in one
// wave: keys in increasing order, one ballot each; a pair's rank is the
// number of lower lanes with the same key.
__device__ void worklist_wave(const RouteParams& p, const int32_t* idx, const int8_t* prec,
                              const int* widths, WorkList* wl, int32_t* perm, int32_t* pos) {
  const int lane = threadIdx.x & 63;
  const int N = p.T * p.K;
  int key = -1;
  if (lane < N) {
    const int pr = prec[lane];
    if (pr != PREC_SKIP) key = idx[lane] * 2 + (pr == PREC_LOW);
    else pos[lane] = -1;
  }
  const uint64_t lower = (1ull << lane) - 1ull;
  int off = 0, ng = 0, mx = 0;
  for (int k = 0; k < 2 * p.E; ++k) {
    const uint64_t m = __ballot(key == k);
    if (m == 0) continue;
    const int c = __popcll(m);
    if (key == k) {
      const int at = off + __popcll(m & lower);
      perm[at] = lane;
      pos[lane] = at;
    }
    if (lane == 0) {
      Group g;
      g.expert = k >> 1;
      g.bits = copy_bits(widths[k >> 1], k & 1);
      g.offset = off;
      g.count = c;
      wl->groups[ng] = g;
    }
    ++ng;
    off += c;
    mx = c > mx ? c : mx;
  }
  if (lane == 0) {
    wl->n_groups = ng;
    wl->max_count = mx;
  }
}

// Decode: one block routes every token and builds the work list.
__global__ __launch_bounds__(kRouteThreads) void route_decode_kernel(
    RouteParams p, RouteOut o, WorkList* wl, int32_t* perm, int32_t* pos) {
  __shared__ float lg[kDecodeMaxTokens * kMaxExperts];
  __shared__ int tags[kMaxExperts], widths[kMaxExperts];
  __shared__ int32_t s_idx[kDecodeMaxTokens * kMaxTopK];
  __shared__ int8_t s_prec[kDecodeMaxTokens * kMaxTopK];
  __shared__ __attribute__((aligned(16))) f16 xs[kFastXBytes / 2];
  TableRow tr;
  tr.load(p);
  const bool fast = fast_gate(p.T, p.d);
  if (fast) gate_fast(p, xs, lg);
  else if (p.T == 1) gate_logits<1, 8>(p, 0, p.T, lg);
  else if (p.T == 2) gate_logits<2, 8>(p, 0, p.T, lg);
  else gate_logits<4, 4>(p, 0, p.T, lg);
  tr.store(p, tags, widths);
  __syncthreads();
  decide_wave(p, lg, tags, o, s_idx, s_prec);
  __syncthreads();
  if (p.T * p.K <= 64) {
    if (threadIdx.x < 64) worklist_wave(p, s_idx, s_prec, widths, wl, perm, pos);
  } else {
    build_worklist(p, s_idx, s_prec, widths, wl, perm, pos);
  }
}

// Prefill: many blocks route their tokens; a second kernel builds the list.
__global__ __launch_bounds__(kPrefillThreads) void route_tokens_kernel(
    RouteParams p, RouteOut o) {
  __shared__ float lg[kPrefillTokPerBlock * kMaxExperts];
  __shared__ int tags[kMaxExperts], widths[kMaxExperts];
  const int t0 = blockIdx.x * kPrefillTokPerBlock;
  const int t1 = min(t0 + kPrefillTokPerBlock, p.T);
  stage_table(p, tags, widths);
  gate_logits<kPrefillTokPerBlock, 8>(p, t0, t1, lg);
  __syncthreads();
  for (int t = t0 + (int)threadIdx.x; t < t1; t += blockDim.x)
    decide_token(p, t, lg + (t - t0) * p.E, tags, o);
}

__global__ __launch_bounds__(kRouteThreads) void worklist_kernel(
    RouteParams p, RouteOut o, WorkList* wl, int32_t* perm, int32_t* pos) {
  __shared__ int tags[kMaxExperts], widths[kMaxExperts];
  stage_table(p, tags, widths);
  __syncthreads();
  build_worklist(p, o.idx, o.prec, widths, wl, perm, pos);
}

}  // namespace

bool route_decode_fuses_norm(int T, int d) { return fast_gate(T, d); }

hipError_t launch_route_decode(const RouteParams& p, RouteOut o, WorkList* wl,
                               int32_t* perm, int32_t* pos, hipStream_t s) {
  // the fused RMSNorm exists on the LDS-staged gate path only
  if (p.h_res && !fast_gate(p.T, p.d)) return hipErrorInvalidValue;
  route_decode_kernel<<<1, kRouteThreads, 0, s>>>(p, o, wl, perm, pos);
  return hipGetLastError();
}

hipError_t launch_route_prefill(const RouteParams& p, RouteOut o, WorkList* wl,
                                int32_t* perm, int32_t* pos, hipStream_t s) {
  const int blocks = (p.T + kPrefillTokPerBlock - 1) / kPrefillTokPerBlock;
  route_tokens_kernel<<<blocks, kPrefillThreads, 0, s>>>(p, o);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  worklist_kernel<<<1, kRouteThreads, 0, s>>>(p, o, wl, perm, pos);
  return hipGetLastError();
}

}  // namespace moe
