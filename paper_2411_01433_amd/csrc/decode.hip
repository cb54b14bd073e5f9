// Decode-path expert kernels: fused dequantise-GEMV for the SwiGLU experts
// of Eq. 1 at fp16, int4 or int2, and the weighted combine.
//
//   up:    h[p, r] = silu(W1[r,:] . x_t) * (W3[r,:] . x_t)   (fp16 out)
//   down:  part[s, p, r] = W2[r, cols of split s] . h[p, cols of split s]
//   combine: y[t] = sum_k w[t,k] * sum_s part[s, t*K+k]      (skip -> 0)
//
// One block handles one (expert, precision) work group and a tile of rows,
// so the weights of every selected expert copy are streamed from HBM once
// per step whatever the number of tokens routed to it.  Lanes of a wave
// read consecutive 16-byte pieces of a row (1 KiB per wave-wide load); the
// group's activations are staged in LDS in the element order the
// dequantiser produces, and each lane accumulates with v_dot2_f32_f16
// (fp16 x fp16 products are exact in fp32).  A low-precision group is
// summed as q . x in fp32 and scaled once by its fp16 scale.
#include "moe_internal.h"

namespace moe {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kRowsPerWave = 2;
constexpr int kRowsPerBlock = kWaves * kRowsPerWave;
constexpr int kLdsHalves = 32768;  // at most 64 KiB of staged activations
constexpr int kMaxChunkTokens = 8;

__device__ inline f16x2 as_h2(uint32_t v) { return __builtin_bit_cast(f16x2, v); }

__device__ inline float dot2(uint32_t a, uint32_t b, float acc) {
  return __builtin_amdgcn_fdot2(as_h2(a), as_h2(b), acc, false);
}

__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// int4 word holding elements e0..e7 (e_j at bits 4j) -> four fp16 pairs
// (e_k, e_{k+4}) - 8, k = 0..3, using 0x6400|u == 1024 + u exactly.
__device__ inline void dequant4(uint32_t w, uint32_t out[4]) {
  const f16x2 bias = as_h2(0x64086408u);  // 1032
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    f16x2 v = as_h2(((w >> (4 * k)) & 0x000F000Fu) | 0x64006400u) - bias;
    out[k] = __builtin_bit_cast(uint32_t, v);
  }
}

// int2 word holding e0..e15 (e_j at bits 2j) -> eight pairs (e_k, e_{k+8}) - 2.
__device__ inline void dequant2(uint32_t w, uint32_t out[8]) {
  const f16x2 bias = as_h2(0x64026402u);  // 1026
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    f16x2 v = as_h2(((w >> (2 * k)) & 0x00030003u) | 0x64006400u) - bias;
    out[k] = __builtin_bit_cast(uint32_t, v);
  }
}

// Position of element j of a 16-element block in the staged layout.
template <int BITS>
__device__ inline int staged_pos(int j) {
  if (BITS == 4) {  // per 8: x0 x4 x1 x5 x2 x6 x3 x7
    const int b = j & 8, i = j & 7;
    return b + (i < 4 ? 2 * i : 2 * (i - 4) + 1);
  }
  if (BITS == 2) return j < 8 ? 2 * j : 2 * (j - 8) + 1;  // x0 x8 x1 x9 ...
  return j;
}

// Stage rows [j0, j0+n) of the group's pair list into LDS [nt][width]:
// source row = perm[..]/K (token rows of x) or perm[..] (pair rows of h),
// columns [c0, c0+width).  Rows n..nt-1 are zero.
template <int BITS>
__device__ void stage(f16* lds, const f16* src, int64_t ld, const int32_t* pairs,
                      int n, int nt, int K, bool by_token, int c0, int width) {
  const int bpr = width / 16;
  for (int b = threadIdx.x; b < nt * bpr; b += kThreads) {
    const int j = b / bpr, cb = (b - j * bpr) * 16;
    u32x4 lo = {0, 0, 0, 0}, hi = {0, 0, 0, 0};
    if (j < n) {
      const int p = pairs[j];
      const int64_t row = by_token ? p / K : p;
      const u32x4* s = reinterpret_cast<const u32x4*>(src + row * ld + c0 + cb);
      lo = s[0];
      hi = s[1];
    }
    f16x8 a = __builtin_bit_cast(f16x8, lo), c = __builtin_bit_cast(f16x8, hi);
    f16 v[16], o[16];
#pragma unroll
    for (int i = 0; i < 8; ++i) { v[i] = a[i]; v[8 + i] = c[i]; }
#pragma unroll
    for (int i = 0; i < 16; ++i) o[staged_pos<BITS>(i)] = v[i];
    f16x8 oa, oc;
#pragma unroll
    for (int i = 0; i < 8; ++i) { oa[i] = o[i]; oc[i] = o[8 + i]; }
    u32x4* d = reinterpret_cast<u32x4*>(lds + j * width + cb);
    d[0] = __builtin_bit_cast(u32x4, oa);
    d[1] = __builtin_bit_cast(u32x4, oc);
  }
}

// Row dot products of NM matrices (same row index, same activations) for
// kRowsPerWave rows starting at row0, columns [c0, c0+width) of rows of
// length ld, against NT staged activation rows.  acc is per lane (partial).
template <int BITS, int NT, int NM>
struct RowDot;

template <int NT, int NM>
struct RowDot<16, NT, NM> {
  static __device__ void run(const ExpertEntry& ex, const int* mats, int row0,
                             int64_t ld, int c0, int width, const f16* xs,
                             float (&acc)[NM][kRowsPerWave][NT]) {
    const int lane = threadIdx.x & 63;
    for (int c = lane * 8; c < width; c += 64 * 8) {
      u32x4 wv[NM][kRowsPerWave];
#pragma unroll
      for (int m = 0; m < NM; ++m)
#pragma unroll
        for (int i = 0; i < kRowsPerWave; ++i)
          wv[m][i] = *reinterpret_cast<const u32x4*>(
              ex.w[mats[m]] + (int64_t)(row0 + i) * ld + c0 + c);
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const u32x4 xv = *reinterpret_cast<const u32x4*>(xs + t * width + c);
#pragma unroll
        for (int m = 0; m < NM; ++m)
#pragma unroll
          for (int i = 0; i < kRowsPerWave; ++i) {
            float a = acc[m][i][t];
            a = dot2(wv[m][i].x, xv.x, a);
            a = dot2(wv[m][i].y, xv.y, a);
            a = dot2(wv[m][i].z, xv.z, a);
            a = dot2(wv[m][i].w, xv.w, a);
            acc[m][i][t] = a;
          }
      }
    }
  }
};

template <int NT, int NM>
struct RowDot<4, NT, NM> {
  static __device__ void run(const ExpertEntry& ex, const int* mats, int row0,
                             int64_t ld, int c0, int width, const f16* xs,
                             float (&acc)[NM][kRowsPerWave][NT]) {
    const int lane = threadIdx.x & 63;
    const int64_t ldq = ld / 2, lds_ = ld / kGroup;
    for (int c = lane * 32; c < width; c += 64 * 32) {
      const int64_t col = c0 + c;
      u32x4 qv[NM][kRowsPerWave];
      float sv[NM][kRowsPerWave];
#pragma unroll
      for (int m = 0; m < NM; ++m)
#pragma unroll
        for (int i = 0; i < kRowsPerWave; ++i) {
          const int64_t r = row0 + i;
          qv[m][i] = *reinterpret_cast<const u32x4*>(ex.q[mats[m]] + r * ldq + col / 2);
          sv[m][i] = (float)ex.s[mats[m]][r * lds_ + col / kGroup];
        }
#pragma unroll
      for (int m = 0; m < NM; ++m)
#pragma unroll
        for (int i = 0; i < kRowsPerWave; ++i) {
          uint32_t dq[16];
          dequant4(qv[m][i].x, dq + 0);
          dequant4(qv[m][i].y, dq + 4);
          dequant4(qv[m][i].z, dq + 8);
          dequant4(qv[m][i].w, dq + 12);
#pragma unroll
          for (int t = 0; t < NT; ++t) {
            const u32x4* xp = reinterpret_cast<const u32x4*>(xs + t * width + c);
            float g = 0.0f;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
              const u32x4 xv = xp[k];
              g = dot2(dq[4 * k + 0], xv.x, g);
              g = dot2(dq[4 * k + 1], xv.y, g);
              g = dot2(dq[4 * k + 2], xv.z, g);
              g = dot2(dq[4 * k + 3], xv.w, g);
            }
            acc[m][i][t] = fmaf(sv[m][i], g, acc[m][i][t]);
          }
        }
    }
  }
};

template <int NT, int NM>
struct RowDot<2, NT, NM> {
  static __device__ void run(const ExpertEntry& ex, const int* mats, int row0,
                             int64_t ld, int c0, int width, const f16* xs,
                             float (&acc)[NM][kRowsPerWave][NT]) {
    const int lane = threadIdx.x & 63;
    const int64_t ldq = ld / 4, lds_ = ld / kGroup;
    for (int c = lane * 64; c < width; c += 64 * 64) {
      const int64_t col = c0 + c;
      u32x4 qv[NM][kRowsPerWave];
      uint32_t sv[NM][kRowsPerWave];
#pragma unroll
      for (int m = 0; m < NM; ++m)
#pragma unroll
        for (int i = 0; i < kRowsPerWave; ++i) {
          const int64_t r = row0 + i;
          qv[m][i] = *reinterpret_cast<const u32x4*>(ex.q[mats[m]] + r * ldq + col / 4);
          sv[m][i] = *reinterpret_cast<const uint32_t*>(ex.s[mats[m]] + r * lds_ + col / kGroup);
        }
#pragma unroll
      for (int m = 0; m < NM; ++m)
#pragma unroll
        for (int i = 0; i < kRowsPerWave; ++i) {
          const f16x2 s2 = as_h2(sv[m][i]);
          uint32_t dq[32];
          dequant2(qv[m][i].x, dq + 0);
          dequant2(qv[m][i].y, dq + 8);
          dequant2(qv[m][i].z, dq + 16);
          dequant2(qv[m][i].w, dq + 24);
#pragma unroll
          for (int t = 0; t < NT; ++t) {
            const u32x4* xp = reinterpret_cast<const u32x4*>(xs + t * width + c);
            float g0 = 0.0f, g1 = 0.0f;
#pragma unroll
            for (int k = 0; k < 2; ++k) {
              const u32x4 xv = xp[k];
              g0 = dot2(dq[4 * k + 0], xv.x, g0);
              g0 = dot2(dq[4 * k + 1], xv.y, g0);
              g0 = dot2(dq[4 * k + 2], xv.z, g0);
              g0 = dot2(dq[4 * k + 3], xv.w, g0);
            }
#pragma unroll
            for (int k = 2; k < 4; ++k) {
              const u32x4 xv = xp[k];
              g0 = dot2(dq[4 * k + 0], xv.x, g0);
              g0 = dot2(dq[4 * k + 1], xv.y, g0);
              g0 = dot2(dq[4 * k + 2], xv.z, g0);
              g0 = dot2(dq[4 * k + 3], xv.w, g0);
            }
#pragma unroll
            for (int k = 4; k < 8; ++k) {
              const u32x4 xv = xp[k];
              g1 = dot2(dq[4 * k + 0], xv.x, g1);
              g1 = dot2(dq[4 * k + 1], xv.y, g1);
              g1 = dot2(dq[4 * k + 2], xv.z, g1);
              g1 = dot2(dq[4 * k + 3], xv.w, g1);
            }
            float a = fmaf((float)s2[0], g0, acc[m][i][t]);
            acc[m][i][t] = fmaf((float)s2[1], g1, a);
          }
        }
    }
  }
};

// ---------------------------------------------------------------- up-proj
template <int BITS, int NT>
__device__ void up_chunk(const ExpertEntry& ex, const int32_t* pairs, int n,
                         const f16* x, f16* h, int d, int f, int K, int row0,
                         f16* lds) {
  stage<BITS>(lds, x, d, pairs, n, NT, K, true, 0, d);
  __syncthreads();
  float acc[2][kRowsPerWave][NT];
#pragma unroll
  for (int m = 0; m < 2; ++m)
#pragma unroll
    for (int i = 0; i < kRowsPerWave; ++i)
#pragma unroll
      for (int t = 0; t < NT; ++t) acc[m][i][t] = 0.0f;
  const int mats[2] = {0, 1};
  RowDot<BITS, NT, 2>::run(ex, mats, row0, d, 0, d, lds, acc);
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int i = 0; i < kRowsPerWave; ++i)
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const float a = wave_sum(acc[0][i][t]);
      const float b = wave_sum(acc[1][i][t]);
      if (lane == i * NT + t && t < n) {
        const float hv = a / (1.0f + expf(-a)) * b;
        h[(int64_t)pairs[t] * f + row0 + i] = (f16)hv;
      }
    }
  __syncthreads();
}

// Token chunks of at most NTMAX (the host's bound: min(T, LDS capacity)),
// each run by the smallest power-of-two instantiation that holds it.
template <int BITS, int NTMAX>
__device__ void up_group(const ExpertEntry& ex, const int32_t* pairs, int count,
                         const f16* x, f16* h, int d, int f, int K, int row0,
                         f16* lds) {
  for (int j0 = 0; j0 < count; j0 += NTMAX) {
    const int n = min(NTMAX, count - j0);
    if (NTMAX == 1 || n <= 1) up_chunk<BITS, 1>(ex, pairs + j0, n, x, h, d, f, K, row0, lds);
    else if (NTMAX == 2 || n <= 2) up_chunk<BITS, (NTMAX < 2 ? NTMAX : 2)>(ex, pairs + j0, n, x, h, d, f, K, row0, lds);
    else if (NTMAX == 4 || n <= 4) up_chunk<BITS, (NTMAX < 4 ? NTMAX : 4)>(ex, pairs + j0, n, x, h, d, f, K, row0, lds);
    else up_chunk<BITS, NTMAX>(ex, pairs + j0, n, x, h, d, f, K, row0, lds);
  }
}

template <int NTMAX>
__global__ __launch_bounds__(kThreads) void decode_up_kernel(
    const ExpertEntry* __restrict__ table, const WorkList* __restrict__ wl,
    const int32_t* __restrict__ perm, const f16* __restrict__ x,
    f16* __restrict__ h, int d, int f, int K) {
  extern __shared__ f16 lds[];
  if ((int)blockIdx.y >= wl->n_groups) return;
  const Group g = wl->groups[blockIdx.y];
  const ExpertEntry ex = table[g.expert];
  const int row0 = blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6) * kRowsPerWave;
  const int32_t* pairs = perm + g.offset;
  if (g.bits == 16) up_group<16, NTMAX>(ex, pairs, g.count, x, h, d, f, K, row0, lds);
  else if (g.bits == 4) up_group<4, NTMAX>(ex, pairs, g.count, x, h, d, f, K, row0, lds);
  else up_group<2, NTMAX>(ex, pairs, g.count, x, h, d, f, K, row0, lds);
}

// -------------------------------------------------------------- down-proj
template <int BITS, int NT>
__device__ void down_chunk(const ExpertEntry& ex, const int32_t* pairs, int n,
                           const f16* h, float* part, int T, int d, int f,
                           int K, int row0, int split, f16* lds) {
  const int c0 = split * kSplitCols;
  const int width = min(kSplitCols, f - c0);
  stage<BITS>(lds, h, f, pairs, n, NT, K, false, c0, width);
  __syncthreads();
  float acc[1][kRowsPerWave][NT];
#pragma unroll
  for (int i = 0; i < kRowsPerWave; ++i)
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[0][i][t] = 0.0f;
  const int mats[1] = {2};
  RowDot<BITS, NT, 1>::run(ex, mats, row0, f, c0, width, lds, acc);
  const int lane = threadIdx.x & 63;
  float* out = part + (int64_t)split * T * K * d;
#pragma unroll
  for (int i = 0; i < kRowsPerWave; ++i)
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const float v = wave_sum(acc[0][i][t]);
      if (lane == i * NT + t && t < n) out[(int64_t)pairs[t] * d + row0 + i] = v;
    }
  __syncthreads();
}

template <int BITS, int NTMAX>
__device__ void down_group(const ExpertEntry& ex, const int32_t* pairs,
                           int count, const f16* h, float* part, int T, int d,
                           int f, int K, int row0, int split, f16* lds) {
  for (int j0 = 0; j0 < count; j0 += NTMAX) {
    const int n = min(NTMAX, count - j0);
    if (NTMAX == 1 || n <= 1) down_chunk<BITS, 1>(ex, pairs + j0, n, h, part, T, d, f, K, row0, split, lds);
    else if (NTMAX == 2 || n <= 2) down_chunk<BITS, (NTMAX < 2 ? NTMAX : 2)>(ex, pairs + j0, n, h, part, T, d, f, K, row0, split, lds);
    else if (NTMAX == 4 || n <= 4) down_chunk<BITS, (NTMAX < 4 ? NTMAX : 4)>(ex, pairs + j0, n, h, part, T, d, f, K, row0, split, lds);
    else down_chunk<BITS, NTMAX>(ex, pairs + j0, n, h, part, T, d, f, K, row0, split, lds);
  }
}

template <int NTMAX>
__global__ __launch_bounds__(kThreads) void decode_down_kernel(
    const ExpertEntry* __restrict__ table, const WorkList* __restrict__ wl,
    const int32_t* __restrict__ perm, const f16* __restrict__ h,
    float* __restrict__ part, int T, int d, int f, int K, int row_tiles) {
  extern __shared__ f16 lds[];
  if ((int)blockIdx.y >= wl->n_groups) return;
  const Group g = wl->groups[blockIdx.y];
  const ExpertEntry ex = table[g.expert];
  const int tile = blockIdx.x % row_tiles;
  const int split = blockIdx.x / row_tiles;
  const int row0 = tile * kRowsPerBlock + (threadIdx.x >> 6) * kRowsPerWave;
  const int32_t* pairs = perm + g.offset;
  if (g.bits == 16) down_group<16, NTMAX>(ex, pairs, g.count, h, part, T, d, f, K, row0, split, lds);
  else if (g.bits == 4) down_group<4, NTMAX>(ex, pairs, g.count, h, part, T, d, f, K, row0, split, lds);
  else down_group<2, NTMAX>(ex, pairs, g.count, h, part, T, d, f, K, row0, split, lds);
}

// ---------------------------------------------------------------- combine
__device__ inline float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  float s = 0.0f;
  for (int i = 0; i < (int)(blockDim.x >> 6); ++i) s += red[i];
  return s;
}

__global__ __launch_bounds__(kThreads) void combine_decode_kernel(
    const float* __restrict__ part, const float* __restrict__ w,
    const int8_t* __restrict__ prec, int n_split, int T, int d, int K,
    float* __restrict__ y, float* __restrict__ h_res, f16* __restrict__ x_next,
    float eps) {
  __shared__ float red[kThreads / 64];
  const int t = blockIdx.x;
  const int64_t split_stride = (int64_t)T * K * d;
  float ss = 0.0f;
  for (int c = threadIdx.x; c < d; c += blockDim.x) {
    float acc = 0.0f;
    for (int k = 0; k < K; ++k) {
      const int p = t * K + k;
      if (prec[p] == PREC_SKIP) continue;
      float e = 0.0f;
      for (int s = 0; s < n_split; ++s) e += part[s * split_stride + (int64_t)p * d + c];
      acc = fmaf(w[p], e, acc);
    }
    if (h_res) {
      const float v = h_res[(int64_t)t * d + c] + acc;
      h_res[(int64_t)t * d + c] = v;
      ss = fmaf(v, v, ss);
    } else {
      y[(int64_t)t * d + c] = acc;
    }
  }
  if (!h_res) return;
  const float tot = block_sum(ss, red);
  const float r = 1.0f / sqrtf(tot / (float)d + eps);
  for (int c = threadIdx.x; c < d; c += blockDim.x)
    x_next[(int64_t)t * d + c] = (f16)(h_res[(int64_t)t * d + c] * r);
}

int chunk_tokens(int width) {
  int c = kLdsHalves / width;
  return c >= kMaxChunkTokens ? kMaxChunkTokens : (c >= 4 ? 4 : (c >= 2 ? 2 : 1));
}

int lds_tokens(int chunk, int T) {
  const int n = T < chunk ? T : chunk;
  return n <= 1 ? 1 : (n <= 2 ? 2 : (n <= 4 ? 4 : 8));
}

}  // namespace

hipError_t launch_decode_up(const ExpertEntry* table, const WorkList* wl,
                            const int32_t* perm, const f16* x, f16* h, int T,
                            int d, int f, int K, int max_groups, hipStream_t s) {
  const int nt = lds_tokens(chunk_tokens(d), T);
  const size_t lds = (size_t)nt * d * sizeof(f16);
  dim3 grid(f / kRowsPerBlock, max_groups);
  switch (nt) {
    case 1: decode_up_kernel<1><<<grid, kThreads, lds, s>>>(table, wl, perm, x, h, d, f, K); break;
    case 2: decode_up_kernel<2><<<grid, kThreads, lds, s>>>(table, wl, perm, x, h, d, f, K); break;
    case 4: decode_up_kernel<4><<<grid, kThreads, lds, s>>>(table, wl, perm, x, h, d, f, K); break;
    default: decode_up_kernel<8><<<grid, kThreads, lds, s>>>(table, wl, perm, x, h, d, f, K); break;
  }
  return hipGetLastError();
}

hipError_t launch_decode_down(const ExpertEntry* table, const WorkList* wl,
                              const int32_t* perm, const f16* h, float* part,
                              int T, int d, int f, int K, int max_groups,
                              hipStream_t s) {
  const int nt = lds_tokens(chunk_tokens(kSplitCols), T);
  const int width = f < kSplitCols ? f : kSplitCols;
  const size_t lds = (size_t)nt * width * sizeof(f16);
  const int row_tiles = d / kRowsPerBlock;
  const int n_split = (f + kSplitCols - 1) / kSplitCols;
  dim3 grid(row_tiles * n_split, max_groups);
  switch (nt) {
    case 1: decode_down_kernel<1><<<grid, kThreads, lds, s>>>(table, wl, perm, h, part, T, d, f, K, row_tiles); break;
    case 2: decode_down_kernel<2><<<grid, kThreads, lds, s>>>(table, wl, perm, h, part, T, d, f, K, row_tiles); break;
    case 4: decode_down_kernel<4><<<grid, kThreads, lds, s>>>(table, wl, perm, h, part, T, d, f, K, row_tiles); break;
    default: decode_down_kernel<8><<<grid, kThreads, lds, s>>>(table, wl, perm, h, part, T, d, f, K, row_tiles); break;
  }
  return hipGetLastError();
}

hipError_t launch_combine_decode(const float* part, const float* w,
                                 const int8_t* prec, int n_split, int T, int d,
                                 int K, float* y, float* h_res, f16* x_next,
                                 float eps, hipStream_t s) {
  combine_decode_kernel<<<T, kThreads, 0, s>>>(part, w, prec, n_split, T, d, K,
                                               y, h_res, x_next, eps);
  return hipGetLastError();
}

}  // namespace moe
