// Stacking Computer of the Adaptive Expert Predictor (Section 3.3, "Expert
// predictor design", Fig. 7).
//
// Gating inputs of consecutive layers are similar, so the gates of the
// next p layers applied to the current layer's gating input predict which
// experts those layers will select.  Instead of evaluating the p gates one
// after the other, the p weight matrices [E, d] are stacked into one
// [p*E, d] array and evaluated as one product:
//
//   L[t, j*E + e] = x[t, :] . Wg_{l+j}[e, :]                 (fp32 accumulate)
//
// then per token and predicted layer j: top-k over that layer's E logits
// (largest first, exact ties to the lower index) and the softmax over the
// K selected logits, as the layer's own router does.  The adaptive walk:
// j = 1, 2, ... continues while every predicted expert of layer l+j is in
// the expert cache and stops at the first layer with a missing one; its
// missing experts are reported for preloading.
//
// One launch.  Every wave takes (stacked row, batch of up to TB tokens)
// items of the product, so the p*E rows are spread over the whole grid and
// the time stays that of one gate while p*E rows fit in one wave each.  The
// last block to finish (a device-scope counter) does the per-layer top-k
// and the walk, and resets the counter for the next launch.
#include "moe_internal.h"

namespace moe {

namespace {

constexpr int kPredThreads = 256;

__device__ inline float dot2(uint32_t a, uint32_t b, float acc) {
  // operands as scalars: __builtin_bit_cast of a vector component reads
  // component 0 with this compiler
  return __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2, a),
                                __builtin_bit_cast(f16x2, b), acc, false);
}

__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

template <int TB, int KB>
__global__ __launch_bounds__(kPredThreads) void predict_kernel(PredictParams q) {
  const int lane = threadIdx.x & 63;
  const int gw = blockIdx.x * (kPredThreads / 64) + (threadIdx.x >> 6);
  const int n_gw = gridDim.x * (kPredThreads / 64);
  const int R = q.p * q.E;
  const int n_tb = (q.T + TB - 1) / TB;
  // ---- stacked product: one (row, token batch) item per wave at a time
  for (int it = gw; it < R * n_tb; it += n_gw) {
    const int r = it % R;
    const int tb0 = (it / R) * TB;
    const int nt = min(TB, q.T - tb0);
    const f16* gr = q.wstack + (int64_t)r * q.d;
    float acc[TB];
#pragma unroll
    for (int i = 0; i < TB; ++i) acc[i] = 0.0f;
    for (int c0 = 0; c0 < q.d; c0 += KB * 512) {
      u32x4 b[KB], a[TB][KB];
#pragma unroll
      for (int j = 0; j < KB; ++j) {
        const int c = c0 + j * 512 + lane * 8;
        b[j] = c < q.d ? *reinterpret_cast<const u32x4*>(gr + c) : u32x4{0, 0, 0, 0};
#pragma unroll
        for (int i = 0; i < TB; ++i)
          a[i][j] = (i < nt && c < q.d)
                        ? *reinterpret_cast<const u32x4*>(q.x + (int64_t)(tb0 + i) * q.d + c)
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
      const float v = wave_sum(acc[i]);
      if (lane == 0 && i < nt) q.logits[(int64_t)(tb0 + i) * R + r] = v;
    }
  }

  // ---- the last block to finish: per-layer top-k, softmax and the walk
  __shared__ int s_last;
  __shared__ unsigned long long s_need[kMaxPredLayers];
  __threadfence();  // this block's logits are visible device-wide
  __syncthreads();
  if (threadIdx.x == 0) s_last = atomicAdd(q.counter, 1u) == gridDim.x - 1;
  __syncthreads();
  if (!s_last) return;
  __threadfence();  // every block's logits are visible to this one
  if ((int)threadIdx.x < q.p) s_need[threadIdx.x] = 0ull;
  __syncthreads();
  for (int v = threadIdx.x; v < q.T * q.p; v += blockDim.x) {
    const int t = v / q.p, j = v - (v / q.p) * q.p;
    const float* lrow = q.logits + (int64_t)t * R + j * q.E;
    int sel[kMaxTopK];
    float ls[kMaxTopK];
    unsigned long long taken = 0ull;  // E <= 64
    for (int k = 0; k < q.K; ++k) {
      int best = -1;
      float bv = 0.0f;
      for (int e = 0; e < q.E; ++e) {
        if (taken >> e & 1ull) continue;
        const float lv = lrow[e];
        if (best < 0 || lv > bv) {  // strict: exact ties keep the lower index
          best = e;
          bv = lv;
        }
      }
      taken |= 1ull << best;
      sel[k] = best;
      ls[k] = bv;
    }
    float ex[kMaxTopK];
    float z = 0.0f;
    for (int k = 0; k < q.K; ++k) {
      ex[k] = expf(ls[k] - ls[0]);
      z += ex[k];
    }
    const int64_t o = ((int64_t)t * q.p + j) * q.K;
    for (int k = 0; k < q.K; ++k) {
      q.idx[o + k] = sel[k];
      if (q.w) q.w[o + k] = ex[k] / z;
    }
    atomicOr(&s_need[j], taken);
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int first = 0;
    unsigned long long pre = 0ull;
    for (int j = 0; j < q.p; ++j) {
      const unsigned long long m = s_need[j] & ~(unsigned long long)q.cached[j];
      if (m) {
        first = j + 1;
        pre = m;
        break;
      }
    }
    *q.first_miss = first;
    *q.preload = pre;
    *q.counter = 0u;  // ready for the next launch on the stream
  }
}

}  // namespace

hipError_t launch_predict(const PredictParams& q, hipStream_t s) {
  const int waves = kPredThreads / 64;
  const int R = q.p * q.E;
  const int tb = q.T == 1 ? 1 : (q.T == 2 ? 2 : 4);
  const int items = R * ((q.T + tb - 1) / tb);
  const int blocks = std::min((items + waves - 1) / waves, 1024);
  if (q.T == 1) predict_kernel<1, 8><<<blocks, kPredThreads, 0, s>>>(q);
  else if (q.T == 2) predict_kernel<2, 8><<<blocks, kPredThreads, 0, s>>>(q);
  else predict_kernel<4, 4><<<blocks, kPredThreads, 0, s>>>(q);
  return hipGetLastError();
}

}  // namespace moe
