// Internal types shared by the HIP kernels and the host runtime of the
// mixed-precision MoE layer.  Not part of the public ABI (include/moe.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace moe {

typedef _Float16 f16;
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kGroup = 32;          // quantisation group along the input dim
constexpr int kMaxExperts = 64;
constexpr int kMaxTopK = 8;
constexpr int kMaxKeys = 2 * kMaxExperts;  // (expert, high|low) work groups
constexpr int kDecodeMaxTokens = 64;
constexpr int kDecodeDot2MaxTokens = 8;  // most tokens per step the dot2 decode kernels take

enum { PREC_HIGH = 0, PREC_LOW = 1, PREC_SKIP = 2 };
enum { TAG_FP16 = 0, TAG_INT4 = 1, TAG_INT2 = 2, TAG_MISS_INT4 = 3,
       TAG_MISS_INT2 = 4, TAG_INT8 = 5, TAG_MISS_INT8_INT2 = 6 };

// Device-side expert table entry: where each copy of one expert lives and
// which cache state (tag) it is in.
struct ExpertEntry {
  const f16* w[3];       // fp16 W1, W3 ([f, d]) and W2 ([d, f]); borrowed
  const uint8_t* q[3];   // packed codes of the low copy (bits = low_bits)
  const f16* s[3];       // fp16 group scales of the low copy
  const uint8_t* hq[3];  // int8 codes of the high copy when hi_bits == 8
  const f16* hs[3];      // fp16 group scales of the int8 high copy
  int32_t tag;           // TAG_*
  int32_t low_bits;      // 4 or 2 when a low copy exists, else 0
  int32_t hi_bits;       // 16 (fp16 high copy) or 8 (int8 high copy)
  int32_t pad;
};

// One work group: every (token, slot) pair routed to `expert` at one
// precision.  Pairs are listed contiguously in perm[offset, offset+count).
struct Group {
  int32_t expert;
  int32_t bits;    // 16 (fp16 copy), 8 (int8 high copy), 4 or 2
  int32_t offset;
  int32_t count;
};

struct WorkList {
  int32_t n_groups;
  int32_t max_count;   // largest group (tokens of the busiest expert copy)
  int32_t pad[2];
  Group groups[kMaxKeys];
};

// ---- device helpers shared by several kernels ------------------------------

// Sum over the 64 lanes of a wave in registers (every lane gets the sum):
// butterflies inside each 16-lane row by DPP (lane ^ 1, lane ^ 2, mirror in
// 8, mirror in 16), then the rows pairwise by v_permlane16_swap and the
// halves by v_permlane32_swap.  __shfl_xor goes through LDS permutes
// (ds_bpermute), about a hundred cycles per step.
template <int CTRL>
__device__ inline float dpp_f(float v) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
__device__ inline float wave_sum_dpp(float v) {
  v += dpp_f<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp_f<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp_f<0x141>(v);  // row_half_mirror
  v += dpp_f<0x140>(v);  // row_mirror
  const uint32_t u = __builtin_bit_cast(uint32_t, v);
  const auto r16 = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  v = __builtin_bit_cast(float, (uint32_t)r16[0]) + __builtin_bit_cast(float, (uint32_t)r16[1]);
  const uint32_t w = __builtin_bit_cast(uint32_t, v);
  const auto r32 = __builtin_amdgcn_permlane32_swap(w, w, false, false);
  return __builtin_bit_cast(float, (uint32_t)r32[0]) + __builtin_bit_cast(float, (uint32_t)r32[1]);
}

// Residual RMSNorm of the residual glue, x = fp16(v / sqrt(mean(v^2) + eps)),
// for rows t0 .. t0 + nb - 1 (nb <= NB) of h (fp32 [*, d], d a multiple of 64
// and at most 4096 * PIECES), by one block of kNormThreads threads.  Thread i
// holds float4 pieces i, i + 1024, ... of a row in registers (h is read
// once) and sums their squares with fmaf in element order; the sum goes over
// the wave in registers and then over the 16 waves in index order.  Every
// caller forms the same sums in the same order, so x is bit-identical
// whichever kernel computes it (pieces past the row add exact zeros).
// store(t, q, lo, hi) receives piece q of row t as two fp16 pairs.  `red`:
// NB * 16 floats of LDS.  Ends with a barrier (red may be reused).
constexpr int kNormThreads = 1024;
constexpr int kNormPieces = 4;  // float4 pieces per thread: 16384 / (1024 * 4)

template <int NB, int PIECES, class Store>
__device__ inline void rmsnorm_rows(const float* __restrict__ h, int d, float eps, int t0,
                                    int nb, float* red, Store store) {
  const int n4 = d >> 2;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  f32x4 v[NB][PIECES];
  float ss[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    ss[b] = 0.0f;
    const f32x4* src = reinterpret_cast<const f32x4*>(h + (int64_t)(t0 + (b < nb ? b : 0)) * d);
#pragma unroll
    for (int i = 0; i < PIECES; ++i) {
      const int q = threadIdx.x + i * kNormThreads;
      v[b][i] = (b < nb && q < n4) ? src[q] : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
      ss[b] = fmaf(v[b][i].x, v[b][i].x, ss[b]);
      ss[b] = fmaf(v[b][i].y, v[b][i].y, ss[b]);
      ss[b] = fmaf(v[b][i].z, v[b][i].z, ss[b]);
      ss[b] = fmaf(v[b][i].w, v[b][i].w, ss[b]);
    }
  }
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const float s = wave_sum_dpp(ss[b]);
    if (lane == 0) red[b * (kNormThreads / 64) + wave] = s;
  }
  __syncthreads();
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    if (b < nb) {
      float tot = 0.0f;
#pragma unroll
      for (int w = 0; w < kNormThreads / 64; ++w) tot += red[b * (kNormThreads / 64) + w];
      const float r = 1.0f / sqrtf(tot / (float)d + eps);
#pragma unroll
      for (int i = 0; i < PIECES; ++i) {
        const int q = threadIdx.x + i * kNormThreads;
        if (q < n4) {
          const f16x2 lo = {(f16)(v[b][i].x * r), (f16)(v[b][i].y * r)};
          const f16x2 hi = {(f16)(v[b][i].z * r), (f16)(v[b][i].w * r)};
          store(t0 + b, q, __builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi));
        }
      }
    }
  }
  __syncthreads();
}

// Device workspace of one layer call: the work list, the pair permutation
// and its inverse, the routing outputs, the SwiGLU activations h of every
// pair and the per-pair expert outputs (prefill and matrix-core decode).
struct Workspace {
  WorkList* wl = nullptr;
  int32_t* perm = nullptr;   // [T*K] pairs sorted by work group (stable)
  int32_t* pos = nullptr;    // [T*K] position of each pair in that order, -1 if skipped
  int32_t* idx = nullptr;    // [T*K]
  float* w = nullptr;        // [T*K]
  int8_t* prec = nullptr;    // [T*K]
  f16* h = nullptr;          // [T*K, d_ff]
  float* eperm = nullptr;    // [T*K, d_model] in group order
};

// Routing outputs of one call; optional user copies may be null.
struct RouteOut {
  int32_t* idx;        // [T*K] internal
  float* w;            // [T*K] internal
  int8_t* prec;        // [T*K] internal
  int32_t* user_idx;   // optional
  float* user_w;       // optional
  int8_t* user_prec;   // optional
};

struct RouteParams {
  const f16* x;         // [T, d]
  // decode router only: with h_res set, the router forms x itself as
  // fp16(rmsnorm(h_res)) (eps), writes it to x_out and routes it
  const float* h_res = nullptr;   // [T, d]
  f16* x_out = nullptr;           // [T, d]
  float eps = 0.0f;
  const f16* wg;        // [E, d]
  const ExpertEntry* table;
  int32_t T, d, E, K;
  float t1, t2;
};

// Stacking Computer (predict.hip): the gates of the next p layers stacked
// as wstack [p*E, d], applied to the current gating input x [T, d].
constexpr int kMaxPredLayers = 8;

struct PredictParams {
  const f16* x;                 // [T, d]
  const f16* wstack;            // [p*E, d]
  const uint64_t* cached;       // [p] expert-cache bitmask per predicted layer
  float* logits;                // [T, p*E] workspace
  unsigned* counter;            // blocks finished (zero between launches)
  int32_t* idx;                 // [T, p, K]
  float* w;                     // [T, p, K] or null
  int32_t* first_miss;          // [1]
  uint64_t* preload;            // [1]
  int32_t T, d, E, K, p;
};

// Static scratch of the allocation-free decode step (noalloc.hip): its size,
// and its device address on `device` (looked up on the first call, which
// must find `device` current; later calls return the kept address).
size_t scratch_bytes();
hipError_t scratch_setup(int device, void** out);

// ---- launchers (defined in the .hip files) -------------------------------
hipError_t launch_quantize(const f16* w, int64_t rows, int64_t cols, int bits,
                           uint8_t* codes, f16* scales, hipStream_t s);
hipError_t launch_set_entry(ExpertEntry* table, int e, ExpertEntry v,
                            hipStream_t s);
hipError_t launch_route_decode(const RouteParams& p, RouteOut o, WorkList* wl,
                               int32_t* perm, int32_t* pos, hipStream_t s);
// Whether the decode router can form the RMSNorm of h_res itself for T
// tokens of d_model d (its activations then fit in its LDS).
bool route_decode_fuses_norm(int T, int d);
hipError_t launch_route_prefill(const RouteParams& p, RouteOut o, WorkList* wl,
                                int32_t* perm, int32_t* pos, hipStream_t s);
hipError_t launch_decode_up(const ExpertEntry* table, const WorkList* wl,
                            const int32_t* perm, const f16* x, f16* h,
                            int T, int d, int f, int K, int max_groups,
                            hipStream_t s);
hipError_t launch_decode_down(const ExpertEntry* table, const WorkList* wl,
                              const int32_t* perm, const float* gate_w,
                              const f16* h, float* y, float* h_res, int T, int d,
                              int f, int K, hipStream_t s);
hipError_t launch_decode_up_mfma(const ExpertEntry* table, const WorkList* wl,
                                 const int32_t* perm, const f16* x, f16* h, int d,
                                 int f, int K, int max_groups, hipStream_t s);
hipError_t launch_decode_down_mfma(const ExpertEntry* table, const WorkList* wl,
                                   const int32_t* perm, const f16* h, float* e_perm,
                                   int d, int f, int max_groups, hipStream_t s);
hipError_t launch_predict(const PredictParams& q, hipStream_t s);
hipError_t launch_rmsnorm(const float* h_res, f16* x_next, int T, int d,
                          float eps, hipStream_t s);
hipError_t launch_prefill_up(const ExpertEntry* table, const WorkList* wl,
                             const int32_t* perm, const f16* x, f16* h_perm,
                             int T, int d, int f, int K, int max_groups,
                             hipStream_t s);
hipError_t launch_prefill_down(const ExpertEntry* table, const WorkList* wl,
                               const f16* h_perm, float* e_perm, int T, int d,
                               int f, int K, int max_groups, hipStream_t s);
hipError_t launch_combine_prefill(const float* e_perm, const int32_t* pos,
                                  const float* w, const int8_t* prec, int T,
                                  int d, int K, float* y, float* h_res,
                                  f16* x_next, float eps, hipStream_t s);

}  // namespace moe
