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
