// Group-wise symmetric quantiser producing the quantised expert copies
// (Section 2.2 and Section 4.1 "Configurations": int4 replaces fp16, int2
// replaces int8; the int8 copy itself is the high precision of an int8
// model).  Format: group of 32 consecutive weights along a row,
// s = fp16_rne(max|w| / qmax), q = clamp(rne(w / s), -2^(b-1), qmax),
// stored offset-binary and packed little-endian within each byte.
//
// Exactness: w and s are fp16, so w / s is never within 2^-13 of a
// half-integer unless it is one, while one correctly rounded fp32 division
// of a quotient below 128 errs by at most 2^-17: it makes the same rounding
// decision as exact arithmetic.  max|w| / 7 and max|w| / 127 have binary
// expansions of period 3 and 7 (or are exact), so rounding them to fp32 and
// then to fp16 cannot land on an fp16 midpoint (that needs a run of 12 equal
// bits): the double rounding equals a single rounding.  Divisions therefore
// use __fdiv_rn, never a reciprocal.
#include "moe_internal.h"

namespace moe {

// One thread per group of 32 weights: 64 contiguous input bytes, 32 (int8),
// 16 (int4) or 8 (int2) output bytes and one fp16 scale.
template <int BITS>
__global__ __launch_bounds__(256) void quantize_kernel(
    const f16* __restrict__ w, int64_t n_groups, uint8_t* __restrict__ codes,
    f16* __restrict__ scales) {
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= n_groups) return;
  constexpr int kQmax = (1 << (BITS - 1)) - 1;
  constexpr int kQmin = -(1 << (BITS - 1));
  constexpr int kOff = 1 << (BITS - 1);

  const u32x4* src = reinterpret_cast<const u32x4*>(w + g * kGroup);
  f16 v[kGroup];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    u32x4 p = src[i];
    f16x8 h = __builtin_bit_cast(f16x8, p);
#pragma unroll
    for (int j = 0; j < 8; ++j) v[i * 8 + j] = h[j];
  }
  float m = 0.0f;
#pragma unroll
  for (int j = 0; j < kGroup; ++j) m = fmaxf(m, fabsf((float)v[j]));
  const f16 s16 = (f16)__fdiv_rn(m, (float)kQmax);  // RNE to fp16
  const float s = (float)s16;

  uint32_t out[BITS];  // 32 codes * BITS bits = BITS words
#pragma unroll
  for (int i = 0; i < BITS; ++i) out[i] = 0u;
#pragma unroll
  for (int j = 0; j < kGroup; ++j) {
    int q = 0;
    if (s > 0.0f) {
      float r = rintf(__fdiv_rn((float)v[j], s));  // ties to even
      r = fminf(fmaxf(r, (float)kQmin), (float)kQmax);
      q = (int)r;
    }
    const uint32_t u = (uint32_t)(q + kOff);
    const int bit = j * BITS;
    out[bit >> 5] |= u << (bit & 31);
  }
  if (BITS == 8) {
    reinterpret_cast<u32x4*>(codes)[2 * g] = u32x4{out[0], out[1], out[2], out[3]};
    reinterpret_cast<u32x4*>(codes)[2 * g + 1] = u32x4{out[4], out[5], out[6], out[7]};
  } else if (BITS == 4) {
    reinterpret_cast<u32x4*>(codes)[g] = u32x4{out[0], out[1], out[2], out[3]};
  } else {
    reinterpret_cast<uint2*>(codes)[g] = make_uint2(out[0], out[1]);
  }
  scales[g] = s16;
}

hipError_t launch_quantize(const f16* w, int64_t rows, int64_t cols, int bits,
                           uint8_t* codes, f16* scales, hipStream_t s) {
  const int64_t n_groups = rows * (cols / kGroup);
  if (n_groups == 0) return hipSuccess;
  const int threads = 256;
  const int64_t blocks = (n_groups + threads - 1) / threads;
  if (bits == 8)
    quantize_kernel<8><<<dim3((unsigned)blocks), dim3(threads), 0, s>>>(
        w, n_groups, codes, scales);
  else if (bits == 4)
    quantize_kernel<4><<<dim3((unsigned)blocks), dim3(threads), 0, s>>>(
        w, n_groups, codes, scales);
  else
    quantize_kernel<2><<<dim3((unsigned)blocks), dim3(threads), 0, s>>>(
        w, n_groups, codes, scales);
  return hipGetLastError();
}

// Stream-ordered update of one expert table entry (value passed by kernel
// argument, so no host buffer has to outlive the call).
__global__ void set_entry_kernel(ExpertEntry* table, int e, ExpertEntry v) {
  if (threadIdx.x == 0) table[e] = v;
}

hipError_t launch_set_entry(ExpertEntry* table, int e, ExpertEntry v,
                            hipStream_t s) {
  set_entry_kernel<<<1, 64, 0, s>>>(table, e, v);
  return hipGetLastError();
}

}  // namespace moe
