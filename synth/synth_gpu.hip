// Device-side twin of synth/gen.py: element i of the stream named by `key`
// is table[(mix64(key + (c + 1) * GOLDEN) >> 16 j) & 0xFFFF] with c = i / 4,
// j = i % 4, and mix64 the SplitMix64 output function (Steele, Lea and
// Flood, OOPSLA 2014).  The 65536-entry fp16 quantile table is computed on
// the host and uploaded, so both sides only index the same values.
// Input generation only: no part of the MoE method lives here.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

__device__ inline uint64_t mix64(uint64_t z) {
  z ^= z >> 30;
  z *= 0xBF58476D1CE4E5B9ull;
  z ^= z >> 27;
  z *= 0x94D049BB133111EBull;
  z ^= z >> 31;
  return z;
}

// one 64-bit word (four elements) per thread
__global__ __launch_bounds__(256) void normal_fp16_kernel(
    uint64_t key, const uint16_t* __restrict__ table, uint16_t* __restrict__ out,
    int64_t n, int64_t start) {
  const int64_t first_word = start >> 2;
  const int64_t w = first_word + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t e0 = w * 4;  // stream index of lane 0 of this word
  if (e0 >= start + n) return;
  const uint64_t r = mix64(key + (uint64_t)(w + 1) * 0x9E3779B97F4A7C15ull);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t e = e0 + j;
    if (e >= start && e < start + n)
      out[e - start] = table[(r >> (16 * j)) & 0xFFFFu];
  }
}

}  // namespace

extern "C" int synth_normal_fp16(uint64_t key, const void* table, void* out,
                                 int64_t n, int64_t start, void* stream) {
  if (n <= 0) return 0;
  if (!table || !out || start < 0) return 1;
  const int64_t words = ((start + n + 3) >> 2) - (start >> 2);
  const int64_t blocks = (words + 255) / 256;
  if (blocks > 0x7fffffffLL) return 1;
  normal_fp16_kernel<<<dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream>>>(
      key, (const uint16_t*)table, (uint16_t*)out, n, start);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}
