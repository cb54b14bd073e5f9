// Decode-path expert kernels: fused dequantise-GEMV for the SwiGLU experts
// of Eq. 1 at fp16, int8 (the high copy of an int8 model), int4 or int2,
// with the weighted combine fused into the down-projection.
//
//   up:    h[p, r] = silu(W1[r,:] . x_t) * (W3[r,:] . x_t)        (fp16 out)
//   down:  y[t, r] = sum over the (token, slot) pairs p of token t of
//                    w[p] * (W2[r,:] . h[p])                      (Eq. 1)
//
// Block shape: a tile of output rows (UpRows / DownRows) is shared by the 4
// waves of a block; the waves split
// the reduction dimension (wave w takes lane-chunks w, w+4, ...), so one
// activation load of a lane serves every row of the tile (x2 matrices for
// the up-projection).
// Per lane and chunk a wave reads one piece per row:
//   fp16  16 bytes =  8 weights   (chunk =  512 columns)
//   int8  16 bytes = 16 weights   (chunk = 1024 columns, half a group)
//   int4   8 bytes = 16 weights   (chunk = 1024 columns, half a group)
//   int2   4 bytes = 16 weights   (chunk = 1024 columns, half a group)
// so each wave-wide load covers 1 KiB, 512 B or 256 B of one row.  Codes are
// turned into fp16 pairs with the 0x6400|u == 1024+u trick, the matching
// activation pairs are permuted in registers once per token, and
// v_dot2_f32_f16 accumulates q.x in fp32 (exact products); a lane's half
// group is then scaled once by its fp16 scale.
//
// Up-projection blocks each take one (expert, precision) work group and a
// row tile, so every selected expert copy is streamed from HBM once per step
// whatever the number of tokens routed to it.  Down-projection blocks each
// take a row tile of d_model and loop over all work groups, accumulating
// w[p] * e into the token's output row in LDS in work-list order, so the
// combine needs no extra pass and the sum order is fixed (deterministic).
#include "moe_internal.h"

namespace moe {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

// Output rows per block for a token tile of up to NTMAX tokens.  Small
// tiles measured fastest at one or two tokens: more blocks in flight hide
// the start-up latency of each block (4 rows: 112 us per Mixtral-shaped
// T=1 step against 128 us with 8 rows and 132 us with 16; 2-row up tiles
// with 4-row down tiles: 109 us).
template <int NTMAX> struct UpRows { static constexpr int value = NTMAX <= 2 ? 2 : 4; };
template <int NTMAX> struct DownRows { static constexpr int value = NTMAX <= 2 ? 4 : 8; };

// Scalar-argument casts on purpose: clang's __builtin_bit_cast applied
// directly to a vector component expression (v.y) reads component 0.
__device__ inline f16x2 as_h2(uint32_t v) { return __builtin_bit_cast(f16x2, v); }

__device__ inline float dot2(uint32_t a, uint32_t b, float acc) {
  return __builtin_amdgcn_fdot2(as_h2(a), as_h2(b), acc, false);
}

__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// low half of a | low half of b  /  high half of a | high half of b
__device__ inline uint32_t lo_lo(uint32_t a, uint32_t b) {
  return __builtin_amdgcn_perm(b, a, 0x05040100u);
}
__device__ inline uint32_t hi_hi(uint32_t a, uint32_t b) {
  return __builtin_amdgcn_perm(b, a, 0x07060302u);
}

// Pointers taken from the expert table are generic; reading through them
// would emit flat loads (which also hold the LDS counter).  They always
// point to device memory, so they are cast to the global address space.
template <class T>
__device__ inline const __attribute__((address_space(1))) T* gmem(const T* p) {
  return (const __attribute__((address_space(1))) T*)p;
}

// Elements per lane per chunk for each weight format.
template <int BITS> struct Fmt;
template <> struct Fmt<16> { static constexpr int kEpl = 8; };
template <> struct Fmt<8> { static constexpr int kEpl = 16; };
template <> struct Fmt<4> { static constexpr int kEpl = 16; };
template <> struct Fmt<2> { static constexpr int kEpl = 16; };

// Activations of one lane for one chunk, as the dword pairs the weight
// pieces are dotted with.  fp16: natural order (4 dwords).  int8: per 4
// elements (x0,x2)(x1,x3) (8 dwords).  int4: per 8 elements
// (x0,x4)(x1,x5)(x2,x6)(x3,x7) (8 dwords).  int2: per 16 elements
// (x0,x8)(x1,x9)...(x7,x15) (8 dwords).
template <int BITS>
__device__ inline void load_act(const f16* p, uint32_t (&a)[Fmt<BITS>::kEpl / 2]) {
  if constexpr (BITS == 16) {
    const u32x4 v = *reinterpret_cast<const u32x4*>(p);
    a[0] = v.x; a[1] = v.y; a[2] = v.z; a[3] = v.w;
  } else {
    const u32x4 v0 = reinterpret_cast<const u32x4*>(p)[0];
    const u32x4 v1 = reinterpret_cast<const u32x4*>(p)[1];
    if constexpr (BITS == 8) {  // blocks of 4: dwords (x0x1)(x2x3)
      a[0] = lo_lo(v0.x, v0.y); a[1] = hi_hi(v0.x, v0.y);
      a[2] = lo_lo(v0.z, v0.w); a[3] = hi_hi(v0.z, v0.w);
      a[4] = lo_lo(v1.x, v1.y); a[5] = hi_hi(v1.x, v1.y);
      a[6] = lo_lo(v1.z, v1.w); a[7] = hi_hi(v1.z, v1.w);
    } else if constexpr (BITS == 4) {  // blocks of 8: dwords (x0x1)(x2x3)(x4x5)(x6x7)
      a[0] = lo_lo(v0.x, v0.z); a[1] = hi_hi(v0.x, v0.z);
      a[2] = lo_lo(v0.y, v0.w); a[3] = hi_hi(v0.y, v0.w);
      a[4] = lo_lo(v1.x, v1.z); a[5] = hi_hi(v1.x, v1.z);
      a[6] = lo_lo(v1.y, v1.w); a[7] = hi_hi(v1.y, v1.w);
    } else {  // one block of 16: dwords d0..d7 = (x0x1)..(x14x15)
      a[0] = lo_lo(v0.x, v1.x); a[1] = hi_hi(v0.x, v1.x);
      a[2] = lo_lo(v0.y, v1.y); a[3] = hi_hi(v0.y, v1.y);
      a[4] = lo_lo(v0.z, v1.z); a[5] = hi_hi(v0.z, v1.z);
      a[6] = lo_lo(v0.w, v1.w); a[7] = hi_hi(v0.w, v1.w);
    }
  }
}

// One weight piece of one row for one chunk: loaded, then multiplied with
// the activation pairs of load_act, and its group scale.  Weights are read
// exactly once per step, so they are loaded nontemporally (streaming hint):
// on MI355X that lifts a pure read stream from ~6.2 to ~6.9 TB/s.
//
// Codes become fp16 without shifting each one into place: a code u whose
// lowest bit sits at bit p of a 16-bit half, or-ed with the exponent of
// 2^(10-p), is the fp16 number 2^(10-p) + u (one and-or per pair of codes
// 16 bits apart).  The products then carry the offset o = 2^(10-p) + z of
// each code (z: the format's zero point, 2^(bits-1)), which is removed once
// per chunk and token on the activation side:
//   sum_j (u_j - z) x_j = sum_j (o_j + u_j - z) x_j - sum_j o_j x_j,
// where the second sum (bias()) depends on the token only and serves every
// row of the tile.  All products are exact in fp32 (11 x 11 bits); the
// fp32 sums of the offset products lose about 2^-24 of their magnitude
// (at most ~1000x the activations) per addition.
template <int BITS> struct Piece;

__device__ inline uint32_t and_or(uint32_t w, uint32_t mask, uint32_t expo) {
  return (w & mask) | expo;
}

template <> struct Piece<16> {
  u32x4 v;
  __device__ inline void load(const ExpertEntry& ex, int m, int64_t row, int64_t ld, int64_t col) {
    v = __builtin_nontemporal_load(gmem(reinterpret_cast<const u32x4*>(ex.w[m] + row * ld + col)));
  }
  static __device__ inline float bias(const uint32_t (&)[4]) { return 0.0f; }
  __device__ inline float dot(const uint32_t (&a)[4], float, float acc) const {
    acc = dot2(v.x, a[0], acc);
    acc = dot2(v.y, a[1], acc);
    acc = dot2(v.z, a[2], acc);
    return dot2(v.w, a[3], acc);
  }
};

template <> struct Piece<8> {
  u32x4 v;
  f16 s;
  __device__ inline void load(const ExpertEntry& ex, int m, int64_t row, int64_t ld, int64_t col) {
    v = __builtin_nontemporal_load(gmem(reinterpret_cast<const u32x4*>(ex.hq[m] + row * ld + col)));
    s = __builtin_nontemporal_load(gmem(ex.hs[m] + row * (ld / kGroup) + col / kGroup));
  }
  // every pair carries 1024 + 128 (p = 0 after the byte shift, z = 128)
  static __device__ inline float bias(const uint32_t (&a)[8]) {
    float b = 0.0f;
#pragma unroll
    for (int k = 0; k < 8; ++k) b = dot2(a[k], 0x64806480u, b);  // 1152
    return b;
  }
  // word holding e0..e3 (e_j in byte j) -> pairs (e0, e2), (e1, e3)
  static __device__ inline float dot_word(uint32_t w, const uint32_t* a, float g) {
    g = dot2(and_or(w, 0x00FF00FFu, 0x64006400u), a[0], g);
    return dot2(and_or(w >> 8, 0x00FF00FFu, 0x64006400u), a[1], g);
  }
  __device__ inline float dot(const uint32_t (&a)[8], float bias, float acc) const {
    float g = dot_word(v.x, a, 0.0f);
    g = dot_word(v.y, a + 2, g);
    g = dot_word(v.z, a + 4, g);
    g = dot_word(v.w, a + 6, g);
    return fmaf((float)s, g - bias, acc);
  }
};

template <> struct Piece<4> {
  u32x2 v;
  f16 s;
  __device__ inline void load(const ExpertEntry& ex, int m, int64_t row, int64_t ld, int64_t col) {
    v = __builtin_nontemporal_load(gmem(reinterpret_cast<const u32x2*>(ex.q[m] + row * (ld / 2) + col / 2)));
    s = __builtin_nontemporal_load(gmem(ex.s[m] + row * (ld / kGroup) + col / kGroup));
  }
  // pair k of a word: codes at bits 4k, 16 + 4k; k = 0, 2 sit at p = 0
  // (offset 1024 + 8), k = 1, 3 at p = 4 (64 + 8), k = 2, 3 after a shift by 8
  static __device__ inline float bias(const uint32_t (&a)[8]) {
    float b = 0.0f;
#pragma unroll
    for (int k = 0; k < 8; ++k) b = dot2(a[k], (k & 1) ? 0x54805480u : 0x64086408u, b);  // 72 : 1032
    return b;
  }
  // word holding e0..e7 (e_j at bits 4j) -> pairs (e_k, e_{k+4})
  static __device__ inline float dot_word(uint32_t w, const uint32_t* a, float g) {
    const uint32_t w8 = w >> 8;
    g = dot2(and_or(w, 0x000F000Fu, 0x64006400u), a[0], g);
    g = dot2(and_or(w, 0x00F000F0u, 0x54005400u), a[1], g);
    g = dot2(and_or(w8, 0x000F000Fu, 0x64006400u), a[2], g);
    return dot2(and_or(w8, 0x00F000F0u, 0x54005400u), a[3], g);
  }
  __device__ inline float dot(const uint32_t (&a)[8], float bias, float acc) const {
    float g = dot_word(v.x, a, 0.0f);
    g = dot_word(v.y, a + 4, g);
    return fmaf((float)s, g - bias, acc);
  }
};

template <> struct Piece<2> {
  uint32_t v;
  f16 s;
  __device__ inline void load(const ExpertEntry& ex, int m, int64_t row, int64_t ld, int64_t col) {
    v = __builtin_nontemporal_load(gmem(reinterpret_cast<const uint32_t*>(ex.q[m] + row * (ld / 4) + col / 4)));
    s = __builtin_nontemporal_load(gmem(ex.s[m] + row * (ld / kGroup) + col / kGroup));
  }
  // pair k: codes at bits 2k, 16 + 2k; k = 0..4 in place (p = 2k), k = 5..7
  // after a shift by 10 (p = 2k - 10); offsets 2^(10-p) + 2
  static constexpr uint32_t kMask[8] = {0x00030003u, 0x000C000Cu, 0x00300030u, 0x00C000C0u,
                                        0x03000300u, 0x00030003u, 0x000C000Cu, 0x00300030u};
  static constexpr uint32_t kExpo[8] = {0x64006400u, 0x5C005C00u, 0x54005400u, 0x4C004C00u,
                                        0x44004400u, 0x64006400u, 0x5C005C00u, 0x54005400u};
  static constexpr uint32_t kOff[8] = {0x64026402u, 0x5C085C08u, 0x54205420u, 0x4C804C80u,  // 1026 258 66 18
                                       0x46004600u, 0x64026402u, 0x5C085C08u, 0x54205420u}; // 6 1026 258 66
  static __device__ inline float bias(const uint32_t (&a)[8]) {
    float b = 0.0f;
#pragma unroll
    for (int k = 0; k < 8; ++k) b = dot2(a[k], kOff[k], b);
    return b;
  }
  // word holding e0..e15 (e_j at bits 2j) -> pairs (e_k, e_{k+8})
  __device__ inline float dot(const uint32_t (&a)[8], float bias, float acc) const {
    const uint32_t w10 = v >> 10;
    float g = 0.0f;
#pragma unroll
    for (int k = 0; k < 8; ++k) g = dot2(and_or(k < 5 ? v : w10, kMask[k], kExpo[k]), a[k], g);
    return fmaf((float)s, g - bias, acc);
  }
};

// Partial dot products of this wave's chunks for ROWS rows of NM matrices
// (matrix ids mats) against NT activation rows act_rows[t] (length ld).
template <int BITS, int NT, int NM, int ROWS>
__device__ inline void tile_dots(const ExpertEntry& ex, const int (&mats)[NM],
                                 int64_t row0, int64_t ld,
                                 const f16* const (&act_rows)[NT],
                                 float (&acc)[NM][ROWS][NT]) {
  constexpr int kEpl = Fmt<BITS>::kEpl;
  constexpr int kChunk = 64 * kEpl;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n_chunks = (int)((ld + kChunk - 1) / kChunk);
  for (int c = wave; c < n_chunks; c += kWaves) {
    const int64_t col = (int64_t)c * kChunk + lane * kEpl;
    if (col >= ld) continue;  // ragged last chunk (ld is a multiple of 64)
    uint32_t a[NT][kEpl / 2];
    float bb[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) load_act<BITS>(act_rows[t] + col, a[t]);
#pragma unroll
    for (int t = 0; t < NT; ++t) bb[t] = Piece<BITS>::bias(a[t]);
#pragma unroll
    for (int m = 0; m < NM; ++m) {
      Piece<BITS> pc[ROWS];
#pragma unroll
      for (int i = 0; i < ROWS; ++i) pc[i].load(ex, mats[m], row0 + i, ld, col);
#pragma unroll
      for (int i = 0; i < ROWS; ++i)
#pragma unroll
        for (int t = 0; t < NT; ++t) acc[m][i][t] = pc[i].dot(a[t], bb[t], acc[m][i][t]);
    }
  }
}

// tile_dots with this wave's chunks in a ring of two register slots: the
// next chunk's loads are in flight while the current one is multiplied.
// Every load is unconditional (lanes past the row end load column 0 and
// skip the products; slots past the wave's last chunk reload it), so the
// compiler's wait counts stay exact.
template <int BITS, int NT, int NM, int ROWS>
__device__ inline void tile_dots_ring(const ExpertEntry& ex, const int (&mats)[NM],
                                      int64_t row0, int64_t ld,
                                      const f16* const (&act_rows)[NT],
                                      float (&acc)[NM][ROWS][NT]) {
  constexpr int kEpl = Fmt<BITS>::kEpl;
  constexpr int kChunk = 64 * kEpl;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int n_chunks = (int)((ld + kChunk - 1) / kChunk);
  const int nw = (n_chunks - wave + kWaves - 1) / kWaves;  // this wave's chunks
  if (nw <= 0) return;
  uint32_t a[2][NT][kEpl / 2];
  Piece<BITS> pc[2][NM][ROWS];
  auto col_of = [&](int i) {
    return (int64_t)(wave + min(i, nw - 1) * kWaves) * kChunk + lane * kEpl;
  };
  auto load = [&](int sl, int i) {
    int64_t col = col_of(i);
    col = col < ld ? col : 0;
#pragma unroll
    for (int t = 0; t < NT; ++t) load_act<BITS>(act_rows[t] + col, a[sl][t]);
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int r = 0; r < ROWS; ++r) pc[sl][m][r].load(ex, mats[m], row0 + r, ld, col);
  };
  auto dots = [&](int sl, int i) {
    if (col_of(i) < ld) {
      float bb[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t) bb[t] = Piece<BITS>::bias(a[sl][t]);
#pragma unroll
      for (int m = 0; m < NM; ++m)
#pragma unroll
        for (int r = 0; r < ROWS; ++r)
#pragma unroll
          for (int t = 0; t < NT; ++t) acc[m][r][t] = pc[sl][m][r].dot(a[sl][t], bb[t], acc[m][r][t]);
    }
  };
  load(0, 0);
  load(1, 1);
  int i = 0;
  for (; i + 2 <= nw; i += 2) {
    dots(0, i);
    load(0, i + 2);
    dots(1, i + 1);
    load(1, i + 3);
  }
  if (i < nw) dots(0, i);
}

// Sum the per-lane partials over the lanes of each wave and then over the
// waves; afterwards red[kWaves*V + v] (v = (m*ROWS + i)*NT + t) holds the
// full value.
template <int NM, int NT, int ROWS>
__device__ inline void block_reduce(float (&acc)[NM][ROWS][NT], float* red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  constexpr int V = NM * ROWS * NT;
#pragma unroll
  for (int m = 0; m < NM; ++m)
#pragma unroll
    for (int i = 0; i < ROWS; ++i)
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const float s = wave_sum_dpp(acc[m][i][t]);
        if (lane == 0) red[wave * V + (m * ROWS + i) * NT + t] = s;
      }
  __syncthreads();
  for (int v = threadIdx.x; v < V; v += kThreads) {
    float s = red[v];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) s += red[w * V + v];
    red[kWaves * V + v] = s;
  }
  __syncthreads();
}

// ---------------------------------------------------------------- up-proj
template <int BITS, int NT, int ROWS>
__device__ void up_tile(const ExpertEntry& ex, const int32_t* pairs, int n,
                        const f16* x, f16* h, int d, int f, int K, int64_t row0,
                        float* red) {
  const f16* rows[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) rows[t] = x + (int64_t)(pairs[t < n ? t : 0] / K) * d;
  float acc[2][ROWS][NT];
#pragma unroll
  for (int m = 0; m < 2; ++m)
#pragma unroll
    for (int i = 0; i < ROWS; ++i)
#pragma unroll
      for (int t = 0; t < NT; ++t) acc[m][i][t] = 0.0f;
  const int mats[2] = {0, 1};
  tile_dots<BITS, NT, 2, ROWS>(ex, mats, row0, d, rows, acc);
  block_reduce<2, NT, ROWS>(acc, red);
  const float* fin = red + kWaves * 2 * ROWS * NT;
  for (int v = threadIdx.x; v < ROWS * NT; v += kThreads) {
    const int i = v / NT, t = v - (v / NT) * NT;
    if (t < n) {
      const float a = fin[(0 * ROWS + i) * NT + t];
      const float b = fin[(1 * ROWS + i) * NT + t];
      h[(int64_t)pairs[t] * f + row0 + i] = (f16)(a / (1.0f + expf(-a)) * b);
    }
  }
  __syncthreads();
}

template <int BITS, int NTMAX>
__device__ void up_group(const ExpertEntry& ex, const int32_t* pairs, int count,
                         const f16* x, f16* h, int d, int f, int K, int64_t row0,
                         float* red) {
  constexpr int R = UpRows<NTMAX>::value;
  for (int j0 = 0; j0 < count; j0 += NTMAX) {
    const int n = min(NTMAX, count - j0);
    if (NTMAX == 1 || n <= 1) up_tile<BITS, 1, R>(ex, pairs + j0, n, x, h, d, f, K, row0, red);
    else if (NTMAX == 2 || n <= 2) up_tile<BITS, (NTMAX < 2 ? NTMAX : 2), R>(ex, pairs + j0, n, x, h, d, f, K, row0, red);
    else if (NTMAX == 4 || n <= 4) up_tile<BITS, (NTMAX < 4 ? NTMAX : 4), R>(ex, pairs + j0, n, x, h, d, f, K, row0, red);
    else up_tile<BITS, NTMAX, R>(ex, pairs + j0, n, x, h, d, f, K, row0, red);
  }
}

template <int NTMAX>
__global__ __launch_bounds__(kThreads) void decode_up_kernel(
    const ExpertEntry* __restrict__ table, const WorkList* __restrict__ wl,
    const int32_t* __restrict__ perm, const f16* __restrict__ x,
    f16* __restrict__ h, int d, int f, int K) {
  __shared__ float red[(kWaves + 1) * 2 * UpRows<NTMAX>::value * NTMAX];
  if ((int)blockIdx.y >= wl->n_groups) return;
  const Group g = wl->groups[blockIdx.y];
  const ExpertEntry ex = table[g.expert];
  const int64_t row0 = (int64_t)blockIdx.x * UpRows<NTMAX>::value;
  const int32_t* pairs = perm + g.offset;
  if (g.bits == 16) up_group<16, NTMAX>(ex, pairs, g.count, x, h, d, f, K, row0, red);
  else if (g.bits == 8) up_group<8, NTMAX>(ex, pairs, g.count, x, h, d, f, K, row0, red);
  else if (g.bits == 4) up_group<4, NTMAX>(ex, pairs, g.count, x, h, d, f, K, row0, red);
  else up_group<2, NTMAX>(ex, pairs, g.count, x, h, d, f, K, row0, red);
}

// ------------------------------------------------- down-proj + combine
template <int BITS, int NT, int ROWS, bool RING>
__device__ void down_tile(const ExpertEntry& ex, const int32_t* pairs, int n,
                          const f16* h, const float* gate_w, int f, int K,
                          int64_t row0, float* red, float* yacc) {
  const f16* rows[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) rows[t] = h + (int64_t)pairs[t < n ? t : 0] * f;
  float acc[1][ROWS][NT];
#pragma unroll
  for (int i = 0; i < ROWS; ++i)
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[0][i][t] = 0.0f;
  const int mats[1] = {2};
  // one-token steps, fp16 copies: the two-slot ring fits the 4 waves per
  // SIMD that keep every block of the step resident; the two-token kernel
  // would lose a wave, and code groups measured slower with it (int8 W2
  // 24.9 -> 26.3 us per int8-model step)
  if constexpr (RING && BITS == 16) tile_dots_ring<BITS, NT, 1, ROWS>(ex, mats, row0, f, rows, acc);
  else tile_dots<BITS, NT, 1, ROWS>(ex, mats, row0, f, rows, acc);
  block_reduce<1, NT, ROWS>(acc, red);
  const float* fin = red + kWaves * ROWS * NT;
  for (int v = threadIdx.x; v < ROWS * NT; v += kThreads) {
    const int i = v / NT, t = v - (v / NT) * NT;
    if (t < n) {
      const int p = pairs[t];
      // a token occurs once per work group: no two threads share a cell
      yacc[(p / K) * ROWS + i] += gate_w[p] * fin[i * NT + t];
    }
  }
  __syncthreads();
}

template <int BITS, int NTMAX>
__device__ void down_group(const ExpertEntry& ex, const int32_t* pairs, int count,
                           const f16* h, const float* gate_w, int f, int K,
                           int64_t row0, float* red, float* yacc) {
  constexpr int R = DownRows<NTMAX>::value;
  for (int j0 = 0; j0 < count; j0 += NTMAX) {
    const int n = min(NTMAX, count - j0);
    if (NTMAX == 1 || n <= 1) down_tile<BITS, 1, R, NTMAX == 1>(ex, pairs + j0, n, h, gate_w, f, K, row0, red, yacc);
    else if (NTMAX == 2 || n <= 2) down_tile<BITS, (NTMAX < 2 ? NTMAX : 2), R, false>(ex, pairs + j0, n, h, gate_w, f, K, row0, red, yacc);
    else if (NTMAX == 4 || n <= 4) down_tile<BITS, (NTMAX < 4 ? NTMAX : 4), R, false>(ex, pairs + j0, n, h, gate_w, f, K, row0, red, yacc);
    else down_tile<BITS, NTMAX, R, false>(ex, pairs + j0, n, h, gate_w, f, K, row0, red, yacc);
  }
}

// y[t, rows] (or h_res[t, rows] += ...) for one row tile, all work groups.
template <int NTMAX>
__global__ __launch_bounds__(kThreads) void decode_down_kernel(
    const ExpertEntry* __restrict__ table, const WorkList* __restrict__ wl,
    const int32_t* __restrict__ perm, const float* __restrict__ gate_w,
    const f16* __restrict__ h, float* __restrict__ y, float* __restrict__ h_res,
    int T, int d, int f, int K) {
  constexpr int R = DownRows<NTMAX>::value;
  __shared__ float red[(kWaves + 1) * R * NTMAX];
  __shared__ float yacc[kDecodeMaxTokens * R];
  const int64_t row0 = (int64_t)blockIdx.x * R;
  for (int v = threadIdx.x; v < T * R; v += kThreads) yacc[v] = 0.0f;
  __syncthreads();
  const int n_groups = wl->n_groups;
  for (int gi = 0; gi < n_groups; ++gi) {
    const Group g = wl->groups[gi];
    const ExpertEntry ex = table[g.expert];
    const int32_t* pairs = perm + g.offset;
    if (g.bits == 16) down_group<16, NTMAX>(ex, pairs, g.count, h, gate_w, f, K, row0, red, yacc);
    else if (g.bits == 8) down_group<8, NTMAX>(ex, pairs, g.count, h, gate_w, f, K, row0, red, yacc);
    else if (g.bits == 4) down_group<4, NTMAX>(ex, pairs, g.count, h, gate_w, f, K, row0, red, yacc);
    else down_group<2, NTMAX>(ex, pairs, g.count, h, gate_w, f, K, row0, red, yacc);
  }
  for (int v = threadIdx.x; v < T * R; v += kThreads) {
    const int t = v / R, i = v - t * R;
    const int64_t o = (int64_t)t * d + row0 + i;
    if (h_res) h_res[o] += yacc[v];
    else y[o] = yacc[v];
  }
}

// ------------------------------------------------------ residual RMSNorm
// One block of 1024 threads per token (rmsnorm_rows in moe_internal.h).
__global__ __launch_bounds__(kNormThreads) void rmsnorm_kernel(
    const float* __restrict__ h_res, f16* __restrict__ x_next, int d, float eps) {
  __shared__ float red[kNormThreads / 64];
  rmsnorm_rows<1, kNormPieces>(h_res, d, eps, blockIdx.x, 1, red,
                               [&](int t, int q, uint32_t lo, uint32_t hi) {
                                 *reinterpret_cast<u32x2*>(x_next + (int64_t)t * d + 4 * q) =
                                     u32x2{lo, hi};
                               });
}

// The host takes these kernels for one or two tokens per step, and for up
// to kDecodeDot2MaxTokens while the step's pairs do not outnumber the
// experts; tiles hold one or two tokens (a group of more streams its rows
// once per tile).
int nt_max(int T) { return T <= 1 ? 1 : 2; }

}  // namespace

hipError_t launch_decode_up(const ExpertEntry* table, const WorkList* wl,
                            const int32_t* perm, const f16* x, f16* h, int T,
                            int d, int f, int K, int max_groups, hipStream_t s) {
  if (T < 1 || T > kDecodeDot2MaxTokens) return hipErrorInvalidValue;
  dim3 grid(f / UpRows<2>::value, max_groups);
  if (nt_max(T) == 1) decode_up_kernel<1><<<grid, kThreads, 0, s>>>(table, wl, perm, x, h, d, f, K);
  else decode_up_kernel<2><<<grid, kThreads, 0, s>>>(table, wl, perm, x, h, d, f, K);
  return hipGetLastError();
}

hipError_t launch_decode_down(const ExpertEntry* table, const WorkList* wl,
                              const int32_t* perm, const float* gate_w,
                              const f16* h, float* y, float* h_res, int T, int d,
                              int f, int K, hipStream_t s) {
  if (T < 1 || T > kDecodeDot2MaxTokens) return hipErrorInvalidValue;
  dim3 grid(d / DownRows<2>::value);
  if (nt_max(T) == 1)
    decode_down_kernel<1><<<grid, kThreads, 0, s>>>(table, wl, perm, gate_w, h, y, h_res, T, d, f, K);
  else
    decode_down_kernel<2><<<grid, kThreads, 0, s>>>(table, wl, perm, gate_w, h, y, h_res, T, d, f, K);
  return hipGetLastError();
}

hipError_t launch_rmsnorm(const float* h_res, f16* x_next, int T, int d,
                          float eps, hipStream_t s) {
  rmsnorm_kernel<<<T, kNormThreads, 0, s>>>(h_res, x_next, d, eps);
  return hipGetLastError();
}

}  // namespace moe
