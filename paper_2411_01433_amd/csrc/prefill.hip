// Prefill path: the experts of Eq. 1 as an MFMA grouped GEMM with the
// quantised copies (int4 / int2 low copies, the int8 high copy of an int8
// model) dequantised in registers, then the weighted combine.
//
//   up:    H[j, r] = silu(X_g W1^T)[j, r] * (X_g W3^T)[j, r]     (fp16 out)
//   down:  E[j, r] = (H_g W2^T)[j, r]                             (fp32 out)
//   combine: y[t] = sum_k w[t,k] * E[pos(t,k)]                    (Eq. 1)
//
// X_g is the group's tokens: the router's stable counting sort lists every
// (token, slot) pair of a work group contiguously (perm[]); the up kernel
// gathers those token rows while staging them in LDS (the permute step),
// and H / E are kept in that group order (row j of the group at position
// offset + j), so the down kernel reads contiguous rows and the combine
// finds each pair through pos[].
//
// Tiling (v_mfma_f32_16x16x32_f16: lane l holds A[l%16][8(l/16)+i],
// B[8(l/16)+i][l%16] and C[4(l/16)+i][l%16]): M = tokens (A = activations
// from LDS, up to 160 per pass = 10 tiles), N = weight rows (B = weight
// rows, each lane's 8 k-values contiguous in memory), K = reduction dim in
// stages of 64.  A block of 4 waves owns 64 rows of W1 and W3 (16 per wave)
// in the up-projection and 128 rows of W2 (32 per wave) in the
// down-projection; each wave covers its rows for all the pass's tokens (up
// to 160), so every weight element is fetched from HBM once per pass and
// used by every token of the group.  Activations are double-buffered in
// LDS (one barrier per stage, later stages fetched into registers ahead of
// use) and weight fragments go straight into a ring of registers (see
// gemm_pass for the pipeline):
//   fp16: lane group g (= l/16) reads 16 B at k = 32s + 8g for step s;
//   int8: lane group g reads the 16 B of columns 16g..16g+15 of the stage
//         and step s uses its words 2s, 2s+1;
//   int4: lane group g reads the 8 B half group of columns 16g..16g+15 of
//         the stage and step s uses its word s;
//   int2: lane group g reads the 4 B of the same columns, half-word s.
// One load instruction covers 64 of each row's 128 stage bytes, so weight
// loads are plain (the line stays in L2 for the other half; nontemporal
// loads measured 20% more HBM traffic here).  Low codes are turned into
// fp16 with the 0x6400|u == 1024+u trick and scaled by the group's fp16
// scale (w = fp16(q*s)); the pair order this produces,
// (e0,e4)(e1,e5)(e2,e6)(e3,e7), is matched by staging the activations in
// LDS with the same permutation inside every 8 elements.
#include <type_traits>

#include "moe_internal.h"

namespace moe {

namespace {

// 4 waves per block; two blocks per compute unit in the up-projection, so
// that a stage barrier holds only its block's waves and the other block
// runs meanwhile.
constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr int kStageK = 64;               // reduction columns per stage (2 MFMA steps)
constexpr int kSteps = kStageK / 32;
constexpr int kPassTok = 160;             // tokens per pass (10 MFMA tiles)
constexpr int kTokTiles = kPassTok / 16;
constexpr int kLdsRow = kStageK + 8;      // halves per staged row (16 B pad)
constexpr int kUpRowsW = 16;              // weight rows per wave, up-projection
// staging: thread t owns rows (t >> 3) + 32 i of the pass and 8-column piece t & 7
constexpr int kPieces = kStageK / 8;
constexpr int kStageRowsPerThread = kPassTok / (kThreads / kPieces);

typedef __attribute__((address_space(1))) const u32x4* gvec4;

template <class T>
__device__ inline const __attribute__((address_space(1))) T* gmem(const T* p) {
  return (const __attribute__((address_space(1))) T*)p;
}

__device__ inline f16x2 as_h2(uint32_t v) { return __builtin_bit_cast(f16x2, v); }
__device__ inline uint32_t as_u32(f16x2 v) { return __builtin_bit_cast(uint32_t, v); }

__device__ inline f16x8 pack8(uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
  return __builtin_bit_cast(f16x8, u32x4{a, b, c, d});
}

// Position of element i of an 8-block in the staged activation layout for
// low-precision groups: x0 x4 x1 x5 x2 x6 x3 x7.
__device__ inline int perm8(int i) { return i < 4 ? 2 * i : 2 * (i - 4) + 1; }

// Activation staging of one pass.  Thread t owns rows (t >> 3) + 32 i of
// the pass and the 8-column piece t & 7 of every stage; the source rows
// are resolved once per pass (group row j is token perm[off + j] / K of x,
// or row off + j of H which is already in group order), then each stage
// is fetched into registers ahead of use and written to LDS [row][k].
// Rows beyond n repeat row n - 1 (row j of a product depends on row j of
// the activations only, and those rows are not stored) and stages past the
// end reload stage 0: every load is unconditional, so that no branch hides
// a load from the compiler's wait counting, which would then wait for all
// loads in flight (the weight prefetch included) at every stage.
// Rows are held as 32-bit byte offsets from a block-uniform base (the
// gathered token rows of x lie within T * d_model halves, a group's rows of
// H within kPassTok * d_ff), which leaves registers for a deeper ring.
struct ActStager {
  const char* base;
  uint32_t row[kStageRowsPerThread];
  u32x4 v[3][kStageRowsPerThread];  // up to three stages in flight

  __device__ void init(const f16* src, int64_t ld, const int32_t* perm, int off,
                       int j0, int n, int K, bool gather) {
    base = reinterpret_cast<const char*>(gather ? src : src + (int64_t)(off + j0) * ld);
#pragma unroll
    for (int i = 0; i < kStageRowsPerThread; ++i) {
      const int r = min((int)(threadIdx.x / kPieces) + (kThreads / kPieces) * i, n - 1);
      const int64_t sr = gather ? perm[off + j0 + r] / K : (int64_t)r;
      row[i] = (uint32_t)((sr * ld + (threadIdx.x % kPieces) * 8) * 2);
    }
  }
  template <int SLOT>
  __device__ void fetch(int64_t ld, int64_t k0) {
    const char* b = base + 2 * (k0 < ld ? k0 : 0);
#pragma unroll
    for (int i = 0; i < kStageRowsPerThread; ++i)
      v[SLOT][i] = *reinterpret_cast<const u32x4*>(b + row[i]);
  }
  template <int SLOT, bool PERMUTE>
  __device__ void store(f16* lds) const {
#pragma unroll
    for (int i = 0; i < kStageRowsPerThread; ++i) {
      u32x4 x = v[SLOT][i];
      if (PERMUTE) {
        const f16x8 a = __builtin_bit_cast(f16x8, x);
        f16x8 b;
#pragma unroll
        for (int e = 0; e < 8; ++e) b[perm8(e)] = a[e];
        x = __builtin_bit_cast(u32x4, b);
      }
      const int r = (threadIdx.x / kPieces) + (kThreads / kPieces) * i;
      *reinterpret_cast<u32x4*>(lds + r * kLdsRow + (threadIdx.x % kPieces) * 8) = x;
    }
  }
};

// int4 / int2 groups stage their activations permuted (perm8); fp16 and
// int8 groups in column order.
template <int BITS> constexpr bool kPermuted = BITS == 4 || BITS == 2;

// A fragment (activations) of token tile tt for step s of the stage.
template <int BITS>
__device__ inline f16x8 a_frag(const f16* lds, int tt, int s) {
  const int l = threadIdx.x & 63, g = l >> 4;
  const int col = BITS == 16 ? 32 * s + 8 * g : 16 * g + 8 * s;
  return *reinterpret_cast<const f16x8*>(lds + (tt * 16 + (l & 15)) * kLdsRow + col);
}

// Per-lane sources of one matrix M for one pass: the lane's weight row
// (codes or fp16) and scale row, advanced to its lane group's first column
// of a stage (fp16: 8g; codes: 16g, one scale per 32 columns).  Resolved
// once per pass with M a compile-time index, so the expert entry is never
// indexed at run time (that would put it in scratch memory, and a scratch
// load makes the wait before it cover every load in flight).
// Held as block-uniform bases and 32-bit per-lane byte offsets (a matrix
// is at most 2^30 weights), which the loads take as base + offset.
template <int BITS> struct WRow {
  const uint8_t* w;   // block-uniform
  const uint8_t* s;   // block-uniform
  uint32_t wo, so;    // this lane's byte offsets
};

template <int BITS, int M>
__device__ inline WRow<BITS> wrow(const ExpertEntry& ex, int64_t row, int64_t ld) {
  const int g = (threadIdx.x & 63) >> 4;
  WRow<BITS> r;
  if (BITS == 16) {
    r.w = reinterpret_cast<const uint8_t*>(ex.w[M]);
    r.wo = (uint32_t)((row * ld + 8 * g) * 2);
    r.s = nullptr;
    r.so = 0;
  } else {
    r.w = BITS == 8 ? ex.hq[M] : ex.q[M];
    r.s = reinterpret_cast<const uint8_t*>(BITS == 8 ? ex.hs[M] : ex.s[M]);
    r.wo = (uint32_t)(row * (ld * BITS / 8) + 16 * g * BITS / 8);
    r.so = (uint32_t)((row * (ld / kGroup) + (g >> 1)) * 2);
  }
  return r;
}

// Weight fragments of one 16-row tile of one matrix for one stage at
// column k0 (a multiple of 64).
template <int BITS> struct WFrag;

template <> struct WFrag<16> {
  u32x4 v[kSteps];
  __device__ inline void load(const WRow<16>& r, int64_t k0) {
#pragma unroll
    for (int s = 0; s < kSteps; ++s)
      v[s] = *gmem(reinterpret_cast<const u32x4*>(r.w + 2 * (k0 + 32 * s) + r.wo));
  }
  __device__ inline f16x8 get(int s) const { return __builtin_bit_cast(f16x8, v[s]); }
};

// Scales are held zero-extended in a register of their own: packed two to
// a register, each insertion waits for its load at once.
__device__ inline f16x2 splat_scale(uint32_t sc) {
  return as_h2(__builtin_amdgcn_perm(sc, sc, 0x01000100u));
}
__device__ inline uint32_t load_scale(const uint8_t* p) {
  return *gmem(reinterpret_cast<const uint16_t*>(p));
}

template <> struct WFrag<8> {
  u32x4 q;
  uint32_t sc;
  // lane group g holds the 16 codes of columns [k0 + 16g, k0 + 16g + 16)
  __device__ inline void load(const WRow<8>& r, int64_t k0) {
    q = *gmem(reinterpret_cast<const u32x4*>(r.w + k0 + r.wo));
    sc = load_scale(r.s + 2 * (k0 / kGroup) + r.so);
  }
  // bytes e0..e3 of a word, middle bytes swapped (e0 e2 e1 e3), pair as
  // (e0,e1)(e2,e3) in column order, scaled
  __device__ inline f16x8 get(int s) const {
    const f16x2 bias = as_h2(0x64806480u);  // 1152 = 1024 + 128
    const f16x2 s2 = splat_scale(sc);
    uint32_t o[4];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const uint32_t w = __builtin_amdgcn_perm(q[2 * s + k], q[2 * s + k], 0x03010200u);
      o[2 * k] = as_u32((as_h2((w & 0x00FF00FFu) | 0x64006400u) - bias) * s2);
      o[2 * k + 1] = as_u32((as_h2(((w >> 8) & 0x00FF00FFu) | 0x64006400u) - bias) * s2);
    }
    return pack8(o[0], o[1], o[2], o[3]);
  }
};

template <> struct WFrag<4> {
  u32x2 q;
  uint32_t sc;
  // lane group g holds the 16 codes of columns [k0 + 16g, k0 + 16g + 16)
  __device__ inline void load(const WRow<4>& r, int64_t k0) {
    q = *gmem(reinterpret_cast<const u32x2*>(r.w + k0 / 2 + r.wo));
    sc = load_scale(r.s + 2 * (k0 / kGroup) + r.so);
  }
  // word with e0..e7 at bits 4j -> (e0,e4)(e1,e5)(e2,e6)(e3,e7), scaled
  __device__ inline f16x8 get(int s) const {
    const uint32_t w = s == 0 ? q.x : q.y;
    const f16x2 bias = as_h2(0x64086408u);  // 1032 = 1024 + 8
    const f16x2 s2 = splat_scale(sc);
    uint32_t o[4];
#pragma unroll
    for (int k = 0; k < 4; ++k)
      o[k] = as_u32((as_h2(((w >> (4 * k)) & 0x000F000Fu) | 0x64006400u) - bias) * s2);
    return pack8(o[0], o[1], o[2], o[3]);
  }
};

template <> struct WFrag<2> {
  uint32_t q;
  uint32_t sc;
  // lane group g holds the 16 codes of columns [k0 + 16g, k0 + 16g + 16)
  __device__ inline void load(const WRow<2>& r, int64_t k0) {
    q = *gmem(reinterpret_cast<const uint32_t*>(r.w + k0 / 4 + r.wo));
    sc = load_scale(r.s + 2 * (k0 / kGroup) + r.so);
  }
  // half-word s holds e0..e7 at bits 2j; move byte 1 to byte 2 so that the
  // mask 0x00030003 pairs (e_k, e_{k+4})
  __device__ inline f16x8 get(int s) const {
    const uint32_t w = q >> (16 * s);
    const uint32_t v = (w & 0xFFu) | ((w & 0xFF00u) << 8);
    const f16x2 bias = as_h2(0x64026402u);  // 1026 = 1024 + 2
    const f16x2 s2 = splat_scale(sc);
    uint32_t o[4];
#pragma unroll
    for (int k = 0; k < 4; ++k)
      o[k] = as_u32((as_h2(((v >> (2 * k)) & 0x00030003u) | 0x64006400u) - bias) * s2);
    return pack8(o[0], o[1], o[2], o[3]);
  }
};

// One pass (up to kPassTok tokens) of one group over NM matrices:
// acc[rt][tt][m] accumulates the tokens of tile tt against the weight rows
// of tile rt.  Software pipeline over the stages k (64 columns each): the
// weight fragments sit in a ring of WRING register slots (stage k in slot
// k % WRING, reloaded with stage k + WRING as soon as its products are
// issued; 2 slots for the up-projection, 3 for the down-projection) and
// the activations of stage k + ADEPTH are fetched into register slot
// k % ADEPTH right after stage k's barrier.  The memory
// counter completes in order, so a weight load issued before an activation
// fetch must also be complete when that activation is stored: the weights
// get about ADEPTH stages to arrive, whatever the ring depth.  ADEPTH is 3
// for the down-projection and 1 for the up-projection (2 fits in its
// registers but measured no faster).  The stage loop is unrolled by kUnroll so that every ring index
// is static: rotating register slots would copy registers whose loads are
// still in flight, and make every stage wait for all of them.
constexpr int kUnroll = 6;  // multiple of WRING (2, 3), ADEPTH (1, 3) and the 2 LDS buffers

// Products of one stage, two token tiles at a time: the four fragments
// of a tile pair (two tiles x two k-steps) are read from LDS together and
// feed 4 * RT * NM products, ordered so that the products into one
// accumulator are 2 * RT * NM apart (no stall on the previous result).  A
// pair is computed whole when its first tile holds tokens: the second
// tile's rows then repeat the pass's last token and are not stored.
template <int BITS, int NM, int RT>
__device__ inline void stage_mma(const f16* cur, const WFrag<BITS> (&w)[RT][NM], int ntile,
                                 f32x4 (&acc)[RT][kTokTiles][NM]) {
  static_assert(kTokTiles % 2 == 0, "tile pairs");
  f16x8 b[kSteps][RT][NM];
#pragma unroll
  for (int s = 0; s < kSteps; ++s)
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int m = 0; m < NM; ++m) b[s][rt][m] = w[rt][m].get(s);
#pragma unroll
  for (int tp = 0; tp < kTokTiles; tp += 2) {
    // pair 0 always holds a token: every path consumes the weight
    // registers, so their reload needs no wait for an unconsumed load
    if (tp == 0 || tp < ntile) {
      f16x8 a[kSteps][2];
#pragma unroll
      for (int s = 0; s < kSteps; ++s)
#pragma unroll
        for (int t = 0; t < 2; ++t) a[s][t] = a_frag<BITS>(cur, tp + t, s);
#pragma unroll
      for (int s = 0; s < kSteps; ++s)
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int m = 0; m < NM; ++m)
              acc[rt][tp + t][m] = __builtin_amdgcn_mfma_f32_16x16x32_f16(
                  a[s][t], b[s][rt][m], acc[rt][tp + t][m], 0, 0, 0);
    }
  }
}

template <int BITS, int M0, int NM, int RT, int ADEPTH, int WRING>
__device__ void gemm_pass(const ExpertEntry& ex, int64_t wrow0, int64_t ld,
                          const f16* act, int64_t act_ld, const int32_t* perm,
                          int off, int j0, int n, int K, bool gather, f16* lds,
                          f32x4 (&acc)[RT][kTokTiles][NM]) {
  static_assert(NM == 1 || NM == 2, "one or two matrices");
  static_assert(kUnroll == 6 && kUnroll % WRING == 0 && kUnroll % ADEPTH == 0, "ring");
  const int l = threadIdx.x & 63;
  const int ntile = (n + 15) >> 4;
  const int64_t nst = ld / kStageK;  // ld is a multiple of kStageK
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int tt = 0; tt < kTokTiles; ++tt)
#pragma unroll
      for (int m = 0; m < NM; ++m) acc[rt][tt][m] = f32x4{0, 0, 0, 0};
  WRow<BITS> src[RT][NM];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int64_t row = wrow0 + rt * 16 + (l & 15);
    src[rt][0] = wrow<BITS, M0>(ex, row, ld);
    if constexpr (NM == 2) src[rt][1] = wrow<BITS, M0 + 1>(ex, row, ld);
  }
  // ring slots past the last stage (never multiplied) reload the last
  // stage, which the ring loaded a few stages before and L2 still holds
  // (stage 0 would come from HBM again): unconditional loads, see ActStager
  auto load_w = [&](WFrag<BITS> (&w)[RT][NM], int64_t k) {
    const int64_t kc = (k < nst ? k : nst - 1) * kStageK;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int m = 0; m < NM; ++m) w[rt][m].load(src[rt][m], kc);
  };
  ActStager st;
  st.init(act, act_ld, perm, off, j0, n, K, gather);
  st.fetch<0>(act_ld, 0);
  if (ADEPTH >= 2) st.fetch<1>(act_ld, kStageK);
  if (ADEPTH >= 3) st.fetch<2>(act_ld, 2 * kStageK);
  // issue order as in the loop (activations, then weights), so that the
  // wait before the first store is the loop's
  __builtin_amdgcn_sched_barrier(0);
  WFrag<BITS> w[WRING][RT][NM];
#pragma unroll
  for (int u = 0; u < WRING; ++u) load_w(w[u], u);
  // one stage; u = k % kUnroll is a compile-time constant.  The stages of
  // the main loop are unconditional: a skippable stage would let the
  // compiler assume its loads missing and wait for every load in flight
  // (the tail, under kUnroll stages, accepts that).
  auto stage = [&](int64_t k, auto uc) {
    constexpr int u = decltype(uc)::value;
    constexpr int kSlot = u % ADEPTH;
    // the buffer written here was last read two stages ago, before the
    // previous stage's barrier
    f16* cur = lds + (u & 1) * (kPassTok * kLdsRow);
    st.store<kSlot, kPermuted<BITS>>(cur);
    __syncthreads();
    st.fetch<kSlot>(act_ld, (k + ADEPTH) * kStageK);
    stage_mma<BITS, NM, RT>(cur, w[u % WRING], ntile, acc);
    load_w(w[u % WRING], k + WRING);
    // keep stages apart: scheduled across stages, the loads and fragment
    // reads of later stages stretch the registers' live ranges
    __builtin_amdgcn_sched_barrier(0);
  };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I3 = std::integral_constant<int, 3>;
  using I4 = std::integral_constant<int, 4>;
  using I5 = std::integral_constant<int, 5>;
  int64_t k0 = 0;
  for (; k0 + kUnroll <= nst; k0 += kUnroll) {
    stage(k0, I0{}); stage(k0 + 1, I1{}); stage(k0 + 2, I2{});
    stage(k0 + 3, I3{}); stage(k0 + 4, I4{}); stage(k0 + 5, I5{});
  }
  // the last nst - k0 < kUnroll stages
  const int64_t r = nst - k0;
  if (r > 0) stage(k0, I0{});
  if (r > 1) stage(k0 + 1, I1{});
  if (r > 2) stage(k0 + 2, I2{});
  if (r > 3) stage(k0 + 3, I3{});
  if (r > 4) stage(k0 + 4, I4{});
  __syncthreads();  // the LDS buffers are reused by the next pass
}

template <int BITS>
__device__ __forceinline__ void up_group(const ExpertEntry& ex, const Group& g, const int32_t* perm,
                         const f16* x, f16* h, int d, int f, int K, int tile, f16* lds) {
  constexpr int RT = kUpRowsW / 16;
  const int l = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t wrow0 = (int64_t)tile * kWaves * kUpRowsW + wave * kUpRowsW;
  for (int j0 = 0; j0 < g.count; j0 += kPassTok) {
    const int n = min(kPassTok, g.count - j0);
    f32x4 acc[RT][kTokTiles][2];
    gemm_pass<BITS, 0, 2, RT, 1, 2>(ex, wrow0, d, x, d, perm, g.offset, j0, n, K, true, lds, acc);
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const int64_t row = wrow0 + rt * 16 + (l & 15);
#pragma unroll
      for (int tt = 0; tt < kTokTiles; ++tt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int j = tt * 16 + 4 * (l >> 4) + i;
          if (j < n && row < f) {
            const float a = acc[rt][tt][0][i], b = acc[rt][tt][1][i];
            h[(int64_t)(g.offset + j0 + j) * f + row] = (f16)(a / (1.0f + expf(-a)) * b);
          }
        }
    }
  }
}

// Work items are (group, row tile) in group-major order.  The hardware
// hands consecutive blocks to the 8 XCDs in turn (block b to XCD b % 8), so
// block b takes item (b % 8) * per + b / 8, per = ceil(items / 8): each XCD
// runs one contiguous eighth of the items, i.e. the tiles of one or two
// groups, whose gathered activation rows then sit in that XCD's L2 only
// instead of being fetched by all eight (up- and down-projection of the
// 512-token Mixtral-shaped stack: 21.2 -> 20.9 ms per pass).
__device__ inline bool xcd_item(int n_groups, int n_tiles, int& gi, int& tile) {
  const int total = n_groups * n_tiles, per = (total + 7) >> 3;
  const int slot = blockIdx.x >> 3, item = (blockIdx.x & 7) * per + slot;
  if (slot >= per || item >= total) return false;
  gi = item / n_tiles;
  tile = item - gi * n_tiles;
  return true;
}

__global__ __launch_bounds__(kThreads, 2) void prefill_up_kernel(
    const ExpertEntry* __restrict__ table, const WorkList* __restrict__ wl,
    const int32_t* __restrict__ perm, const f16* __restrict__ x, f16* __restrict__ h,
    int d, int f, int K, int n_tiles) {
  __shared__ f16 lds[2 * kPassTok * kLdsRow];
  int gi, tile;
  if (!xcd_item(wl->n_groups, n_tiles, gi, tile)) return;
  const Group g = wl->groups[gi];
  const ExpertEntry ex = table[g.expert];
  if (g.bits == 16) up_group<16>(ex, g, perm, x, h, d, f, K, tile, lds);
  else if (g.bits == 8) up_group<8>(ex, g, perm, x, h, d, f, K, tile, lds);
  else if (g.bits == 4) up_group<4>(ex, g, perm, x, h, d, f, K, tile, lds);
  else up_group<2>(ex, g, perm, x, h, d, f, K, tile, lds);
}

// RT 16-row tiles of W2 per wave, each activation fragment read from LDS
// serving all of them
template <int BITS, int RT>
__device__ __forceinline__ void down_group(const ExpertEntry& ex, const Group& g, const f16* h,
                           float* e, int d, int f, int tile, f16* lds) {
  const int l = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t wrow0 = (int64_t)(tile * kWaves + wave) * (16 * RT);
  for (int j0 = 0; j0 < g.count; j0 += kPassTok) {
    const int n = min(kPassTok, g.count - j0);
    f32x4 acc[RT][kTokTiles][1];
    gemm_pass<BITS, 2, 1, RT, 3, 3>(ex, wrow0, f, h, f, nullptr, g.offset, j0, n, 1, false, lds, acc);
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const int64_t row = wrow0 + rt * 16 + (l & 15);
#pragma unroll
      for (int tt = 0; tt < kTokTiles; ++tt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int j = tt * 16 + 4 * (l >> 4) + i;
          if (j < n && row < d) e[(int64_t)(g.offset + j0 + j) * d + row] = acc[rt][tt][0][i];
        }
    }
  }
}

// RT = 2 (32 rows per wave, 128 per block) when d_model allows it: twice
// the products per LDS fragment read, at one block of 4 waves per compute
// unit with up to 512 registers each (down-projection of a Mixtral-shaped
// 512-token layer 284 -> 256 us against RT = 1 at two blocks per unit).
template <int RT>
__global__ __launch_bounds__(kThreads, RT == 2 ? 1 : 2) void prefill_down_kernel(
    const ExpertEntry* __restrict__ table, const WorkList* __restrict__ wl,
    const f16* __restrict__ h, float* __restrict__ e, int d, int f, int n_tiles) {
  __shared__ f16 lds[2 * kPassTok * kLdsRow];
  int gi, tile;
  if (!xcd_item(wl->n_groups, n_tiles, gi, tile)) return;
  const Group g = wl->groups[gi];
  const ExpertEntry ex = table[g.expert];
  if (g.bits == 16) down_group<16, RT>(ex, g, h, e, d, f, tile, lds);
  else if (g.bits == 8) down_group<8, RT>(ex, g, h, e, d, f, tile, lds);
  else if (g.bits == 4) down_group<4, RT>(ex, g, h, e, d, f, tile, lds);
  else down_group<2, RT>(ex, g, h, e, d, f, tile, lds);
}

// One block per token; thread i owns the float4 pieces i, i + 1024, ... of
// the token's row (d is a multiple of 64): y[t] = sum_k w[t,k] *
// E[pos(t,k)] in slot order (skip -> 0); with h_res: h_res[t] += that and,
// with x_next, x_next[t] = fp16(rmsnorm(h_res[t])) by rmsnorm_rows (the
// same piece layout, so each thread reads back the pieces it wrote).
constexpr int kCombineThreads = kNormThreads;

__global__ __launch_bounds__(kCombineThreads) void combine_prefill_kernel(
    const float* __restrict__ e, const int32_t* __restrict__ pos,
    const float* __restrict__ w, const int8_t* __restrict__ prec, int d, int K,
    float* __restrict__ y, float* __restrict__ h_res, f16* __restrict__ x_next,
    float eps) {
  __shared__ float red[kCombineThreads / 64];
  __shared__ int s_pos[kMaxTopK];
  __shared__ float s_w[kMaxTopK];
  const int t = blockIdx.x;
  if (threadIdx.x < K) {
    const int p = t * K + threadIdx.x;
    s_pos[threadIdx.x] = prec[p] == PREC_SKIP ? -1 : pos[p];
    s_w[threadIdx.x] = w[p];
  }
  __syncthreads();
  const int64_t base = (int64_t)t * d;
  const int n4 = d >> 2;
#pragma unroll
  for (int i = 0; i < kNormPieces; ++i) {
    const int q = threadIdx.x + i * kCombineThreads;
    if (q < n4) {
      const int c = 4 * q;
      f32x4 acc = {0, 0, 0, 0};
      for (int k = 0; k < K; ++k)
        if (s_pos[k] >= 0) {
          const f32x4 v = *reinterpret_cast<const f32x4*>(e + (int64_t)s_pos[k] * d + c);
          acc += s_w[k] * v;
        }
      if (h_res) {
        f32x4* hp = reinterpret_cast<f32x4*>(h_res + base + c);
        *hp = *hp + acc;
      } else {
        *reinterpret_cast<f32x4*>(y + base + c) = acc;
      }
    }
  }
  if (!h_res || !x_next) return;  // no norm asked for (the next layer forms it)
  rmsnorm_rows<1, kNormPieces>(h_res + base, d, eps, 0, 1, red,
                               [&](int, int q, uint32_t lo, uint32_t hi) {
                                 *reinterpret_cast<u32x2*>(x_next + base + 4 * q) = u32x2{lo, hi};
                               });
}

}  // namespace

hipError_t launch_prefill_up(const ExpertEntry* table, const WorkList* wl,
                             const int32_t* perm, const f16* x, f16* h, int T,
                             int d, int f, int K, int max_groups, hipStream_t s) {
  (void)T;
  // whole stages and whole row tiles: every load stays inside the matrices
  if (d % kStageK || f % (kWaves * kUpRowsW)) return hipErrorInvalidValue;
  const int rows_per_block = kWaves * kUpRowsW;
  const int n_tiles = (f + rows_per_block - 1) / rows_per_block;
  prefill_up_kernel<<<(max_groups * n_tiles + 7) / 8 * 8, kThreads, 0, s>>>(table, wl, perm, x, h, d, f, K, n_tiles);
  return hipGetLastError();
}

hipError_t launch_prefill_down(const ExpertEntry* table, const WorkList* wl,
                               const f16* h, float* e, int T, int d, int f, int K,
                               int max_groups, hipStream_t s) {
  (void)T;
  (void)K;
  // whole stages and whole row tiles: every load stays inside the matrices
  if (f % kStageK || d % (kWaves * 16)) return hipErrorInvalidValue;
  if (d % (kWaves * 32) == 0) {
    const int n_tiles = d / (kWaves * 32);
    prefill_down_kernel<2><<<(max_groups * n_tiles + 7) / 8 * 8, kThreads, 0, s>>>(table, wl, h, e, d, f, n_tiles);
  } else {
    const int n_tiles = d / (kWaves * 16);
    prefill_down_kernel<1><<<(max_groups * n_tiles + 7) / 8 * 8, kThreads, 0, s>>>(table, wl, h, e, d, f, n_tiles);
  }
  return hipGetLastError();
}

hipError_t launch_combine_prefill(const float* e, const int32_t* pos, const float* w,
                                  const int8_t* prec, int T, int d, int K, float* y,
                                  float* h_res, f16* x_next, float eps, hipStream_t s) {
  combine_prefill_kernel<<<T, kCombineThreads, 0, s>>>(e, pos, w, prec, d, K, y, h_res, x_next, eps);
  return hipGetLastError();
}

}  // namespace moe
