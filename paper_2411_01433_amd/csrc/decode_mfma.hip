// Decode-path expert kernels on the matrix cores, for steps with several
// tokens per expert copy.  Same mathematics as decode.hip:
//
//   up:    h[p, r] = silu(W1[r,:] . x_t) * (W3[r,:] . x_t)          (fp16)
//   down:  e[q, r] = W2[r,:] . h[p]   for the pair p at work-list slot q
//          (fp32; the combine kernel forms sum_k w[t,k] e[pos(t,k), :])
//
// With several tokens per weight row the dot2 kernels spend more VALU issue
// per streamed byte than the HBM stream leaves (int4: dequantise plus one
// dot2 per token per weight pair).  Here one v_mfma_f32_16x16x32_f16 takes
// 16 weight rows x 32 columns (B operand, dequantised once) against up to
// 16 tokens (A operand), so the per-token cost moves to the matrix cores.
// MFMA lane layout: A[l%16][8(l/16)+i], B[8(l/16)+i][l%16], C[4(l/16)+i][l%16].
//
// Weight streaming.  A block owns 16 rows of one or two matrices; its waves
// take turns along the reduction dimension in stages of 128 bytes per row
// (64 fp16 columns, 128 int8, 256 int4 or 512 int2 codes).  Each of the two 16-byte loads of a stage covers
// 8 rows x one full 128-byte line: lane l reads chunk l/8 of row
// 8i + l%8 (i = 0, 1).  A DPP row rotation by 8 with bank masks then moves
// the chunks so that lane (n = l%16, g = l/16) holds chunks 2g and 2g+1 of
// row n, which is the B-fragment layout (columns of lane group g: a
// contiguous quarter of the stage).  Half-line or quarter-line accesses,
// which the fragment layout would give if loaded directly, stream
// measurably slower from HBM.
//
// A ring of D stages per wave keeps loads in flight while the matrix cores
// work; activations are loaded with their stage (the wait counter is in
// order, so a late activation load would drain the ring).
#include "moe_internal.h"

namespace moe {

namespace {

constexpr int kWaves = 2;  // waves per block; they split the reduction of 16 rows

template <class T>
__device__ inline const __attribute__((address_space(1))) T* gmem(const T* p) {
  return (const __attribute__((address_space(1))) T*)p;
}
__device__ inline f16x2 as_h2(uint32_t v) { return __builtin_bit_cast(f16x2, v); }
__device__ inline uint32_t as_u32(f16x2 v) { return __builtin_bit_cast(uint32_t, v); }
__device__ inline f16x8 pack8(uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
  return __builtin_bit_cast(f16x8, u32x4{a, b, c, d});
}

// Geometry of one stage.
template <int BITS> struct Geo {
  static constexpr int kCols = 1024 / BITS;      // 128 bytes of each row
  static constexpr int kLaneCols = kCols / 4;    // columns of one lane group
  static constexpr int kChunkCols = kCols / 8;   // columns of one 16-byte chunk
  static constexpr int kSteps = kCols / 32;      // MFMA k-steps
  static constexpr int kScales = BITS == 16 ? 0 : kLaneCols / kGroup;  // per lane
};

// Ring depth (stages in flight per wave).  The up-projection (two
// matrices) runs at 3 waves per SIMD (168 registers) with rings of 3 / 2 /
// 1 / 1 stages; the down-projection at 3 waves per SIMD with 4 / 3 / 2 / 1.
// A wave's bytes in flight are ring depth x 4 KB (up) or 2 KB (down);
// low-bit groups gain most from the third wave (int4 up 3.38 -> 3.66 TB/s
// at 8 tokens, with one stage instead of two), fp16 is unchanged.
template <int BITS, int NM>
constexpr int ring_depth() {
  return NM == 2 ? (BITS == 16 ? 3 : BITS == 8 ? 2 : 1)
                 : (BITS == 16 ? 4 : BITS == 8 ? 3 : BITS == 4 ? 2 : 1);
}

// DPP: lane i of each 16-lane row reads lane i^8 (rotation by 8); BANKS
// picks the 4-lane banks that take the moved value, the rest keep `old`.
constexpr int kRowRor8 = 0x128;
template <int BANKS>
__device__ inline uint32_t dpp8(uint32_t old, uint32_t src) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)src, kRowRor8, 0xF, BANKS, false);
}

// One stage of one matrix: the two raw 16-byte loads and, for codes, the
// scales of this lane's two chunks (packed f16 pairs).
template <int BITS> struct WStage {
  u32x4 v[2];
  uint32_t s[BITS == 2 ? 2 : 1];
};

// Per-lane sources of one matrix for one 16-row tile.
template <int BITS> struct WSrc {
  const uint8_t* row;    // load lane's row and chunk (the second load adds row8)
  int64_t row8;          // bytes between the two loads (8 rows)
  const f16* srow;       // scales of row n, from this lane group's first group
  int chunk;             // chunk index of the load lane (l / 8)
  int ngr;               // groups per row
  const uint8_t* dummy;  // target of ring loads past the last stage: this lane's activations
};

template <int BITS>
__device__ inline WSrc<BITS> wsrc(const ExpertEntry& ex, int m, int64_t row0, int64_t ld) {
  const int l = threadIdx.x & 63;
  const int64_t rb = ld * BITS / 8;
  const uint8_t* base = BITS == 16 ? reinterpret_cast<const uint8_t*>(ex.w[m])
                        : BITS == 8 ? ex.hq[m] : ex.q[m];
  WSrc<BITS> s;
  s.chunk = l >> 3;
  s.row = base + (row0 + (l & 7)) * rb + 16 * s.chunk;
  s.row8 = 8 * rb;
  s.ngr = (int)(ld / kGroup);
  s.dummy = nullptr;
  s.srow = BITS == 16 ? nullptr
                      : (BITS == 8 ? ex.hs[m] : ex.s[m]) + (row0 + (l & 15)) * s.ngr +
                            Geo<BITS>::kScales * (l >> 4);
  return s;
}

// Load stage kk (first column, a multiple of the stage width).  Chunks past
// the row end (the last stage of a code row may be partial) read the row's
// first chunk instead and get scale 0 at use; scales are read in aligned
// group pairs clamped to the row.  Nothing outside the row is touched,
// except by a ring slot past the wave's last stage (kk < 0), which reads
// 32 bytes of the lane's activation row (s.dummy) instead.
template <int BITS>
__device__ inline void load_w(const WSrc<BITS>& s, int64_t kk, int64_t ld, WStage<BITS>& w) {
  using G = const __attribute__((address_space(1))) u32x4*;
  int64_t off = kk * BITS / 8;
  if (BITS != 16) {
    const bool ok = kk + (int64_t)(s.chunk + 1) * Geo<BITS>::kChunkCols <= ld;
    off = ok ? off : -16 * (int64_t)s.chunk;
  }
  // kk < 0: a ring slot past the wave's last stage; its data is never
  // used, so the loads read this lane's activation row, which L2 holds
  // (reloading the wave's last stage re-read it from HBM: the streaming
  // loads do not keep it; one shared line would be a hot spot)
  // Weights stream with the nontemporal hint (each line is read once, by
  // one load); scales do not: a row's 128-byte scale line serves several
  // stages (8 for int4, 4 for int2), and streamed it was fetched again for
  // each (skewed 8-token Mixtral layer 237.9 -> 233.2 us per step).
  const bool past = kk < 0;
  const uint8_t* p = past ? s.dummy : s.row + off;
  w.v[0] = __builtin_nontemporal_load(reinterpret_cast<G>(gmem(p)));
  w.v[1] = __builtin_nontemporal_load(reinterpret_cast<G>(gmem(past ? p : p + s.row8)));
  if (BITS != 16) {
    using S = const __attribute__((address_space(1))) uint32_t*;
    const int g = (threadIdx.x & 63) >> 4;
    const int gi = (int)(kk / kGroup) + Geo<BITS>::kScales * g;  // first group of the lane
#pragma unroll
    for (int h = 0; h < (BITS == 2 ? 2 : 1); ++h) {
      // int8: one group per lane, read with its even neighbour
      const int idx = min(BITS == 8 ? (gi & ~1) : gi + 2 * h, s.ngr - 2);
      w.s[h] = *reinterpret_cast<S>(gmem(past ? reinterpret_cast<const f16*>(s.dummy)
                                             : s.srow - Geo<BITS>::kScales * g + idx));
    }
  }
}

// B fragments of this lane after the exchange: chunk 2g (c0) and 2g+1 (c1)
// of row n, 4 dwords each.
template <int BITS>
__device__ inline void exchange(const WStage<BITS>& w, u32x4& c0, u32x4& c1) {
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    c0[d] = dpp8<0xC>(w.v[0][d], w.v[1][d]);  // lanes l%16 >= 8 take v1 of lane l^8
    c1[d] = dpp8<0x3>(w.v[1][d], w.v[0][d]);  // lanes l%16 < 8 take v0 of lane l^8
  }
}

// Dequantisation pairs codes that sit 16 bits apart in a code word, so one
// and-or (v_bitop3) gives two fp16 halves: a code u whose lowest bit sits at
// bit p of a half becomes the fp16 2^(10-p) + u exactly when the exponent
// field is that of 2^(10-p) (0x6400: 1024 + u at p = 0, 0x5400: 64 + u at
// p = 4 ...).  A packed subtract removes 2^(10-p) + 2^(b-1) and a packed
// multiply applies the group scale.  The B fragment's 8 k-slots then hold
// the columns of its codes in pair order, and the A fragment is permuted to
// match (the reduction order is free):
//   int4, word e0..e7 (e_j at bits 4j): slots e0 e4 e1 e5 e2 e6 e3 e7
//   int2, word e0..e15 (e_j at bits 2j), step half H: slots e(4H) e(4H+8)
//        e(4H+1) e(4H+9) e(4H+2) e(4H+10) e(4H+3) e(4H+11)
constexpr uint32_t kAndOr = 0xEA;  // v_bitop3 truth table of (a & b) | c

__device__ inline uint32_t pair_bits(uint32_t w, uint32_t mask, uint32_t expo) {
  return __builtin_amdgcn_bitop3_b32(w, mask, expo, kAndOr);
}
__device__ inline uint32_t scaled(uint32_t v, uint32_t bias, f16x2 s2) {
  return as_u32((as_h2(v) - as_h2(bias)) * s2);
}

__device__ inline f16x8 deq4(uint32_t w, f16x2 s2) {
  const uint32_t w8 = w >> 8;
  return pack8(scaled(pair_bits(w, 0x000F000Fu, 0x64006400u), 0x64086408u, s2),   // 1024 + 8
               scaled(pair_bits(w, 0x00F000F0u, 0x54005400u), 0x54805480u, s2),   // 64 + 8
               scaled(pair_bits(w8, 0x000F000Fu, 0x64006400u), 0x64086408u, s2),
               scaled(pair_bits(w8, 0x00F000F0u, 0x54005400u), 0x54805480u, s2));
}

// int2 pairs k = 4H .. 4H+3 of a word: code k at bit 2k of each half (k <= 4
// in place, k >= 5 after a shift by 10).
template <int H>
__device__ inline f16x8 deq2(uint32_t w, f16x2 s2) {
  if (H == 0) {
    return pack8(scaled(pair_bits(w, 0x00030003u, 0x64006400u), 0x64026402u, s2),   // 1024 + 2
                 scaled(pair_bits(w, 0x000C000Cu, 0x5C005C00u), 0x5C085C08u, s2),   // 256 + 2
                 scaled(pair_bits(w, 0x00300030u, 0x54005400u), 0x54205420u, s2),   // 64 + 2
                 scaled(pair_bits(w, 0x00C000C0u, 0x4C004C00u), 0x4C804C80u, s2));  // 16 + 2
  } else {
    const uint32_t w10 = w >> 10;
    return pack8(scaled(pair_bits(w, 0x03000300u, 0x44004400u), 0x46004600u, s2),   // 4 + 2
                 scaled(pair_bits(w10, 0x00030003u, 0x64006400u), 0x64026402u, s2),
                 scaled(pair_bits(w10, 0x000C000Cu, 0x5C005C00u), 0x5C085C08u, s2),
                 scaled(pair_bits(w10, 0x00300030u, 0x54005400u), 0x54205420u, s2));
  }
}

// int8: codes e0..e7 in the bytes of (w0, w1).  A byte swap first puts e0,
// e1 (and e2, e3) 16 bits apart, so the and-or pairs come out in column
// order: (e0,e1)(e2,e3)(e4,e5)(e6,e7), no activation permutation needed.
__device__ inline uint32_t swap_mid_bytes(uint32_t w) {  // b0 b1 b2 b3 -> b0 b2 b1 b3
  return __builtin_amdgcn_perm(w, w, 0x03010200u);
}
__device__ inline f16x8 deq8(uint32_t w0, uint32_t w1, f16x2 s2) {
  const uint32_t a = swap_mid_bytes(w0), b = swap_mid_bytes(w1);
  return pack8(scaled(pair_bits(a, 0x00FF00FFu, 0x64006400u), 0x64806480u, s2),        // 1024 + 128
               scaled(pair_bits(a >> 8, 0x00FF00FFu, 0x64006400u), 0x64806480u, s2),
               scaled(pair_bits(b, 0x00FF00FFu, 0x64006400u), 0x64806480u, s2),
               scaled(pair_bits(b >> 8, 0x00FF00FFu, 0x64006400u), 0x64806480u, s2));
}

// low halves of (a, b) / high halves of (a, b) as one dword
__device__ inline uint32_t lo_lo(uint32_t a, uint32_t b) {
  return __builtin_amdgcn_perm(b, a, 0x05040100u);
}
__device__ inline uint32_t hi_hi(uint32_t a, uint32_t b) {
  return __builtin_amdgcn_perm(b, a, 0x07060302u);
}

// Slot position of element e of an 8-column (int4) or 16-column (int2)
// block: the layout in which the up-projection stores h for low-precision
// groups, so that the down-projection's natural-order fragment loads are
// already permuted.
template <int BITS>
__device__ inline int slot_of(int e) {
  constexpr int kHalfBlock = BITS == 4 ? 4 : 8;
  return e < kHalfBlock ? 2 * e : 2 * (e - kHalfBlock) + 1;
}

// Activation fragments of one stage, as loaded: lane (t, g) holds columns
// kk + kLaneCols g + 8j .. +7 of its token row for the steps j.  Chunks past
// the row end read column 0 instead (their weights are zero).
template <int BITS> struct AStage {
  f16x8 a[Geo<BITS>::kSteps];
};

template <int BITS>
__device__ inline void load_a(const f16* arow, int64_t kk, int64_t ld, AStage<BITS>& a) {
  using GG = Geo<BITS>;
  const int g = (threadIdx.x & 63) >> 4;
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    int64_t col = kk + GG::kLaneCols * g + GG::kChunkCols * c;
    if (BITS != 16) col = col + GG::kChunkCols <= ld ? col : 0;
    constexpr int kH = GG::kSteps / 2;
#pragma unroll
    for (int j = 0; j < kH; ++j)
      a.a[c * kH + j] = *reinterpret_cast<const f16x8*>(arow + col + 8 * j);
  }
}

// A fragment of step i in the k-slot order of the dequantised codes (PERM,
// the up-projection, whose activations are in column order); the
// down-projection's activations were stored in slot order already.  The
// permutation is applied at use, not at load: applied at load it would pin
// a wait for the stage just issued ahead of the scheduling barrier and
// drain the ring.
//   int4: x0..x7 -> x0 x4 x1 x5 x2 x6 x3 x7
//   int2: x0..x15 over steps 2q, 2q+1 -> x0 x8 x1 x9 x2 x10 x3 x11 | x4 x12 .. x7 x15
template <int BITS, bool PERM>
__device__ inline f16x8 a_frag(const AStage<BITS>& a, int i) {
  if (!PERM || BITS == 16 || BITS == 8) return a.a[i];
  if (BITS == 4) {
    const u32x4 v = __builtin_bit_cast(u32x4, a.a[i]);
    return __builtin_bit_cast(
        f16x8, u32x4{lo_lo(v[0], v[2]), hi_hi(v[0], v[2]), lo_lo(v[1], v[3]), hi_hi(v[1], v[3])});
  }
  const u32x4 v0 = __builtin_bit_cast(u32x4, a.a[i & ~1]);
  const u32x4 v1 = __builtin_bit_cast(u32x4, a.a[i | 1]);
  const int o = (i & 1) * 2;
  return __builtin_bit_cast(f16x8, u32x4{lo_lo(v0[o], v1[o]), hi_hi(v0[o], v1[o]),
                                         lo_lo(v0[o + 1], v1[o + 1]), hi_hi(v0[o + 1], v1[o + 1])});
}

// Scales of this lane's chunks for stage kk, zero for chunks past the end:
// sc[c][q] multiplies the q-th quantisation group of chunk c.
template <int BITS>
__device__ inline void chunk_scales(const WStage<BITS>& w, int64_t kk, int64_t ld,
                                    f16x2 (&sc)[2][2]) {
  using GG = Geo<BITS>;
  const int g = (threadIdx.x & 63) >> 4;
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const bool ok = kk + GG::kLaneCols * g + GG::kChunkCols * (c + 1) <= ld;
    // integer splats: a vector-element read of the packed pair went through
    // scratch memory
    const uint32_t sp = BITS == 2 ? w.s[c] : w.s[0];
    const uint32_t lo = __builtin_amdgcn_perm(sp, sp, 0x01000100u);
    const uint32_t hi = __builtin_amdgcn_perm(sp, sp, 0x03020302u);
    if (BITS == 8) {  // one group per lane group: the half of s[0] its parity picks
      sc[c][0] = sc[c][1] = as_h2(ok ? (((kk / kGroup + g) & 1) ? hi : lo) : 0u);
    } else if (BITS == 4) {  // one group per chunk: halves of s[0]
      sc[c][0] = sc[c][1] = as_h2(ok ? (c == 1 ? hi : lo) : 0u);
    } else {          // two groups per chunk: s[c]
      sc[c][0] = as_h2(ok ? lo : 0u);
      sc[c][1] = as_h2(ok ? hi : 0u);
    }
  }
}

// acc[m] += A . W_m over one stage; each A fragment serves every matrix.
template <int BITS, int NM>
__device__ inline void consume(const WStage<BITS> (&w)[NM], const AStage<BITS>& a, int64_t kk,
                               int64_t ld, f32x4 (&acc)[NM]) {
  constexpr bool kPerm = NM == 2;
  u32x4 c0[NM], c1[NM];
#pragma unroll
  for (int m = 0; m < NM; ++m) exchange<BITS>(w[m], c0[m], c1[m]);
  if (BITS == 16) {
#pragma unroll
    for (int m = 0; m < NM; ++m) {
      acc[m] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a.a[0], __builtin_bit_cast(f16x8, c0[m]), acc[m], 0, 0, 0);
      acc[m] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a.a[1], __builtin_bit_cast(f16x8, c1[m]), acc[m], 0, 0, 0);
    }
  } else {
    f16x2 sc[NM][2][2];
#pragma unroll
    for (int m = 0; m < NM; ++m) chunk_scales<BITS>(w[m], kk, ld, sc[m]);
    constexpr int kHalf = Geo<BITS>::kSteps / 2;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
#pragma unroll
      for (int j = 0; j < kHalf; ++j) {
        const f16x8 af = a_frag<BITS, kPerm>(a, c * kHalf + j);
#pragma unroll
        for (int m = 0; m < NM; ++m) {
          const u32x4& cw = c == 0 ? c0[m] : c1[m];
          const uint32_t word = cw[BITS == 8 ? 2 * j : BITS == 4 ? j : j / 2];
          f16x8 b;
          if (BITS == 8) b = deq8(word, cw[2 * j + 1], sc[m][c][0]);
          else if (BITS == 4) b = deq4(word, sc[m][c][0]);
          else if (j & 1) b = deq2<1>(word, sc[m][c][j / 4]);
          else b = deq2<0>(word, sc[m][c][j / 4]);
          acc[m] = __builtin_amdgcn_mfma_f32_16x16x32_f16(af, b, acc[m], 0, 0, 0);
        }
      }
    }
  }
}

// acc[m] (C tile: 16 tokens x 16 rows) = A(tokens, S) . W_m(rows, S)^T for
// the 16-row tile at row0 of the matrices mats[], over this wave's stages
// S = {wave, wave + kWaves, ...}: the waves of a block interleave 128-byte
// stages of the same rows.  Every load is unconditional (ring slots past
// the wave's last stage reload it and are not multiplied) so that the
// compiler's wait counts stay exact and the steady-state loop carries no
// branch.
template <int BITS, int NM>
__device__ inline void tile_gemm(const ExpertEntry& ex, const int (&mats)[NM], int64_t row0,
                                 int64_t ld, const f16* arow, int wave, f32x4 (&acc)[NM]) {
  using GG = Geo<BITS>;
  constexpr int D = ring_depth<BITS, NM>();
  const int64_t nst = ((ld + GG::kCols - 1) / GG::kCols - wave + kWaves - 1) / kWaves;
  if (nst <= 0) return;
  WSrc<BITS> src[NM];
#pragma unroll
  for (int m = 0; m < NM; ++m) {
    src[m] = wsrc<BITS>(ex, mats[m], row0, ld);
    src[m].dummy = reinterpret_cast<const uint8_t*>(arow);
  }
  auto col = [&](int64_t i) { return (wave + (i < nst ? i : nst - 1) * kWaves) * (int64_t)GG::kCols; };
  auto wcol = [&](int64_t i) { return i < nst ? col(i) : (int64_t)-1; };  // -1: past the end
  WStage<BITS> w[D][NM];
  AStage<BITS> a[D];
#pragma unroll
  for (int u = 0; u < D; ++u) {
    const int64_t kk = col(u);
#pragma unroll
    for (int m = 0; m < NM; ++m) load_w<BITS>(src[m], wcol(u), ld, w[u][m]);
    load_a<BITS>(arow, kk, ld, a[u]);
  }
  int64_t i0 = 0;
  for (; i0 + D <= nst; i0 += D) {
#pragma unroll
    for (int u = 0; u < D; ++u) {
      consume<BITS, NM>(w[u], a[u], col(i0 + u), ld, acc);
      const int64_t kk = col(i0 + u + D);
#pragma unroll
      for (int m = 0; m < NM; ++m) load_w<BITS>(src[m], wcol(i0 + u + D), ld, w[u][m]);
      load_a<BITS>(arow, kk, ld, a[u]);
      // keep the ring order: the scheduler would otherwise sink the loads
      // below the products and wait for nearly all of them each round
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  // the last nst - i0 < D stages sit in slots 0 .. nst - i0 - 1
#pragma unroll
  for (int u = 0; u < D - 1; ++u)
    if (u < nst - i0) consume<BITS, NM>(w[u], a[u], col(i0 + u), ld, acc);
}

// Sum of the waves' partial tiles in a fixed order; the result is valid in
// wave 0.  red holds kWaves * NM * 256 floats.
template <int NM>
__device__ inline void block_sum(f32x4 (&acc)[NM], float* red) {
  const int l = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int m = 0; m < NM; ++m)
    *reinterpret_cast<f32x4*>(red + ((wave * NM + m) * 64 + l) * 4) = acc[m];
  __syncthreads();
  if (wave == 0) {
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int v = 1; v < kWaves; ++v)
        acc[m] += *reinterpret_cast<const f32x4*>(red + ((v * NM + m) * 64 + l) * 4);
  }
  __syncthreads();
}

// ---------------------------------------------------------------- up-proj
template <int BITS>
__device__ void up_group(const ExpertEntry& ex, const Group& g, const int32_t* perm,
                         const f16* x, f16* h, int d, int f, int K, int64_t row0, float* red) {
  const int l = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
  const int mats[2] = {0, 1};
  for (int j0 = 0; j0 < g.count; j0 += 16) {
    const int n = min(16, g.count - j0);
    const int32_t* pairs = perm + g.offset + j0;
    // lanes past the last token repeat it: row m of the product depends on
    // row m of A only, and those rows are not stored
    const f16* arow = x + (int64_t)(pairs[min(l & 15, n - 1)] / K) * d;
    f32x4 acc[2] = {f32x4{0, 0, 0, 0}, f32x4{0, 0, 0, 0}};
    tile_gemm<BITS, 2>(ex, mats, row0, d, arow, wave, acc);
    block_sum<2>(acc, red);
    if (wave == 0) {
      const int64_t row = row0 + (l & 15);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int tok = 4 * (l >> 4) + i;
        if (tok < n) {
          const float a = acc[0][i], b = acc[1][i];
          // low-precision groups store h in the down-projection's slot order
          constexpr int kBlk = BITS == 4 ? 8 : 16;
          const int64_t hc = BITS >= 8 ? row
                             : (row & ~(int64_t)(kBlk - 1)) + slot_of<BITS>((int)(row & (kBlk - 1)));
          h[(int64_t)pairs[tok] * f + hc] = (f16)(a / (1.0f + expf(-a)) * b);
        }
      }
    }
  }
}

__global__ __launch_bounds__(64 * kWaves) __attribute__((amdgpu_waves_per_eu(3, 3)))
void decode_up_mfma_kernel(
    const ExpertEntry* __restrict__ table, const WorkList* __restrict__ wl,
    const int32_t* __restrict__ perm, const f16* __restrict__ x, f16* __restrict__ h,
    int d, int f, int K) {
  __shared__ float red[kWaves * 2 * 256];
  if ((int)blockIdx.y >= wl->n_groups) return;
  const Group g = wl->groups[blockIdx.y];
  const ExpertEntry ex = table[g.expert];
  const int64_t row0 = (int64_t)blockIdx.x * 16;
  if (g.bits == 16) up_group<16>(ex, g, perm, x, h, d, f, K, row0, red);
  else if (g.bits == 8) up_group<8>(ex, g, perm, x, h, d, f, K, row0, red);
  else if (g.bits == 4) up_group<4>(ex, g, perm, x, h, d, f, K, row0, red);
  else up_group<2>(ex, g, perm, x, h, d, f, K, row0, red);
}

// -------------------------------------------------------------- down-proj
template <int BITS>
__device__ void down_group(const ExpertEntry& ex, const Group& g, const int32_t* perm,
                           const f16* h, float* e, int d, int f, int64_t row0, float* red) {
  const int l = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
  const int mats[1] = {2};
  for (int j0 = 0; j0 < g.count; j0 += 16) {
    const int n = min(16, g.count - j0);
    const int32_t* pairs = perm + g.offset + j0;
    const f16* arow = h + (int64_t)pairs[min(l & 15, n - 1)] * f;
    f32x4 acc[1] = {f32x4{0, 0, 0, 0}};
    tile_gemm<BITS, 1>(ex, mats, row0, f, arow, wave, acc);
    block_sum<1>(acc, red);
    if (wave == 0) {
      const int64_t row = row0 + (l & 15);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int tok = 4 * (l >> 4) + i;
        if (tok < n) e[(int64_t)(g.offset + j0 + tok) * d + row] = acc[0][i];
      }
    }
  }
}

__global__ __launch_bounds__(64 * kWaves, 2) void decode_down_mfma_kernel(
    const ExpertEntry* __restrict__ table, const WorkList* __restrict__ wl,
    const int32_t* __restrict__ perm, const f16* __restrict__ h, float* __restrict__ e,
    int d, int f) {
  __shared__ float red[kWaves * 256];
  if ((int)blockIdx.y >= wl->n_groups) return;
  const Group g = wl->groups[blockIdx.y];
  const ExpertEntry ex = table[g.expert];
  const int64_t row0 = (int64_t)blockIdx.x * 16;
  if (g.bits == 16) down_group<16>(ex, g, perm, h, e, d, f, row0, red);
  else if (g.bits == 8) down_group<8>(ex, g, perm, h, e, d, f, row0, red);
  else if (g.bits == 4) down_group<4>(ex, g, perm, h, e, d, f, row0, red);
  else down_group<2>(ex, g, perm, h, e, d, f, row0, red);
}

}  // namespace

hipError_t launch_decode_up_mfma(const ExpertEntry* table, const WorkList* wl,
                                 const int32_t* perm, const f16* x, f16* h, int d,
                                 int f, int K, int max_groups, hipStream_t s) {
  dim3 grid(f / 16, max_groups);
  decode_up_mfma_kernel<<<grid, 64 * kWaves, 0, s>>>(table, wl, perm, x, h, d, f, K);
  return hipGetLastError();
}

hipError_t launch_decode_down_mfma(const ExpertEntry* table, const WorkList* wl,
                                   const int32_t* perm, const f16* h, float* e_perm,
                                   int d, int f, int max_groups, hipStream_t s) {
  dim3 grid(d / 16, max_groups);
  decode_down_mfma_kernel<<<grid, 64 * kWaves, 0, s>>>(table, wl, perm, h, e_perm, d, f);
  return hipGetLastError();
}

}  // namespace moe
