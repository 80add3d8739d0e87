// Look-up-table sign application shared by the single-launch decode kernel
// (decode.hip) and the streaming list kernels (stream.hip).  Both files are
// compiled without floating-point contraction, and every sum below has one
// fixed order, so the two produce bit-identical results for a linear.
//
// For 4 consecutive reduction indices with values a0..a3, a 16-entry table
// holds every signed sum sum_i (bit i of m ? -a_i : +a_i) (Proposition 1:
// the binary factors only flip signs).  A packed 32-bit word (LB layout v1:
// 32 consecutive reduction indices of one output) is then 8 nibble look-ups.
#pragma once
#include "device_common.h"

namespace lb {
namespace lut {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kChunk = 32;         // blocks of 32 inputs per stage-1 chunk
constexpr int kMaxRuns = 16;       // d_in runs per latent (partial sums per z value)
constexpr int kBlk = 8 * 16 + 16;  // floats of one block's 8 nibble tables, padded (bank spread)

// Table swizzle: entry m of nibble table q of a block sits at m ^ tsw(q).
// tsw keeps 4-entry groups contiguous (128-bit writes) and spreads the writes
// of a wave's 64 builders over all LDS banks.  XORing a packed word with kKey
// applies tsw(q) to each nibble q at once.
__host__ __device__ constexpr int tsw(int q) { return (q & 6) << 1; }
constexpr uint32_t kKey = 0xCC884400u;
static_assert(((kKey >> 8) & 15) == tsw(2) && ((kKey >> 28) & 15) == tsw(7), "swizzle key");

// The 16 entries of one nibble table over a0..a3 (entry m = sum_i (bit i of m
// ? -a_i : a_i)), written as 4 groups of 4 at their swizzled positions.
__device__ __forceinline__ void build_table(float* t16, int q, float a0, float a1, float a2, float a3) {
  const float s01[4] = {a0 + a1, a1 - a0, a0 - a1, -a0 - a1};
  const float s23[4] = {a2 + a3, a3 - a2, a2 - a3, -a2 - a3};
  const int gs = tsw(q) >> 2;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const f32x4 v = {s01[0] + s23[c], s01[1] + s23[c], s01[2] + s23[c], s01[3] + s23[c]};
    *reinterpret_cast<f32x4*>(t16 + 4 * (c ^ gs)) = v;
  }
}

// build_table without the swizzle (entry m at position m): for kernels whose
// 64 lanes always read one table at a time (the same entries, so a look-up
// is the same value whatever the layout), the word then needs no XOR.
__device__ __forceinline__ void build_table_plain(float* t16, float a0, float a1, float a2, float a3) {
  const float s01[4] = {a0 + a1, a1 - a0, a0 - a1, -a0 - a1};
  const float s23[4] = {a2 + a3, a3 - a2, a2 - a3, -a2 - a3};
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const f32x4 v = {s01[0] + s23[c], s01[1] + s23[c], s01[2] + s23[c], s01[3] + s23[c]};
    *reinterpret_cast<f32x4*>(t16 + 4 * c) = v;
  }
}

// Signed sum of one packed word against the 8 tables of a block (tb8 points
// at the block's first table; wk is the word XORed with kKey).
__device__ __forceinline__ float word_sum(const float* tb8, uint32_t wk) {
  float v[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) v[q] = tb8[16 * q + ((wk >> (4 * q)) & 15)];
  return ((v[0] + v[1]) + (v[2] + v[3])) + ((v[4] + v[5]) + (v[6] + v[7]));
}

// word_sum with the look-up addresses taken from two pre-shifted copies of
// the word: byte j of e = (wk << 2) & 0x3C3C3C3C is 4 x nibble 2j, byte j of
// o = (wk >> 2) & 0x3C3C3C3C is 4 x nibble 2j + 1, so each address is one
// byte extract (plus the table's base) instead of a shift, a mask and a
// scale.  The same entries are read and added in the same order as word_sum.
// (The byte goes to the low byte of an address by one v_perm_b32: selector
// byte j takes byte j of the second operand, 0x0c gives zero.)
__device__ __forceinline__ uint32_t byte_of(uint32_t v, int j) {
  return __builtin_amdgcn_perm(0u, v, 0x0c0c0c00u | static_cast<uint32_t>(j));
}
__device__ __forceinline__ float word_sum_b(const float* tb8, uint32_t wk) {
  const uint32_t e = (wk << 2) & 0x3C3C3C3Cu, o = (wk >> 2) & 0x3C3C3C3Cu;
  const char* b = reinterpret_cast<const char*>(tb8);
  float v[8];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    v[2 * j] = *reinterpret_cast<const float*>(b + 64 * (2 * j) + byte_of(e, j));
    v[2 * j + 1] = *reinterpret_cast<const float*>(b + 64 * (2 * j + 1) + byte_of(o, j));
  }
  return ((v[0] + v[1]) + (v[2] + v[3])) + ((v[4] + v[5]) + (v[6] + v[7]));
}

// Table inputs a_i = x_i g_i of one 4-input group; inputs at or past d_in
// (the tail block of a ragged d_in) are zero.
template <int ACT, int SC, bool VEC>
__device__ __forceinline__ void table_inputs(const uint32_t (&xb)[4], const uint32_t (&gb)[4], int jb, int d_in,
                                             int tailv, float (&a)[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    a[i] = raw4_elem<ACT, VEC>(xb, i) * raw4_elem<SC, VEC>(gb, i);
    if (tailv != 0 && jb + i >= d_in) a[i] = 0.0f;  // x past d_in belongs to the next row
  }
}

// The fixed summation trees both kernels follow.
// Stage 1: a latent's partial sum over a run is the tree over 4 waves w of
// the tree over 4 lane groups m of sequential sums: (v0 + v1) + (v2 + v3).
__device__ __forceinline__ float tree4(float v0, float v1, float v2, float v3) { return (v0 + v1) + (v2 + v3); }
// Stage 2: the two paths' row sums scaled by their row scales, added in fp32.
__device__ __forceinline__ float row_value(float h0, float u0, float h1, float u1) { return h0 * u0 + h1 * u1; }

}  // namespace lut
}  // namespace lb
