// Device helpers shared by the bf16 MFMA attention kernels (gfx950): operand
// types, the query rotation into MFMA operands, the online-softmax front and
// the cross-half lane swap.
#pragma once

#include "kvshot_common.h"

namespace kvshot {
namespace mfma {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));

constexpr float kLn2 = 0.693147180559945309f;

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ int32_t load_scalar_i32(const int32_t* base, int64_t idx) {
  // uniform address -> scalar load (constant address space)
  const __attribute__((address_space(4))) int32_t* cp =
      (const __attribute__((address_space(4))) int32_t*)(base);
  return cp[idx];
}

// Rotate one lane's (d, d + 64) pairs by the table angles and scale.  Operand
// chunk kc holds d = kc * 16 + hh * 8 + e, so chunks kc and kc + 4 pair up in-lane.
__device__ __forceinline__ void rope_rotate_to_bf16(const u32x4 (&raw)[8], const float2* cs, float scale,
                                                    bf16x8 (&dst)[8]) {
#pragma unroll
  for (int kc = 0; kc < 4; ++kc) {
    u32x4 lo, hi;
#pragma unroll
    for (int e2 = 0; e2 < 4; ++e2) {
      const uint32_t a = raw[kc][e2], bq = raw[kc + 4][e2];
      const float x1a = bf16_lo(a), x1b = bf16_hi(a);
      const float x2a = bf16_lo(bq), x2b = bf16_hi(bq);
      const float2 ca = cs[kc * 16 + 2 * e2], cb = cs[kc * 16 + 2 * e2 + 1];
      const float y1a = (x1a * ca.x - x2a * ca.y) * scale, y1b = (x1b * cb.x - x2b * cb.y) * scale;
      const float y2a = (x2a * ca.x + x1a * ca.y) * scale, y2b = (x2b * cb.x + x1b * cb.y) * scale;
      lo[e2] = pack_bf16x2(y1a, y1b);
      hi[e2] = pack_bf16x2(y2a, y2b);
    }
    dst[kc] = as_bf16x8(lo);
    dst[kc + 4] = as_bf16x8(hi);
  }
}

// Same rotation; the scaled query is kept as a bf16 pair hi + lo whose sum
// carries ~16 mantissa bits, so the scores see almost none of its rounding.
__device__ __forceinline__ void rope_rotate_split(const u32x4 (&raw)[8], const float2* cs, float scale,
                                                  bf16x8 (&hi_out)[8], bf16x8 (&lo_out)[8]) {
#pragma unroll
  for (int kc = 0; kc < 4; ++kc) {
    u32x4 h1, h2, l1, l2;
#pragma unroll
    for (int e2 = 0; e2 < 4; ++e2) {
      const uint32_t a = raw[kc][e2], bq = raw[kc + 4][e2];
      const float x1a = bf16_lo(a), x1b = bf16_hi(a);
      const float x2a = bf16_lo(bq), x2b = bf16_hi(bq);
      const float2 ca = cs[kc * 16 + 2 * e2], cb = cs[kc * 16 + 2 * e2 + 1];
      const float y1a = (x1a * ca.x - x2a * ca.y) * scale, y1b = (x1b * cb.x - x2b * cb.y) * scale;
      const float y2a = (x2a * ca.x + x1a * ca.y) * scale, y2b = (x2b * cb.x + x1b * cb.y) * scale;
      h1[e2] = pack_bf16x2(y1a, y1b);
      h2[e2] = pack_bf16x2(y2a, y2b);
      l1[e2] = pack_bf16x2(y1a - bf16_lo(h1[e2]), y1b - bf16_hi(h1[e2]));
      l2[e2] = pack_bf16x2(y2a - bf16_lo(h2[e2]), y2b - bf16_hi(h2[e2]));
    }
    hi_out[kc] = as_bf16x8(h1);
    hi_out[kc + 4] = as_bf16x8(h2);
    lo_out[kc] = as_bf16x8(l1);
    lo_out[kc + 4] = as_bf16x8(l2);
  }
}

struct SoftmaxState {
  float m;   // running max (log2 units), identical in both lane halves
  float l;   // this lane's partial sum over its keys
};

// A row's reference max only moves when a block's max exceeds it by more
// than this (log2 units): weights stay <= 2^8, and the output accumulator is
// rescaled only for the few blocks where some row's max jumps.  The final
// normalisation divides by the sum taken against the same reference, so the
// result is the same softmax.
constexpr float kRescaleSlack = 8.0f;

// Scores of keys that are not visible become -inf (select, never a product).
// Bit v of `valid`: the key of accumulator register v is visible to this lane's row.
__device__ __forceinline__ void apply_mask(f32x16& s, uint32_t valid) {
#pragma unroll
  for (int v = 0; v < 16; ++v) s[v] = ((valid >> v) & 1u) ? s[v] : -INFINITY;
}

// The value lane l ^ 32 holds, with one VALU lane swap between the wave's halves
// (v_permlane32_swap: the first result holds the low half in both halves, the
// second the high half) instead of an LDS permute.  The copy through asm keeps
// the compiler from treating the two operands as one value.
__device__ __forceinline__ float other_half(float x) {
  uint32_t y;
  asm volatile("v_mov_b32 %0, %1" : "=v"(y) : "v"(__float_as_uint(x)));
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), y, false, false);
  return __uint_as_float((threadIdx.x & 32) ? r[0] : r[1]);
}

// Branch-free front of the online-softmax update for one block: new reference
// max, bf16 weights P (as the B operand of O^T += V^T P^T), running sum.
// Returns through `alpha` the factor the output accumulator must be scaled by
// and through `rescale` whether any lane of the wave needs it.
__device__ __forceinline__ void softmax_front(const f32x16& s, SoftmaxState& st, u32x4 (&pw)[2], float& alpha,
                                              bool& rescale) {
  float bm = -INFINITY;
#pragma unroll
  for (int v = 0; v < 16; ++v) bm = fmaxf(bm, s[v]);
  bm = fmaxf(bm, other_half(bm));
  const bool jump = bm > st.m + kRescaleSlack;   // false while both are -inf
  const float mn = jump ? bm : st.m;
  const float mu = mn == -INFINITY ? 0.0f : mn;
  // 1 without a jump, 0 when the old max was -inf (also while every score so
  // far, this block's included, is masked: then -inf - (-inf) must not occur)
  alpha = __builtin_amdgcn_exp2f(st.m - mu);
  float ps = 0.0f;
#pragma unroll
  for (int v = 0; v < 16; v += 2) {
    const float p0 = __builtin_amdgcn_exp2f(s[v] - mu);
    const float p1 = __builtin_amdgcn_exp2f(s[v + 1] - mu);
    ps += p0 + p1;
    pw[v >> 3][(v & 7) >> 1] = pack_bf16x2(p0, p1);
  }
  st.l = st.l * alpha + ps;
  st.m = mn;
  rescale = __any(jump);
}

}  // namespace mfma
}  // namespace kvshot
