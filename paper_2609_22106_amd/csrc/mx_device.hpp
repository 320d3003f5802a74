// Device-side MXFP4 helpers for gfx950: E8M0 scale rule, E2M1 rounding,
// cross-lane reductions, and the block-scaled FP4 MFMA wrapper.
//
// MXFP4 (the format arXiv 2609.22106 uses for W4A4, after the OCP Microscaling
// specification it cites): 32 elements along K share an E8M0 scale
// 2^(code-127); code = clamp(biased_exp(amax) - 2, 0, 254) so the block
// maximum lands in E2M1's top binade [4, 8); each element divided by the scale
// is rounded to the nearest E2M1 value (0, .5, 1, 1.5, 2, 3, 4, 6), ties to
// the even code, saturating at 6.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace prq {
namespace dev {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// 16 bytes of a stream read once: a non-temporal load.  Used for the expert
// decode kernel's weight (128 experts' weights in one call, back to back:
// 24.9 -> 23.3 us); the dense decode kernel's weight loads measured the same
// back to back and 2.8 us slower over the graph-replayed decode step, and the
// quantizer's X copies slower at 2048 and 8192 rows, so both stay cached.
__device__ __forceinline__ uint4 load_stream16(const uint8_t* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

// E8M0 code of a block with largest magnitude `amax` (finite, >= 0).  The
// float32 exponent field is floor(log2 amax) + 127 for normal amax and 0 for
// zero/subnormal amax, so subtracting emax(E2M1) = 2 and clamping at 0 is the
// whole rule (a finite amax has exponent field <= 254, so code <= 252).
__device__ __forceinline__ uint32_t e8m0_code(float amax) {
  int bexp = static_cast<int>((__float_as_uint(amax) >> 23) & 0xFFu);
  return static_cast<uint32_t>(bexp > 2 ? bexp - 2 : 0);
}

// 2^(127 - code): multiplying by it divides by the block scale exactly.
__device__ __forceinline__ float e8m0_reciprocal(uint32_t code) {
  return __uint_as_float((254u - code) << 23);
}

// Nearest E2M1 code of t (|t| < 8 after scaling), ties to the even code,
// saturating at 6.  The sign bit is taken from v, the unscaled value, so a
// negative value that underflows in the scaling still encodes as -0.
__device__ __forceinline__ uint32_t e2m1_code(float t, float v) {
  float a = fabsf(t);
  uint32_t idx = static_cast<uint32_t>(a > 0.25f) + static_cast<uint32_t>(a >= 0.75f) +
                 static_cast<uint32_t>(a > 1.25f) + static_cast<uint32_t>(a >= 1.75f) +
                 static_cast<uint32_t>(a > 2.5f) + static_cast<uint32_t>(a >= 3.5f) +
                 static_cast<uint32_t>(a > 5.0f);
  return idx | ((__float_as_uint(v) >> 31) << 3);
}

// Max over the 4 lanes of a quad (lanes 4q .. 4q+3) with two DPP quad
// permutations (xor 1, xor 2); every lane of the quad must be active.
__device__ __forceinline__ float quad_max(float x) {
  int xi = __float_as_int(x);
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0, xi, 0xB1, 0xF, 0xF, false)));
  xi = __float_as_int(x);
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0, xi, 0x4E, 0xF, 0xF, false)));
  return x;
}

// One 16x16x128 block-scaled MFMA with FP4 (E2M1) A and B operands:
//   C[i][j] += sum_{k<128} 2^(sa-127) A[i][k] * 2^(sb-127) B[k][j]
// Lane l supplies A row (l % 16), K elements [32*(l/16), 32*(l/16)+32) as 16
// bytes of packed nibbles, and that 32-block's E8M0 scale in bits 0-7 of sa;
// likewise B column (l % 16).  Lane l receives C[4*(l/16) + r][l % 16], r=0..3.
__device__ __forceinline__ v4f mfma_fp4_16x16x128(const uint4& a, const uint4& b, uint32_t sa,
                                                   uint32_t sb, v4f c) {
  v8i av = {static_cast<int>(a.x), static_cast<int>(a.y), static_cast<int>(a.z),
            static_cast<int>(a.w), 0, 0, 0, 0};
  v8i bv = {static_cast<int>(b.x), static_cast<int>(b.y), static_cast<int>(b.z),
            static_cast<int>(b.w), 0, 0, 0, 0};
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(av, bv, c, 4, 4, 0,
                                                          static_cast<int>(sa), 0,
                                                          static_cast<int>(sb));
}

typedef float v16f __attribute__((ext_vector_type(16)));

// 32x32x64 block-scaled FP4 MFMA (the full-rate form: twice the products of
// the 16x16x128 form per issue slot): lane l supplies row l % 32, K elements
// [32 (l / 32), +32) of each operand with that block's E8M0 scale, and holds
// C[8 (j / 4) + 4 (l / 32) + j % 4][l % 32] in element j of the result.
__device__ __forceinline__ v16f mfma_fp4_32x32x64(const uint4& a, const uint4& b, uint32_t sa,
                                                  uint32_t sb, v16f c) {
  v8i av = {static_cast<int>(a.x), static_cast<int>(a.y), static_cast<int>(a.z),
            static_cast<int>(a.w), 0, 0, 0, 0};
  v8i bv = {static_cast<int>(b.x), static_cast<int>(b.y), static_cast<int>(b.z),
            static_cast<int>(b.w), 0, 0, 0, 0};
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av, bv, c, 4, 4, 0,
                                                         static_cast<int>(sa), 0,
                                                         static_cast<int>(sb));
}

// The same instruction with the scale bytes taken from byte kSelA of sa and
// byte kSelB of sb (the instruction's scale byte selects), so one register
// can carry the scales of several blocks.
template <int kSelA, int kSelB>
__device__ __forceinline__ v16f mfma_fp4_32x32x64_sel(const uint4& a, const uint4& b, uint32_t sa,
                                                      uint32_t sb, v16f c) {
  static_assert(kSelA >= 0 && kSelA < 4 && kSelB >= 0 && kSelB < 4, "byte select");
  v8i av = {static_cast<int>(a.x), static_cast<int>(a.y), static_cast<int>(a.z),
            static_cast<int>(a.w), 0, 0, 0, 0};
  v8i bv = {static_cast<int>(b.x), static_cast<int>(b.y), static_cast<int>(b.z),
            static_cast<int>(b.w), 0, 0, 0, 0};
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av, bv, c, 4, 4, kSelA,
                                                         static_cast<int>(sa), kSelB,
                                                         static_cast<int>(sb));
}

// Group g with off[g] <= row < off[g+1] for non-decreasing offsets
// (empty groups are skipped): the largest g in [0, G) with off[g] <= row.
__device__ __forceinline__ int find_group(const int32_t* __restrict__ off, int G, int row) {
  int lo = 0, hi = G - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (off[mid] <= row)
      lo = mid;
    else
      hi = mid - 1;
  }
  return lo;
}

// Group of rows visited in increasing order: a binary search for the first
// row, then a step forward past the groups' ends as rows cross them (a load
// only when a row leaves its group).  Same result as find_group for
// non-decreasing offsets; g stays in [0, G) whatever the offsets hold.
struct GroupCursor {
  int g = -1, g_end = 0;
  __device__ __forceinline__ int at(const int32_t* __restrict__ off, int G, int row) {
    if (g < 0 || row >= g_end) {
      if (g < 0) g = find_group(off, G, row);
      while (g + 1 < G && off[g + 1] <= row) ++g;
      g_end = g + 1 < G ? off[g + 1] : 0x7fffffff;
    }
    return g;
  }
};

}  // namespace dev
}  // namespace prq
