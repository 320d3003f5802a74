// Fused activation quantization with the online tail copy (arXiv 2609.22106,
// Sec. "Activation tail construction" and "Kernel design"; Algorithm 1,
// step 11):
//
//   Z~[m, p] = X[m, perm[p]] * d[p],  d[p] = 1 / s_{perm[p]}   (D^-1 P of Eq. 1, float32)
//   Aq/Asc   = MXFP4(Z~) and its k/32 tail blocks written once more after the
//              K/32 main blocks (== MXFP4([Z~, Z~_tail]) since the tail starts
//              on a block boundary)
//
// Memory-bound: per row it reads 2K bytes of bf16 and writes (K+k)/2 code bytes
// and (K+k)/32 scale bytes.  Every thread owns quarter blocks ("units") of 8
// consecutive positions: the 4 lanes of a quad hold one 32-block, whose max is
// reduced with two DPP quad permutations; a thread writes one 32-bit word of 8
// nibbles (a wave writes 256 contiguous bytes) and lane 0 of the quad the scale.
// Two kernels:
//   * rows kernel (few rows, decode): a thread per unit across many
//     workgroups; perm and d of its 8 positions live in registers (no
//     dependent gather: d is given in position order) and the row values are
//     gathered straight from global memory (rows of a few KB stay in L2).
//   * LDS kernel (many rows, prefill): a workgroup keeps the group's perm and d
//     in LDS for a contiguous range of rows; each row is staged into LDS with
//     coalesced 16-byte loads -- the next row is already being loaded into
//     registers while the current one is quantized -- and gathered from LDS.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>

#include "mx_device.hpp"
#include "prq_internal.h"

namespace prq {
namespace {

constexpr int kRowsThreads = 256;
constexpr int kLdsThreads = 512;
constexpr int kMaxRowVec = 4;   // uint4 per thread of a staged row: K <= 4 * 8 * 512 = 16384

struct Unit {
  int src[8];
  float d[8];
};

__device__ __forceinline__ void load_unit(const int32_t* __restrict__ perm,
                                          const float* __restrict__ inv, int g, int K, int u,
                                          Unit* out) {
  const int64_t base = static_cast<int64_t>(g) * K + (u << 3);
  if (perm) {
    const int4 p0 = *reinterpret_cast<const int4*>(perm + base);
    const int4 p1 = *reinterpret_cast<const int4*>(perm + base + 4);
    const int p[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
#pragma unroll
    for (int j = 0; j < 8; ++j)   // an out-of-range entry reads channel 0 (never past the row)
      out->src[j] = static_cast<unsigned>(p[j]) < static_cast<unsigned>(K) ? p[j] : 0;
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) out->src[j] = (u << 3) + j;
  }
  if (inv) {
    const float4 d0 = *reinterpret_cast<const float4*>(inv + base);
    const float4 d1 = *reinterpret_cast<const float4*>(inv + base + 4);
    out->d[0] = d0.x; out->d[1] = d0.y; out->d[2] = d0.z; out->d[3] = d0.w;
    out->d[4] = d1.x; out->d[5] = d1.y; out->d[6] = d1.z; out->d[7] = d1.w;
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) out->d[j] = 1.0f;
  }
}

// Quantize 8 values of a quarter block (the quad holds the whole block) and
// write the word, the scale and, for tail blocks, their copies.
__device__ __forceinline__ void quantize_store(const float (&z)[8], int u, int tail_unit0,
                                               int copy_units, int copy_blocks, uint8_t* arow,
                                               uint8_t* srow) {
  float amax = 0.0f;
#pragma unroll
  for (int j = 0; j < 8; ++j) amax = fmaxf(amax, fabsf(z[j]));
  amax = dev::quad_max(amax);
  const uint32_t code = dev::e8m0_code(amax);
  const float mul = dev::e8m0_reciprocal(code);
  uint32_t w = 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) w |= dev::e2m1_code(z[j] * mul, z[j]) << (4 * j);
  *reinterpret_cast<uint32_t*>(arow + 4 * u) = w;
  if ((u & 3) == 0) srow[u >> 2] = static_cast<uint8_t>(code);
  if (u >= tail_unit0) {  // online copy of the quantized tail and its scales
    *reinterpret_cast<uint32_t*>(arow + 4 * (u + copy_units)) = w;
    if ((u & 3) == 0) srow[(u >> 2) + copy_blocks] = static_cast<uint8_t>(code);
  }
}

template <bool kGrouped>
__global__ __launch_bounds__(kRowsThreads) void act_quant_rows_kernel(
    const uint16_t* __restrict__ X, int64_t ld_x, int M, int K, int k_tail,
    const float* __restrict__ inv, const int32_t* __restrict__ perm,
    const int32_t* __restrict__ offsets, int G, int rows_per_wg, uint8_t* __restrict__ Aq,
    uint8_t* __restrict__ Asc) {
  const int u = blockIdx.x * kRowsThreads + threadIdx.x;
  if (u >= (K >> 3)) return;   // K/8 is a multiple of 4: quads leave together
  const int r0 = blockIdx.y * rows_per_wg;
  const int r1 = min(M, r0 + rows_per_wg);
  const int k_aug = K + k_tail;
  const int64_t row_bytes = k_aug >> 1;
  const int nb = k_aug >> 5;
  Unit un;
  int cur_g = -1;
  for (int r = r0; r < r1; ++r) {
    const int g = kGrouped ? dev::find_group(offsets, G, r) : 0;
    if (g != cur_g) {
      load_unit(perm, inv, g, K, u, &un);
      cur_g = g;
    }
    const uint16_t* xr = X + static_cast<int64_t>(r) * ld_x;
    float z[8];
#pragma unroll
    for (int j = 0; j < 8; ++j)
      z[j] = __uint_as_float(static_cast<uint32_t>(xr[un.src[j]]) << 16) * un.d[j];
    quantize_store(z, u, (K - k_tail) >> 3, k_tail >> 3, k_tail >> 5,
                   Aq + static_cast<int64_t>(r) * row_bytes, Asc + static_cast<int64_t>(r) * nb);
  }
}

inline size_t lds_kernel_bytes(int K) {
  // d (float) + one staged bf16 row + perm (uint16)
  return static_cast<size_t>(K) * 4 + static_cast<size_t>(K) * 2 + static_cast<size_t>(K) * 2;
}

template <bool kGrouped>
__global__ __launch_bounds__(kLdsThreads) void act_quant_lds_kernel(
    const uint16_t* __restrict__ X, int64_t ld_x, int M, int K, int k_tail,
    const float* __restrict__ inv, const int32_t* __restrict__ perm,
    const int32_t* __restrict__ offsets, int G, int rows_per_wg, uint8_t* __restrict__ Aq,
    uint8_t* __restrict__ Asc) {
  extern __shared__ __align__(16) unsigned char smem[];
  float* s_d = reinterpret_cast<float*>(smem);                                       // [K]
  uint16_t* s_row = reinterpret_cast<uint16_t*>(smem + static_cast<size_t>(K) * 4);  // [K]
  uint16_t* s_perm = s_row + K;                                                      // [K]

  const int tid = threadIdx.x;
  const int r0 = blockIdx.x * rows_per_wg;
  const int r1 = min(M, r0 + rows_per_wg);
  const int units = K >> 3;
  const int vecs = K >> 3;    // uint4 per row
  const int k_aug = K + k_tail;
  const int64_t row_bytes = k_aug >> 1;
  const int nb = k_aug >> 5;

  uint4 pre[kMaxRowVec];
  auto prefetch = [&](int r) {
    const uint4* xr = reinterpret_cast<const uint4*>(X + static_cast<int64_t>(r) * ld_x);
#pragma unroll
    for (int i = 0; i < kMaxRowVec; ++i) {
      const int v = tid + i * kLdsThreads;
      if (v < vecs) pre[i] = xr[v];
    }
  };
  if (r0 < r1) prefetch(r0);

  int cur_g = -1;
  for (int r = r0; r < r1; ++r) {
    const int g = kGrouped ? dev::find_group(offsets, G, r) : 0;
    __syncthreads();  // the previous row's readers are done with s_row / s_perm / s_d
    if (g != cur_g) {
      const int32_t* pg = perm ? perm + static_cast<int64_t>(g) * K : nullptr;
      const float* dg = inv ? inv + static_cast<int64_t>(g) * K : nullptr;
      for (int p = tid; p < K; p += kLdsThreads) {
        int src = pg ? pg[p] : p;
        src = static_cast<unsigned>(src) < static_cast<unsigned>(K) ? src : 0;  // never past the row
        s_perm[p] = static_cast<uint16_t>(src);
        s_d[p] = dg ? dg[p] : 1.0f;
      }
      cur_g = g;
    }
    uint4* sr = reinterpret_cast<uint4*>(s_row);
#pragma unroll
    for (int i = 0; i < kMaxRowVec; ++i) {
      const int v = tid + i * kLdsThreads;
      if (v < vecs) sr[v] = pre[i];
    }
    if (r + 1 < r1) prefetch(r + 1);   // in flight while this row is quantized
    __syncthreads();

    uint8_t* arow = Aq + static_cast<int64_t>(r) * row_bytes;
    uint8_t* srow = Asc + static_cast<int64_t>(r) * nb;
    for (int u = tid; u < units; u += kLdsThreads) {
      float z[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int p = (u << 3) + j;
        z[j] = __uint_as_float(static_cast<uint32_t>(s_row[s_perm[p]]) << 16) * s_d[p];
      }
      quantize_store(z, u, (K - k_tail) >> 3, k_tail >> 3, k_tail >> 5, arow, srow);
    }
  }
}

std::once_flag g_attr_once;

}  // namespace

hipError_t launch_act_quant(const uint16_t* X, int64_t ld_x, int M, int K, int k_tail,
                            const float* inv_scale_pos, const int32_t* perm,
                            const int32_t* group_offsets, int G, uint8_t* Aq, uint8_t* Asc,
                            int num_cus, hipStream_t stream) {
  const bool grouped = group_offsets && G > 1;
  const int units = K >> 3;
  if (M <= 64) {
    // Few rows: spread the positions over workgroups, at most ~16 row chunks.
    const int rows_per_wg = std::max(1, (M + 15) / 16);
    const dim3 grid((units + kRowsThreads - 1) / kRowsThreads, (M + rows_per_wg - 1) / rows_per_wg);
    if (grouped)
      act_quant_rows_kernel<true><<<grid, kRowsThreads, 0, stream>>>(
          X, ld_x, M, K, k_tail, inv_scale_pos, perm, group_offsets, G, rows_per_wg, Aq, Asc);
    else
      act_quant_rows_kernel<false><<<grid, kRowsThreads, 0, stream>>>(
          X, ld_x, M, K, k_tail, inv_scale_pos, perm, nullptr, 1, rows_per_wg, Aq, Asc);
    return hipGetLastError();
  }
  const size_t lds = lds_kernel_bytes(K);
  // Raise the dynamic-LDS cap above the 64 KiB default once; a runtime that
  // does not need or know the attribute is left to the launch check below.
  std::call_once(g_attr_once, [] {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&act_quant_lds_kernel<false>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&act_quant_lds_kernel<true>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    (void)hipGetLastError();
  });
  // Two workgroups per CU when the LDS allows it; contiguous row ranges keep
  // a workgroup inside one expert for most of its rows.
  const int wgs_per_cu = lds * 2 <= 160 * 1024 ? 2 : 1;
  const int target = std::max(1, num_cus * wgs_per_cu);
  const int rows_per_wg = std::max(1, (M + target - 1) / target);
  const int grid = (M + rows_per_wg - 1) / rows_per_wg;
  if (grouped)
    act_quant_lds_kernel<true><<<grid, kLdsThreads, lds, stream>>>(
        X, ld_x, M, K, k_tail, inv_scale_pos, perm, group_offsets, G, rows_per_wg, Aq, Asc);
  else
    act_quant_lds_kernel<false><<<grid, kLdsThreads, lds, stream>>>(
        X, ld_x, M, K, k_tail, inv_scale_pos, perm, nullptr, 1, rows_per_wg, Aq, Asc);
  return hipGetLastError();
}

}  // namespace prq
