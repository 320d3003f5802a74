// Fused activation quantization with the online tail copy (arXiv 2609.22106,
// Sec. "Activation tail construction" and "Kernel design"; Algorithm 1,
// step 11):
//
//   Z~[m, p] = X[m, perm[p]] * inv_s[perm[p]]          (D^-1 P of Eq. 1, float32)
//   Aq/Asc   = MXFP4(Z~) and its k/32 tail blocks written once more after the
//              K/32 main blocks (== MXFP4([Z~, Z~_tail]) since the tail starts
//              on a block boundary)
//
// Memory-bound: per row it reads 2K bytes of bf16 and writes (K+k)/2 code bytes
// and (K+k)/32 scale bytes.  Layout of one workgroup (512 threads):
//   * the group's perm (as uint16) and the pre-gathered inverse scales
//     inv_s[perm[p]] live in LDS for all the rows the workgroup handles
//     (reloaded only when a row belongs to another expert);
//   * each row is staged into LDS with coalesced 16-byte loads, then every
//     thread gathers 8 consecutive positions (a quarter block) from LDS;
//   * the block max is reduced over the 4 lanes of a quad with DPP;
//   * each thread writes one 32-bit word of 8 packed nibbles (a wave writes
//     256 contiguous bytes); lane 0 of each quad writes the scale byte.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>

#include "mx_device.hpp"
#include "prq_internal.h"

namespace prq {
namespace {

constexpr int kAqThreads = 512;

__host__ __device__ inline size_t aq_lds_bytes(int K) {
  // perm (uint16) + inverse scales (float) + one staged bf16 row
  return static_cast<size_t>(K) * 2 + static_cast<size_t>(K) * 4 + static_cast<size_t>(K) * 2;
}

template <bool kGrouped>
__global__ __launch_bounds__(kAqThreads) void act_quant_kernel(
    const uint16_t* __restrict__ X, int64_t ld_x, int M, int K, int k_tail,
    const float* __restrict__ inv_scale, const int32_t* __restrict__ perm,
    const int32_t* __restrict__ offsets, int G, int rows_per_wg, uint8_t* __restrict__ Aq,
    uint8_t* __restrict__ Asc) {
  extern __shared__ __align__(16) unsigned char smem[];
  float* s_inv = reinterpret_cast<float*>(smem);                            // [K]
  uint16_t* s_row = reinterpret_cast<uint16_t*>(smem + static_cast<size_t>(K) * 4);  // [K]
  uint16_t* s_perm = s_row + K;                                             // [K]

  const int tid = threadIdx.x;
  const int r0 = blockIdx.x * rows_per_wg;
  const int r1 = min(M, r0 + rows_per_wg);
  const int units = K >> 3;                 // quarter blocks of 8 positions
  const int k_aug = K + k_tail;
  const int64_t row_bytes = k_aug >> 1;
  const int nb = k_aug >> 5;
  const int tail_unit0 = (K - k_tail) >> 3;
  const int copy_units = k_tail >> 3;
  const int copy_blocks = k_tail >> 5;

  int cur_g = -1;
  for (int r = r0; r < r1; ++r) {
    const int g = kGrouped ? dev::find_group(offsets, G, r) : 0;
    __syncthreads();  // the previous row's readers are done with s_row / s_perm
    if (g != cur_g) {
      const int32_t* pg = perm ? perm + static_cast<int64_t>(g) * K : nullptr;
      const float* ig = inv_scale ? inv_scale + static_cast<int64_t>(g) * K : nullptr;
      for (int p = tid; p < K; p += kAqThreads) {
        int src = pg ? pg[p] : p;
        src = static_cast<unsigned>(src) < static_cast<unsigned>(K) ? src : 0;  // never index past the row
        s_perm[p] = static_cast<uint16_t>(src);
        s_inv[p] = ig ? ig[src] : 1.0f;
      }
      cur_g = g;
    }
    const uint4* xr = reinterpret_cast<const uint4*>(X + static_cast<int64_t>(r) * ld_x);
    uint4* sr = reinterpret_cast<uint4*>(s_row);
    for (int i = tid; i < (K >> 3); i += kAqThreads) sr[i] = xr[i];
    __syncthreads();

    uint8_t* arow = Aq + static_cast<int64_t>(r) * row_bytes;
    uint8_t* srow = Asc + static_cast<int64_t>(r) * nb;
    for (int u = tid; u < units; u += kAqThreads) {
      float z[8];
      float amax = 0.0f;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int p = (u << 3) + j;
        const uint32_t h = s_row[s_perm[p]];
        z[j] = __uint_as_float(h << 16) * s_inv[p];
        amax = fmaxf(amax, fabsf(z[j]));
      }
      amax = dev::quad_max(amax);   // the 4 lanes of a quad hold one 32-block
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
  }
}

std::once_flag g_attr_once;

}  // namespace

hipError_t launch_act_quant(const uint16_t* X, int64_t ld_x, int M, int K, int k_tail,
                            const float* inv_scale, const int32_t* perm,
                            const int32_t* group_offsets, int G, uint8_t* Aq, uint8_t* Asc,
                            int num_cus, hipStream_t stream) {
  const size_t lds = aq_lds_bytes(K);
  // Raise the dynamic-LDS cap above the 64 KiB default once; a runtime that
  // does not need or know the attribute is left to the launch check below.
  std::call_once(g_attr_once, [] {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&act_quant_kernel<false>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&act_quant_kernel<true>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    (void)hipGetLastError();
  });
  // Two workgroups per CU when the LDS allows it; contiguous row ranges keep
  // a workgroup inside one expert for most of its rows.
  const int wgs_per_cu = lds * 2 <= 160 * 1024 ? 2 : 1;
  const int target = std::max(1, num_cus * wgs_per_cu);
  const int rows_per_wg = std::max(1, (M + target - 1) / target);
  const int grid = (M + rows_per_wg - 1) / rows_per_wg;
  if (group_offsets && G > 1)
    act_quant_kernel<true><<<grid, kAqThreads, lds, stream>>>(X, ld_x, M, K, k_tail, inv_scale, perm,
                                                            group_offsets, G, rows_per_wg, Aq, Asc);
  else
    act_quant_kernel<false><<<grid, kAqThreads, lds, stream>>>(X, ld_x, M, K, k_tail, inv_scale,
                                                             perm, nullptr, 1, rows_per_wg, Aq, Asc);
  return hipGetLastError();
}

}  // namespace prq
