// The augmented MXFP4 GEMM of arXiv 2609.22106 (Eq. 3): one block-scaled GEMM
// whose reduction runs over K_aug = K + k (main channels, then the k tail
// channels whose activation blocks were copied and whose weight side holds the
// MXFP4 residual of Eq. 2):
//
//   Y[m, n] = sum_b 2^(Asc[m,b]-127) 2^(Wsc[n,b]-127) sum_{i<32} A[m,32b+i] W[n,32b+i]
//
// computed on gfx950's v_mfma_scale_f32_16x16x128_f8f6f4 with FP4 operands and
// E8M0 scales fed straight into the instruction, float32 accumulation.
//
// This file: the LDS-tiled kernel for prefill shapes (the weight-streaming
// decode kernel is in gemm_stream.hip), with a grouped (MoE expert) mode in
// which rows [off[e], off[e+1]) multiply expert e's weight.  The weight comes
// in the packed layout of pack.hip (contiguous kilobyte per 16-row K step).  128x128 output
// tile per 256-thread workgroup, A/B/scale tiles staged in LDS (rows padded to
// 80 bytes so the 16-byte lane reads of one MFMA operand hit distinct banks),
// 4 waves of 64x64 (4x4 MFMA tiles each).
#include <hip/hip_runtime.h>

#include <algorithm>

#include "mx_device.hpp"
#include "prq.h"
#include "prq_internal.h"

namespace prq {
namespace {

using dev::v4f;

constexpr int kTileM = 128, kTileN = 128;
constexpr int kStepK = 128;           // elements per K step = 64 bytes per row
constexpr int kStepBytes = kStepK / 2;
constexpr int kLdsRow = kStepBytes + 16;  // padded LDS row (bytes)
constexpr int kTileThreads = 256;
constexpr uint8_t kNeutralScale = 127;   // scale paired with zero codes past K_aug

__device__ __forceinline__ uint4 load16_or_zero(const uint8_t* p, bool ok) {
  return ok ? *reinterpret_cast<const uint4*>(p) : make_uint4(0, 0, 0, 0);
}

// Row range [row_begin, row_end) and expert of row tile `mt` in the grouped
// layout, where tiles of `tile_rows` rows are numbered expert after expert.
// All threads of the (256-thread) workgroup call it; the per-expert tile
// counts are prefix-summed 256 experts at a time in LDS.  Returns false for
// an index beyond the last expert's last tile.
__device__ bool grouped_tile(const int32_t* __restrict__ off, int E, int M, int mt, int tile_rows,
                             int* e_out, int* row_begin, int* row_end) {
  __shared__ int s_scan[kTileThreads];
  __shared__ int s_hit[3];
  const int tid = threadIdx.x;
  if (tid == 0) s_hit[0] = -1;
  int base = 0;
  for (int e0 = 0; e0 < E; e0 += kTileThreads) {
    const int e = e0 + tid;
    int r0 = 0, r1 = 0, t = 0;
    if (e < E) {  // offsets clamped to [0, M]: malformed offsets cannot address past A
      r0 = min(max(off[e], 0), M);
      r1 = min(max(off[e + 1], r0), M);
      t = (r1 - r0 + tile_rows - 1) / tile_rows;
    }
    s_scan[tid] = t;
    __syncthreads();
    for (int d = 1; d < kTileThreads; d <<= 1) {  // inclusive Hillis-Steele scan
      const int v = tid >= d ? s_scan[tid - d] : 0;
      __syncthreads();
      s_scan[tid] += v;
      __syncthreads();
    }
    const int incl = base + s_scan[tid];
    const int excl = incl - t;
    if (e < E && mt >= excl && mt < incl) {
      s_hit[0] = e;
      s_hit[1] = r0 + (mt - excl) * tile_rows;
      s_hit[2] = min(r1, s_hit[1] + tile_rows);
    }
    base += s_scan[kTileThreads - 1];
    __syncthreads();
  }
  if (s_hit[0] < 0) return false;
  *e_out = s_hit[0];
  *row_begin = s_hit[1];
  *row_end = s_hit[2];
  return true;
}

template <bool kGrouped>
__global__ __launch_bounds__(kTileThreads) void gemm_tile_kernel(
    const uint8_t* __restrict__ Aq, const uint8_t* __restrict__ Asc, int M,
    const int32_t* __restrict__ off, int E, const uint8_t* __restrict__ Wp,
    const uint8_t* __restrict__ Wps, int N, int K_aug, float* __restrict__ Y) {
  __shared__ __align__(16) uint8_t sA[kTileM * kLdsRow];
  __shared__ __align__(16) uint8_t sB[kTileN * kLdsRow];
  __shared__ uint8_t sAs[kTileM * 4];
  __shared__ uint8_t sBs[kTileN * 4];

  int e = 0, row_begin, row_end;
  const int n0 = blockIdx.x * kTileN;
  if (kGrouped) {
    if (!grouped_tile(off, E, M, blockIdx.y, kTileM, &e, &row_begin, &row_end)) return;
  } else {
    row_begin = blockIdx.y * kTileM;
    row_end = min(M, row_begin + kTileM);
  }
  const int64_t row_bytes = K_aug >> 1;
  const int nb = K_aug >> 5;
  const int steps = (K_aug + kStepK - 1) / kStepK;
  const int sgroups = (steps + 3) >> 2;
  const int ntiles = N >> 4;
  const int t0 = n0 >> 4;   // first 16-feature tile of this workgroup
  const uint8_t* We = Wp + (static_cast<int64_t>(e) * ntiles + t0) * steps * 1024;
  const uint32_t* Wse =
      reinterpret_cast<const uint32_t*>(Wps) + (static_cast<int64_t>(e) * ntiles + t0) * sgroups * 64;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int lr = lane & 15, lk = lane >> 4;

  v4f acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

  for (int s = 0; s < steps; ++s) {
    // Stage A and B: 128 rows x 64 bytes each = 512 16-byte chunks per operand.
#pragma unroll
    for (int c = tid; c < kTileM * 4; c += kTileThreads) {
      const int r = c >> 2, part = c & 3;
      const bool kok = s * kStepK + part * 32 < K_aug;
      const int m = row_begin + r;
      const uint4 va = load16_or_zero(Aq + m * row_bytes + s * kStepBytes + part * 16,
                                      kok && m < row_end);
      *reinterpret_cast<uint4*>(&sA[r * kLdsRow + part * 16]) = va;
    }
    // B from the packed weight: chunk c = (tile nt, lane l) is the 16 bytes of
    // row 16 nt + l % 16, K part l / 16 of this step (zero past K_aug).
#pragma unroll
    for (int c = tid; c < kTileN * 4; c += kTileThreads) {
      const int nt = c >> 6, l = c & 63;
      const int r = nt * 16 + (l & 15), part = l >> 4;
      const uint4 vb = load16_or_zero(We + (static_cast<int64_t>(nt) * steps + s) * 1024 + l * 16,
                                      t0 + nt < ntiles);
      *reinterpret_cast<uint4*>(&sB[r * kLdsRow + part * 16]) = vb;
    }
    // Scales: 4 blocks per row per step; packed weight scales hold byte s % 4
    // of lane (b * 16 + r % 16)'s dword in group s / 4.
    for (int c = tid; c < kTileM * 4; c += kTileThreads) {
      const int r = c >> 2, b = c & 3;
      const int blk = s * 4 + b;
      const int m = row_begin + r;
      sAs[c] = (blk < nb && m < row_end) ? Asc[static_cast<int64_t>(m) * nb + blk] : kNeutralScale;
      const int nt = c >> 6, l = c & 63;
      const int rb = nt * 16 + (l & 15), bb = l >> 4;
      sBs[rb * 4 + bb] = t0 + nt < ntiles
          ? static_cast<uint8_t>(Wse[(static_cast<int64_t>(nt) * sgroups + (s >> 2)) * 64 + l] >> (8 * (s & 3)))
          : kNeutralScale;
    }
    __syncthreads();

    uint4 a[4], b[4];
    uint32_t sa[4], sb[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = wm * 64 + i * 16 + lr;
      a[i] = *reinterpret_cast<const uint4*>(&sA[r * kLdsRow + lk * 16]);
      sa[i] = sAs[r * 4 + lk];
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = wn * 64 + j * 16 + lr;
      b[j] = *reinterpret_cast<const uint4*>(&sB[r * kLdsRow + lk * 16]);
      sb[j] = sBs[r * 4 + lk];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = dev::mfma_fp4_16x16x128(a[i], b[j], sa[i], sb[j], acc[i][j]);
    __syncthreads();
  }

  // Lane holds C[4*lk + q][lr] of each 16x16 tile.
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int m = row_begin + wm * 64 + i * 16 + 4 * lk + q;
        const int n = n0 + wn * 64 + j * 16 + lr;
        if (m < row_end && n < N) Y[static_cast<int64_t>(m) * N + n] = acc[i][j][q];
      }
}

}  // namespace

hipError_t launch_gemm_tile(const uint8_t* Aq, const uint8_t* Asc, int M,
                            const int32_t* group_offsets, int E, const uint8_t* Wp,
                            const uint8_t* Wps, int N, int K_aug, float* Y, hipStream_t stream) {
  const int nt = (N + kTileN - 1) / kTileN;
  if (group_offsets) {
    // Upper bound on the number of row tiles over all experts.
    const int mt = (M + kTileM - 1) / kTileM + E;
    gemm_tile_kernel<true><<<dim3(nt, mt), kTileThreads, 0, stream>>>(Aq, Asc, M, group_offsets, E,
                                                                    Wp, Wps, N, K_aug, Y);
  } else {
    const int mt = (M + kTileM - 1) / kTileM;
    gemm_tile_kernel<false><<<dim3(nt, mt), kTileThreads, 0, stream>>>(Aq, Asc, M, nullptr, 1, Wp,
                                                                     Wps, N, K_aug, Y);
  }
  return hipGetLastError();
}

}  // namespace prq
