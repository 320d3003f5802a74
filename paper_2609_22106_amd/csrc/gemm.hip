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
// Two kernels, each with a grouped (MoE expert) mode in which rows
// [off[e], off[e+1]) multiply expert e's weight:
//   * gemm_tile   -- prefill shapes: 128x128 output tile per 256-thread
//                    workgroup, A/B/scale tiles staged in LDS (rows padded to
//                    80 bytes so the 16-byte lane reads of one MFMA operand hit
//                    distinct banks), 4 waves of 64x64 (4x4 MFMA tiles each).
//   * gemm_stream -- decode shapes (few rows per weight): the weight is the
//                    MFMA A operand (16 output features per tile) streamed
//                    from HBM straight into registers once, the activation rows
//                    are the B operand (16 rows per MFMA, up to 64 per pass);
//                    4 waves split the tile's K steps and reduce in LDS;
//                    optional split-K across workgroups with a deterministic
//                    last-arriver reduction (fixed summation order) through a
//                    caller-provided workspace.
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
    const int32_t* __restrict__ off, int E, const uint8_t* __restrict__ Wq,
    const uint8_t* __restrict__ Wsc, int N, int K_aug, float* __restrict__ Y) {
  __shared__ __align__(16) uint8_t sA[kTileM * kLdsRow];
  __shared__ __align__(16) uint8_t sB[kTileN * kLdsRow];
  __shared__ uint8_t sAs[kTileM * 4];
  __shared__ uint8_t sBs[kTileN * 4];

  int e = 0, row_begin, row_end;
  if (kGrouped) {
    if (!grouped_tile(off, E, M, blockIdx.y, kTileM, &e, &row_begin, &row_end)) return;
  } else {
    row_begin = blockIdx.y * kTileM;
    row_end = min(M, row_begin + kTileM);
  }
  const int n0 = blockIdx.x * kTileN;
  const int64_t row_bytes = K_aug >> 1;
  const int nb = K_aug >> 5;
  const uint8_t* We = Wq + static_cast<int64_t>(e) * N * row_bytes;
  const uint8_t* Wse = Wsc + static_cast<int64_t>(e) * N * nb;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int lr = lane & 15, lk = lane >> 4;

  v4f acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

  const int steps = (K_aug + kStepK - 1) / kStepK;
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
      const int n = n0 + r;
      const uint4 vb = load16_or_zero(We + n * row_bytes + s * kStepBytes + part * 16,
                                      kok && n < N);
      *reinterpret_cast<uint4*>(&sB[r * kLdsRow + part * 16]) = vb;
    }
    // Scales: 4 blocks per row per step.
    for (int c = tid; c < kTileM * 4; c += kTileThreads) {
      const int r = c >> 2, b = c & 3;
      const int blk = s * 4 + b;
      const int m = row_begin + r, n = n0 + r;
      sAs[c] = (blk < nb && m < row_end) ? Asc[static_cast<int64_t>(m) * nb + blk] : kNeutralScale;
      sBs[c] = (blk < nb && n < N) ? Wse[static_cast<int64_t>(n) * nb + blk] : kNeutralScale;
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

constexpr int kStreamThreads = 256;
constexpr int kStreamRows = 64;   // activation rows per pass (4 MFMA column groups)

template <bool kGrouped>
__global__ __launch_bounds__(kStreamThreads) void gemm_stream_kernel(
    const uint8_t* __restrict__ Aq, const uint8_t* __restrict__ Asc, int M,
    const int32_t* __restrict__ off, int E, const uint8_t* __restrict__ Wq,
    const uint8_t* __restrict__ Wsc, int N, int K_aug, float* __restrict__ Y, int splits,
    float* __restrict__ partial, uint32_t* __restrict__ counters) {
  __shared__ float s_red[4][4][64][4];   // [wave][column group][lane][q]
  __shared__ int s_last;

  const int tile = blockIdx.x;          // 16 output features
  const int split = blockIdx.y;
  const int e = kGrouped ? blockIdx.z : 0;
  const int row_begin = kGrouped ? min(max(off[e], 0), M) : 0;
  const int row_end = kGrouped ? min(max(off[e + 1], row_begin), M) : M;
  if (row_end <= row_begin) return;     // expert with no rows: its weight is not read

  const int64_t row_bytes = K_aug >> 1;
  const int nb = K_aug >> 5;
  const uint8_t* We = Wq + static_cast<int64_t>(e) * N * row_bytes;
  const uint8_t* Wse = Wsc + static_cast<int64_t>(e) * N * nb;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lk = lane >> 4;
  const int n_w = tile * 16 + lr;       // weight row this lane feeds
  const int steps = (K_aug + kStepK - 1) / kStepK;
  const int s_begin = static_cast<int>(static_cast<int64_t>(steps) * split / splits);
  const int s_end = static_cast<int>(static_cast<int64_t>(steps) * (split + 1) / splits);

  for (int pass_row = row_begin; pass_row < row_end; pass_row += kStreamRows) {
    const int rows = min(kStreamRows, row_end - pass_row);
    const int groups = (rows + 15) >> 4;
    v4f acc[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) acc[g] = v4f{0.f, 0.f, 0.f, 0.f};

    for (int s = s_begin + wave; s < s_end; s += 4) {
      const int kel = s * kStepK + lk * 32;
      const bool kok = kel < K_aug;
      const uint4 w = load16_or_zero(We + n_w * row_bytes + s * kStepBytes + lk * 16, kok);
      const uint32_t sw = kok ? Wse[static_cast<int64_t>(n_w) * nb + s * 4 + lk] : kNeutralScale;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        if (g < groups) {
          const int m = pass_row + g * 16 + lr;
          const bool ok = kok && m < row_end;
          const uint4 a = load16_or_zero(Aq + m * row_bytes + s * kStepBytes + lk * 16, ok);
          const uint32_t sa = ok ? Asc[static_cast<int64_t>(m) * nb + s * 4 + lk] : kNeutralScale;
          acc[g] = dev::mfma_fp4_16x16x128(w, a, sw, sa, acc[g]);
        }
      }
    }

    // Reduce the 4 waves in a fixed order.  acc[g][q] of this lane is
    // Y[pass_row + 16 g + lr][16 tile + 4 lk + q].
#pragma unroll
    for (int g = 0; g < 4; ++g)
#pragma unroll
      for (int q = 0; q < 4; ++q) s_red[wave][g][lane][q] = acc[g][q];
    __syncthreads();
    for (int idx = tid; idx < 4 * 64 * 4; idx += kStreamThreads) {
      const int g = idx >> 8, l = (idx >> 2) & 63, q = idx & 3;
      const int m = pass_row + g * 16 + (l & 15);
      const int n = tile * 16 + 4 * (l >> 4) + q;
      if (g < groups && m < row_end) {
        const float v = s_red[0][g][l][q] + s_red[1][g][l][q] + s_red[2][g][l][q] + s_red[3][g][l][q];
        if (splits == 1)
          Y[static_cast<int64_t>(m) * N + n] = v;
        else
          partial[(static_cast<int64_t>(split) * M + m) * N + n] = v;
      }
    }
    __syncthreads();
  }
  if (splits == 1) return;

  // Split-K: the last workgroup of this tile to arrive sums the partials in
  // split order 0, 1, ... (deterministic) and resets the counter for the next call.
  __threadfence();
  __syncthreads();
  uint32_t* ctr = counters + static_cast<int64_t>(e) * (N >> 4) + tile;
  if (tid == 0) s_last = (atomicAdd(ctr, 1u) == static_cast<uint32_t>(splits - 1));
  __syncthreads();
  if (!s_last) return;
  __threadfence();
  const int count = (row_end - row_begin) * 16;
  for (int idx = tid; idx < count; idx += kStreamThreads) {
    const int m = row_begin + (idx >> 4);
    const int n = tile * 16 + (idx & 15);
    float v = 0.f;
    for (int q = 0; q < splits; ++q) v += partial[(static_cast<int64_t>(q) * M + m) * N + n];
    Y[static_cast<int64_t>(m) * N + n] = v;
  }
  if (tid == 0) *ctr = 0u;
}

}  // namespace

hipError_t launch_gemm_tile(const uint8_t* Aq, const uint8_t* Asc, int M,
                            const int32_t* group_offsets, int E, const uint8_t* Wq,
                            const uint8_t* Wsc, int N, int K_aug, float* Y, hipStream_t stream) {
  const int nt = (N + kTileN - 1) / kTileN;
  if (group_offsets) {
    // Upper bound on the number of row tiles over all experts.
    const int mt = (M + kTileM - 1) / kTileM + E;
    gemm_tile_kernel<true><<<dim3(nt, mt), kTileThreads, 0, stream>>>(Aq, Asc, M, group_offsets, E,
                                                                    Wq, Wsc, N, K_aug, Y);
  } else {
    const int mt = (M + kTileM - 1) / kTileM;
    gemm_tile_kernel<false><<<dim3(nt, mt), kTileThreads, 0, stream>>>(Aq, Asc, M, nullptr, 1, Wq,
                                                                     Wsc, N, K_aug, Y);
  }
  return hipGetLastError();
}

size_t stream_workspace_bytes(int M, int E, int N, int splits) {
  if (splits <= 1) return 0;
  const size_t part = static_cast<size_t>(splits) * M * N * sizeof(float);
  const size_t ctr = static_cast<size_t>(E) * (N / 16) * sizeof(uint32_t);
  return ((part + 255) & ~static_cast<size_t>(255)) + ctr;
}

int choose_stream_splits(int M, int N, int K_aug, int num_cus) {
  const int tiles = N / 16;
  const int steps = (K_aug + kStepK - 1) / kStepK;
  // Enough workgroups to keep every CU streaming, but no split shorter than
  // one K step per wave, and fewer splits as the partials grow with M.
  int want = (4 * num_cus + tiles - 1) / tiles;
  if (M > 16) want = std::min(want, 4);
  return std::max(1, std::min({want, steps / 4 > 0 ? steps / 4 : 1, 64}));
}

int choose_variant(int M_per_group, int N, int K_aug) {
  (void)N;
  (void)K_aug;
  return M_per_group <= 64 ? PRQ_GEMM_STREAM : PRQ_GEMM_TILE;
}

hipError_t launch_gemm_stream(const uint8_t* Aq, const uint8_t* Asc, int M,
                              const int32_t* group_offsets, int E, const uint8_t* Wq,
                              const uint8_t* Wsc, int N, int K_aug, float* Y, int splits,
                              void* workspace, hipStream_t stream) {
  float* partial = nullptr;
  uint32_t* counters = nullptr;
  if (splits > 1) {
    const size_t part = static_cast<size_t>(splits) * M * N * sizeof(float);
    partial = static_cast<float*>(workspace);
    counters = reinterpret_cast<uint32_t*>(static_cast<char*>(workspace) +
                                           ((part + 255) & ~static_cast<size_t>(255)));
  }
  const int tiles = N / 16;
  if (group_offsets)
    gemm_stream_kernel<true><<<dim3(tiles, splits, E), kStreamThreads, 0, stream>>>(
        Aq, Asc, M, group_offsets, E, Wq, Wsc, N, K_aug, Y, splits, partial, counters);
  else
    gemm_stream_kernel<false><<<dim3(tiles, splits, 1), kStreamThreads, 0, stream>>>(
        Aq, Asc, M, nullptr, 1, Wq, Wsc, N, K_aug, Y, splits, partial, counters);
  return hipGetLastError();
}

}  // namespace prq
