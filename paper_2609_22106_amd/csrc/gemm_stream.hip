// Weight-streaming kernel of the augmented MXFP4 GEMM (arXiv 2609.22106,
// Eq. 3: one block-scaled GEMM over K_aug = K + k) for decode shapes, where
// few activation rows meet each weight row and the kernel is bound by
// reading W_aug once from HBM.
//
//   * The weight (in the packed layout of pack.hip) is the MFMA A operand: a
//     wave owns 16 output features (one tile) and a contiguous chunk of kU
//     128-element K steps, i.e. kU contiguous kilobytes of packed weight, and
//     issues every weight load of its chunk before its first MFMA, so a launch
//     has all of W_aug in flight.
//   * Activation rows are the MFMA B operand, 16 per MFMA, kG column groups
//     (16*kG rows) per pass; rows beyond the group's end load zeros.
//   * The waves of a workgroup are reduced through LDS in a fixed order.
//   * With splits > 1 the K range is split over workgroups; each adds its
//     partial tile into a float accumulator in the caller's workspace with
//     device-scope atomics whose results it waits for, then bumps the tile's
//     arrival counter; the last arriver swaps the accumulator back to zero
//     while reading it, writes Y and resets the counter, so the workspace is
//     all-zero between calls.  (With two splits the result is bitwise
//     deterministic since 0 + a + b = 0 + b + a in float.)
// Grouped (MoE) mode: blockIdx.z is the expert; experts without rows return
// before reading their weight.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "mx_device.hpp"
#include "prq.h"
#include "prq_internal.h"

namespace prq {
namespace {

using dev::v4f;

constexpr int kStepK = 128;
constexpr int kStepBytes = kStepK / 2;
constexpr uint32_t kNeutralScale = 127;

__device__ __forceinline__ uint4 ld16(const uint8_t* p, bool ok) {
  return ok ? *reinterpret_cast<const uint4*>(p) : make_uint4(0, 0, 0, 0);
}

template <bool kGrouped, int kWaves, int kU, int kG, int kT>
__global__ __launch_bounds__(kWaves * 64) void gemm_stream_kernel(
    const uint8_t* __restrict__ Aq, const uint8_t* __restrict__ Asc, int M,
    const int32_t* __restrict__ off, const uint8_t* __restrict__ Wp,
    const uint8_t* __restrict__ Wps, int N, int K_aug, float* __restrict__ Y, int splits,
    float* __restrict__ acc_ws, uint32_t* __restrict__ counters) {
  extern __shared__ float s_red[];   // [kWaves][kG][64][4]
  __shared__ int s_last;

  // Workgroup = kT 16-feature tiles x (kWaves / kT) K chunks; wave w works on
  // tile w % kT and chunk w / kT, so the kT waves of one chunk read the same
  // activation bytes (served by the CU's L1 after the first).
  const int split = blockIdx.y;
  const int e = kGrouped ? static_cast<int>(blockIdx.z) : 0;
  const int row_begin = kGrouped ? min(max(off[e], 0), M) : 0;
  const int row_end = kGrouped ? min(max(off[e + 1], row_begin), M) : M;
  if (row_end <= row_begin) return;

  const int64_t row_bytes = K_aug >> 1;
  const int nb = K_aug >> 5;
  const int steps = (K_aug + kStepK - 1) / kStepK;
  const int sgroups = (steps + 3) >> 2;
  const int ntiles = N >> 4;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lk = lane >> 4;
  const int tile = blockIdx.x * kT + wave % kT;
  const bool tile_ok = tile < ntiles;
  const int s_begin = steps * split / splits;        // steps * splits < 2^31
  const int s_end = steps * (split + 1) / splits;
  const int s0 = s_begin + (wave / kT) * kU;
  // Packed weight blocks of this tile: one contiguous kilobyte per K step.
  const int64_t et = static_cast<int64_t>(e) * ntiles + (tile_ok ? tile : 0);
  const uint8_t* Wt = Wp + et * steps * 1024 + lane * 16;
  const uint32_t* Wst = reinterpret_cast<const uint32_t*>(Wps) + et * sgroups * 64 + lane;

  // The wave's whole weight chunk, loaded before any MFMA.
  uint4 w[kU];
  uint32_t sw[kU];
  bool kok[kU];
#pragma unroll
  for (int j = 0; j < kU; ++j) {
    const int s = s0 + j;
    kok[j] = tile_ok && s < s_end;
    w[j] = ld16(Wt + static_cast<int64_t>(s) * 1024, kok[j]);
  }
#pragma unroll
  for (int j = 0; j < kU; ++j) {
    const int s = s0 + j;
    sw[j] = kok[j] ? (Wst[(s >> 2) * 64] >> (8 * (s & 3))) & 0xFFu : kNeutralScale;
  }

  for (int pass_row = row_begin; pass_row < row_end; pass_row += 16 * kG) {
    uint4 a[kU][kG];
    uint32_t sa[kU][kG];
#pragma unroll
    for (int j = 0; j < kU; ++j)
#pragma unroll
      for (int g = 0; g < kG; ++g) {
        const int m = pass_row + g * 16 + lr;
        const bool ok = kok[j] && m < row_end && (s0 + j) * kStepK + lk * 32 < K_aug;
        a[j][g] = ld16(Aq + m * row_bytes + (s0 + j) * kStepBytes + lk * 16, ok);
        sa[j][g] = ok ? Asc[static_cast<int64_t>(m) * nb + (s0 + j) * 4 + lk] : kNeutralScale;
      }
    v4f acc[kG];
#pragma unroll
    for (int g = 0; g < kG; ++g) acc[g] = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < kU; ++j)
#pragma unroll
      for (int g = 0; g < kG; ++g)
        acc[g] = dev::mfma_fp4_16x16x128(w[j], a[j][g], sw[j], sa[j][g], acc[g]);

    // acc[g][q] of this lane is Y[pass_row + 16 g + lr][16 tile + 4 lk + q].
#pragma unroll
    for (int g = 0; g < kG; ++g)
#pragma unroll
      for (int q = 0; q < 4; ++q) s_red[((wave * kG + g) * 64 + lane) * 4 + q] = acc[g][q];  // wave = c*kT + t
    __syncthreads();
    for (int idx = tid; idx < kT * kG * 256; idx += kWaves * 64) {
      const int t = idx / (kG * 256), r = idx % (kG * 256);
      const int g = r >> 8, l = (r >> 2) & 63, q = r & 3;
      const int m = pass_row + g * 16 + (l & 15);
      const int out_tile = blockIdx.x * kT + t;
      if (m < row_end && out_tile < (N >> 4)) {
        float v = 0.0f;
#pragma unroll
        for (int c = 0; c < kWaves / kT; ++c) v += s_red[(((c * kT + t) * kG + g) * 64 + l) * 4 + q];
        const int64_t o = static_cast<int64_t>(m) * N + out_tile * 16 + 4 * (l >> 4) + q;
        if (splits == 1)
          Y[o] = v;
        else
          atomicAdd(&acc_ws[o], v);
      }
    }
    __syncthreads();
  }
  if (splits == 1) return;

  // Every accumulator atomic of this workgroup is complete (vmcnt drained)
  // before the arrival counter moves.
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  uint32_t* ctr = counters + static_cast<int64_t>(e) * (N >> 4) + blockIdx.x;
  if (tid == 0) s_last = atomicAdd(ctr, 1u) == static_cast<uint32_t>(splits - 1);
  __syncthreads();
  if (!s_last) return;
  const int cols = min(16 * kT, N - static_cast<int>(blockIdx.x) * 16 * kT);
  const int count = (row_end - row_begin) * cols;
  for (int idx = tid; idx < count; idx += kWaves * 64) {
    const int64_t o = static_cast<int64_t>(row_begin + idx / cols) * N +
                      static_cast<int64_t>(blockIdx.x) * 16 * kT + idx % cols;
    Y[o] = atomicExch(&acc_ws[o], 0.0f);
  }
  if (tid == 0) atomicExch(ctr, 0u);
}

#define PRQ_STREAM_ARGS grid, Aq, Asc, M, off, Wp, Wps, N, K_aug, Y, splits, acc, ctr, stream
#define PRQ_STREAM_PARAMS                                                                    \
  dim3 grid, const uint8_t *Aq, const uint8_t *Asc, int M, const int32_t *off,             \
      const uint8_t *Wp, const uint8_t *Wps, int N, int K_aug, float *Y, int splits,        \
      float *acc, uint32_t *ctr, hipStream_t stream

template <bool kGrouped, int kWaves, int kU, int kG, int kT>
hipError_t launch_cfg(PRQ_STREAM_PARAMS) {
  const size_t lds = static_cast<size_t>(kWaves) * kG * 64 * 4 * sizeof(float);
  gemm_stream_kernel<kGrouped, kWaves, kU, kG, kT><<<grid, kWaves * 64, lds, stream>>>(
      Aq, Asc, M, off, Wp, Wps, N, K_aug, Y, splits, acc, ctr);
  return hipGetLastError();
}

template <bool kGrouped, int kWaves, int kU, int kG>
hipError_t launch_t(int T, PRQ_STREAM_PARAMS) {
  if (!kGrouped && T == 4 && kWaves >= 4) return launch_cfg<kGrouped, kWaves, kU, kG, 4>(PRQ_STREAM_ARGS);
  return launch_cfg<kGrouped, kWaves, kU, kG, 1>(PRQ_STREAM_ARGS);
}

template <bool kGrouped, int kWaves, int kU>
hipError_t launch_g(int G, int T, PRQ_STREAM_PARAMS) {
  switch (G) {
    case 1: return launch_t<kGrouped, kWaves, kU, 1>(T, PRQ_STREAM_ARGS);
    case 2: return launch_t<kGrouped, kWaves, kU, 2>(T, PRQ_STREAM_ARGS);
    default: return launch_t<kGrouped, kWaves, kU, 4>(T, PRQ_STREAM_ARGS);
  }
}

template <bool kGrouped, int kWaves>
hipError_t launch_u(int U, int G, int T, PRQ_STREAM_PARAMS) {
  switch (U) {
    case 1: return launch_g<kGrouped, kWaves, 1>(G, T, PRQ_STREAM_ARGS);
    case 2: return launch_g<kGrouped, kWaves, 2>(G, T, PRQ_STREAM_ARGS);
    case 3: return launch_g<kGrouped, kWaves, 3>(G, T, PRQ_STREAM_ARGS);
    case 4: return launch_g<kGrouped, kWaves, 4>(G, T, PRQ_STREAM_ARGS);
    case 6: return launch_g<kGrouped, kWaves, 6>(G, T, PRQ_STREAM_ARGS);
    default: return launch_g<kGrouped, kWaves, 8>(G, T, PRQ_STREAM_ARGS);
  }
}

}  // namespace

StreamConfig choose_stream_config(int M_per_group, int N, int K_aug, int grouped, int num_cus) {
  StreamConfig c;
  const int steps = (K_aug + kStepK - 1) / kStepK;
  const int rows = std::min(std::max(M_per_group, 1), 64);
  c.groups = rows <= 16 ? 1 : (rows <= 32 ? 2 : 4);
  const int tiles = N / 16;
  if (grouped) {  // many (expert, tile) workgroups already: no split-K
    c.splits = 1;
    c.waves = steps <= 32 ? 4 : 16;
    c.unroll = (steps + c.waves - 1) / c.waves;
    if (c.unroll > 8) c.ok = false;
  } else {
    // Enough workgroups to cover every CU; one wave per unrolled chunk.
    c.splits = tiles >= num_cus ? 1 : (c.groups == 1 ? 1 : 2);
    const int per_split = (steps + c.splits - 1) / c.splits;
    c.waves = 16;
    c.unroll = (per_split + c.waves - 1) / c.waves;
    while (c.unroll > 8) {
      c.splits *= 2;
      c.unroll = ((steps + c.splits - 1) / c.splits + c.waves - 1) / c.waves;
    }
  }
  static const int kU[] = {1, 2, 3, 4, 6, 8};
  for (int u : kU)
    if (u >= c.unroll) {
      c.unroll = u;
      break;
    }
  (void)num_cus;
  return c;
}

bool stream_config_covers(const StreamConfig& c, int K_aug) {
  const int steps = (K_aug + kStepK - 1) / kStepK;
  const bool shape = (c.waves == 4 || c.waves == 8 || c.waves == 16) &&
                     (c.unroll == 1 || c.unroll == 2 || c.unroll == 3 || c.unroll == 4 ||
                      c.unroll == 6 || c.unroll == 8) &&
                     (c.groups == 1 || c.groups == 2 || c.groups == 4) && c.splits >= 1 &&
                     c.splits <= steps;
  const bool tiles_ok = c.tiles == 1 || (c.tiles == 4 && c.waves >= 4);
  return shape && tiles_ok &&
         static_cast<int64_t>(c.waves / c.tiles) * c.unroll >= (steps + c.splits - 1) / c.splits;
}

int choose_variant(int M_per_group, int N, int K_aug) {
  (void)N;
  (void)K_aug;
  return M_per_group <= 64 ? PRQ_GEMM_STREAM : PRQ_GEMM_TILE;
}

size_t stream_workspace_bytes(int M, int E, int N, int splits) {
  if (splits <= 1) return 0;
  const size_t acc = (static_cast<size_t>(M) * N * sizeof(float) + 255) & ~static_cast<size_t>(255);
  return acc + static_cast<size_t>(E) * (N / 16) * sizeof(uint32_t);
}

hipError_t launch_gemm_stream(const uint8_t* Aq, const uint8_t* Asc, int M,
                              const int32_t* group_offsets, int E, const uint8_t* Wp,
                              const uint8_t* Wps, int N, int K_aug, float* Y,
                              const StreamConfig& cfg, void* workspace, hipStream_t stream) {
  float* acc = nullptr;
  uint32_t* ctr = nullptr;
  if (cfg.splits > 1) {
    acc = static_cast<float*>(workspace);
    const size_t a = (static_cast<size_t>(M) * N * sizeof(float) + 255) & ~static_cast<size_t>(255);
    ctr = reinterpret_cast<uint32_t*>(static_cast<char*>(workspace) + a);
  }
  const int T = group_offsets ? 1 : cfg.tiles;
  const dim3 grid((N / 16 + T - 1) / T, cfg.splits, group_offsets ? E : 1);
  const int U = cfg.unroll, G = cfg.groups;
  const int32_t* off = group_offsets;
  const int splits = cfg.splits;
  if (group_offsets) {
    switch (cfg.waves) {
      case 4: return launch_u<true, 4>(U, G, 1, PRQ_STREAM_ARGS);
      case 8: return launch_u<true, 8>(U, G, 1, PRQ_STREAM_ARGS);
      default: return launch_u<true, 16>(U, G, 1, PRQ_STREAM_ARGS);
    }
  }
  switch (cfg.waves) {
    case 4: return launch_u<false, 4>(U, G, T, PRQ_STREAM_ARGS);
    case 8: return launch_u<false, 8>(U, G, T, PRQ_STREAM_ARGS);
    default: return launch_u<false, 16>(U, G, T, PRQ_STREAM_ARGS);
  }
}

}  // namespace prq
