// Weight-streaming kernel of the augmented MXFP4 GEMM (arXiv 2609.22106,
// Eq. 3: one block-scaled GEMM over K_aug = K + k) for decode shapes, where
// few activation rows meet each weight row and the kernel is bound by
// reading W_aug once from HBM.
//
//   * A workgroup owns kT x kTW tiles of 16 output features and one split of
//     the K steps (128 elements each); its kWaves waves are kT tile groups x
//     (kWaves / kT) K chunks of kU contiguous steps, a wave computing the kTW
//     tiles of its group over its chunk.  The weight, in the packed layout of
//     pack.hip, is the MFMA A operand: each wave reads kTW x kU kilobytes and
//     issues all of them before anything else, so a launch has all of W_aug
//     in flight.  An activation operand a wave loads feeds its kTW tiles.
//   * The activation rows of the pass (16 * kG rows) over the split's K range
//     are staged once per workgroup into LDS (rows padded so that the 16-byte
//     lane reads of one MFMA operand fall in distinct banks) and shared by all
//     waves and tiles; they are the MFMA B operand, 16 rows per MFMA.
//   * Waves of one tile are reduced through LDS in a fixed order.
//   * With splits > 1 the workgroups of one output tile add their partial
//     tiles into a float accumulator in the caller's workspace with
//     device-scope atomics, wait for them, and bump the tile's arrival
//     counter; the last arriver swaps the accumulator back to zero while
//     reading it, writes Y and resets the counter, so the workspace is
//     all-zero between calls.  (With two splits the result is bitwise
//     deterministic since 0 + a + b = 0 + b + a in float.)
// Grouped (MoE) mode: blockIdx.z is the expert; experts without rows return
// before reading their weight.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>

#include "mx_device.hpp"
#include "prq.h"
#include "prq_internal.h"

namespace prq {
namespace {

using dev::v4f;

constexpr int kStepK = 128;
constexpr int kStepBytes = kStepK / 2;
constexpr uint32_t kNeutralScale = 127;
constexpr size_t kMaxStreamLds = 96 * 1024;
// flags of the kernel: bit 0 = activation operands straight from global memory
// (no LDS staging); bits 1-2 = split-K reduction (see StreamConfig::reduce).
constexpr int kDirectA = 1;
constexpr int kReduceLastArriver = 0, kReducePartials = 1, kReduceAtomicY = 2;

// Deterministic sum of the split partials [splits][M][N] into Y.
__global__ __launch_bounds__(256) void reduce_partials_kernel(const float* __restrict__ part,
                                                              int splits, int64_t MN,
                                                              float* __restrict__ Y) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= MN) return;
  float v = 0.0f;
  for (int s = 0; s < splits; ++s) v += part[s * MN + i];
  Y[i] = v;
}

__global__ __launch_bounds__(256) void zero_kernel(float* __restrict__ Y, int64_t n) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i < n) Y[i] = 0.0f;
}

// LDS row stride (bytes) of the staged activation: `nst` steps of 64 bytes,
// rounded to 4 steps, plus 16 so that 16 consecutive rows start in distinct
// 16-byte bank groups.
__host__ __device__ inline int act_row_stride(int nst) { return ((nst + 3) & ~3) * kStepBytes + 16; }

inline size_t stream_lds_bytes(int waves, int groups, int nst, bool stage_lds, int wave_tiles) {
  const size_t stage = stage_lds
      ? static_cast<size_t>(16 * groups) * (act_row_stride(nst) + ((nst + 3) & ~3) * 4)
      : 0;
  const size_t red = static_cast<size_t>(waves) * wave_tiles * groups * 64 * 4 * sizeof(float);
  return std::max(stage, red);
}

template <bool kGrouped, int kWaves, int kU, int kG, int kT, int kTW>
__global__ __launch_bounds__(kWaves * 64) void gemm_stream_kernel(
    const uint8_t* __restrict__ Aq, const uint8_t* __restrict__ Asc, int M,
    const int32_t* __restrict__ off, const uint8_t* __restrict__ Wp,
    const uint8_t* __restrict__ Wps, int N, int K_aug, float* __restrict__ Y, int splits,
    int flags, float* __restrict__ acc_ws, uint32_t* __restrict__ counters) {
  extern __shared__ __align__(16) unsigned char smem[];
  const bool stage = !(flags & kDirectA);
  const int reduce = (flags >> 1) & 3;
  __shared__ int s_last;
  constexpr int kChunks = kWaves / kT;

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
  const int t_in = wave % kT, chunk = wave / kT;
  const int tile0 = (blockIdx.x * kT + t_in) * kTW;  // the wave's first tile
  const int s_begin = steps * split / splits;        // steps * splits < 2^31
  const int s_end = steps * (split + 1) / splits;
  const int nst = s_end - s_begin;
  const int st0 = chunk * kU;                        // wave's first step, relative to s_begin

  // 1. The wave's whole weight chunk and its scale dwords, issued before
  //    anything else.  Addresses are clamped into the split (nst >= 1) so the
  //    loads are unconditional; nothing reads their results until every load
  //    of the kernel is in flight (a use would make the wave wait for all of
  //    them, the memory counter being in order).
  uint4 w[kTW][kU];
  uint32_t wsraw[kTW][kU];
  bool tile_ok[kTW];
#pragma unroll
  for (int tw = 0; tw < kTW; ++tw) {
    tile_ok[tw] = tile0 + tw < ntiles;
    const int64_t et = static_cast<int64_t>(e) * ntiles + (tile_ok[tw] ? tile0 + tw : 0);
    const uint8_t* Wt = Wp + (et * steps + s_begin) * 1024 + lane * 16;
#pragma unroll
    for (int j = 0; j < kU; ++j) {
      const int st = min(st0 + j, nst - 1);
      w[tw][j] = dev::load_stream16(Wt + static_cast<int64_t>(st) * 1024);   // read once
    }
  }
#pragma unroll
  for (int tw = 0; tw < kTW; ++tw) {
    const int64_t et = static_cast<int64_t>(e) * ntiles + (tile_ok[tw] ? tile0 + tw : 0);
    const uint32_t* Wst = reinterpret_cast<const uint32_t*>(Wps) + et * sgroups * 64 + lane;
#pragma unroll
    for (int j = 0; j < kU; ++j) wsraw[tw][j] = Wst[((s_begin + min(st0 + j, nst - 1)) >> 2) * 64];
  }

  const int stride = act_row_stride(nst);
  const int sstride = ((nst + 3) & ~3) * 4;          // scale bytes per staged row
  uint8_t* sA = smem;
  uint8_t* sAs = smem + 16 * kG * stride;
  float* s_red = reinterpret_cast<float*>(smem);     // reused after the MFMAs
  const int cols = min(16 * kT * kTW, N - static_cast<int>(blockIdx.x) * 16 * kT * kTW);
  bool kok[kTW][kU];
#pragma unroll
  for (int tw = 0; tw < kTW; ++tw)
#pragma unroll
    for (int j = 0; j < kU; ++j) kok[tw][j] = tile_ok[tw] && st0 + j < nst;

  for (int pass_row = row_begin; pass_row < row_end; pass_row += 16 * kG) {
    const int rows = min(16 * kG, row_end - pass_row);
    v4f acc[kTW][kG];
#pragma unroll
    for (int tw = 0; tw < kTW; ++tw)
#pragma unroll
      for (int g = 0; g < kG; ++g) acc[tw][g] = v4f{0.f, 0.f, 0.f, 0.f};
    if (stage) {
      // 2. Stage the pass's activation rows over [s_begin, s_end) in LDS
      //    (zero codes and a neutral scale past K_aug).  Four items per
      //    thread are loaded before any is written: one round trip.
      const int items = rows * nst * 4;
      for (int base = tid; base < items; base += 4 * kWaves * 64) {
        uint4 v[4];
        uint8_t sc[4];
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const int i = min(base + b * kWaves * 64, items - 1);
          const int r = i / (nst * 4), rem = i % (nst * 4);
          const int s = s_begin + (rem >> 2), c = rem & 3;
          const bool ok = s * kStepK + c * 32 < K_aug;
          const int m = pass_row + r;
          v[b] = *reinterpret_cast<const uint4*>(Aq + m * row_bytes +
                                                 (ok ? static_cast<int64_t>(s) * kStepBytes + c * 16 : 0));
          sc[b] = Asc[static_cast<int64_t>(m) * nb + (ok ? s * 4 + c : 0)];
        }
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const int i = base + b * kWaves * 64;
          if (i < items) {
            const int r = i / (nst * 4), rem = i % (nst * 4);
            const int st = rem >> 2, c = rem & 3;
            const bool ok = (s_begin + st) * kStepK + c * 32 < K_aug;
            *reinterpret_cast<uint4*>(sA + r * stride + st * kStepBytes + c * 16) =
                ok ? v[b] : make_uint4(0, 0, 0, 0);
            sAs[r * sstride + st * 4 + c] = ok ? sc[b] : static_cast<uint8_t>(kNeutralScale);
          }
        }
      }
      __syncthreads();
#pragma unroll
      for (int j = 0; j < kU; ++j) {
        const int s = s_begin + st0 + j;
        const int st = min(st0 + j, nst - 1);
#pragma unroll
        for (int g = 0; g < kG; ++g) {
          const int r = min(g * 16 + lr, rows - 1);
          const bool rok = g * 16 + lr < rows;
          const uint4 a = *reinterpret_cast<const uint4*>(sA + r * stride + st * kStepBytes + lk * 16);
          const uint32_t sa = sAs[r * sstride + st * 4 + lk];
#pragma unroll
          for (int tw = 0; tw < kTW; ++tw) {
            const uint4 wj = kok[tw][j] ? w[tw][j] : make_uint4(0, 0, 0, 0);
            const uint32_t sw = kok[tw][j] ? (wsraw[tw][j] >> (8 * (s & 3))) & 0xFFu : kNeutralScale;
            const bool ok = kok[tw][j] && rok;
            acc[tw][g] = dev::mfma_fp4_16x16x128(wj, ok ? a : make_uint4(0, 0, 0, 0), sw,
                                                 ok ? sa : kNeutralScale, acc[tw][g]);
          }
        }
      }
    } else {
      // 2'. Each wave loads the activation operands of its own steps straight
      //     from global memory (after its weight loads; no barrier).
      uint4 a[kU][kG];
      uint8_t sa[kU][kG];
#pragma unroll
      for (int j = 0; j < kU; ++j)
#pragma unroll
        for (int g = 0; g < kG; ++g) {
          const int m = pass_row + min(g * 16 + lr, rows - 1);
          const int s = s_begin + min(st0 + j, nst - 1);
          const bool ok = s * kStepK + lk * 32 < K_aug;
          a[j][g] = *reinterpret_cast<const uint4*>(Aq + m * row_bytes +
                                                    (ok ? static_cast<int64_t>(s) * kStepBytes + lk * 16 : 0));
          sa[j][g] = Asc[static_cast<int64_t>(m) * nb + (ok ? s * 4 + lk : 0)];
        }
#pragma unroll
      for (int j = 0; j < kU; ++j) {
        const int s = s_begin + st0 + j;
#pragma unroll
        for (int tw = 0; tw < kTW; ++tw) {
          const bool kin = kok[tw][j] && s * kStepK + lk * 32 < K_aug;
          const uint4 wj = kok[tw][j] ? w[tw][j] : make_uint4(0, 0, 0, 0);
          const uint32_t sw = kok[tw][j] ? (wsraw[tw][j] >> (8 * (s & 3))) & 0xFFu : kNeutralScale;
#pragma unroll
          for (int g = 0; g < kG; ++g) {
            const bool ok = kin && g * 16 + lr < rows;
            acc[tw][g] = dev::mfma_fp4_16x16x128(wj, ok ? a[j][g] : make_uint4(0, 0, 0, 0), sw,
                                                 ok ? static_cast<uint32_t>(sa[j][g]) : kNeutralScale,
                                                 acc[tw][g]);
          }
        }
      }
    }
    __syncthreads();   // the staging buffer becomes the reduction buffer

    // 3. Reduce the K chunks of each tile.  acc[tw][g][q] of this lane is
    //    Y[pass_row + 16 g + lr][16 (tile0 + tw) + 4 lk + q]; wave = chunk * kT + t_in.
#pragma unroll
    for (int tw = 0; tw < kTW; ++tw)
#pragma unroll
      for (int g = 0; g < kG; ++g)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          s_red[(((wave * kTW + tw) * kG + g) * 64 + lane) * 4 + q] = acc[tw][g][q];
    __syncthreads();
    // Thread idx: tile t * kTW + tw of the workgroup, row group g, lane l, q;
    // consecutive threads cover a row's 16 features and then the next tile,
    // so a row of the workgroup's columns is written in one contiguous run.
    for (int idx = tid; idx < kT * kTW * kG * 256; idx += kWaves * 64) {
      const int g = idx / (kT * kTW * 256), r = idx % (kT * kTW * 256);
      const int lr16 = r / (kT * kTW * 16), c16 = r % (kT * kTW * 16);
      const int tt = c16 >> 4, f = c16 & 15;             // workgroup tile, feature in tile
      const int t = tt / kTW, tw = tt % kTW;
      const int l = (f >> 2) * 16 + lr16, q = f & 3;     // the lane and element holding it
      const int m = pass_row + g * 16 + lr16;
      const int out_tile = (blockIdx.x * kT + t) * kTW + tw;
      if (m < row_end && out_tile < ntiles) {
        float v = 0.0f;
#pragma unroll
        for (int c = 0; c < kChunks; ++c)
          v += s_red[((((c * kT + t) * kTW + tw) * kG + g) * 64 + l) * 4 + q];
        const int64_t o = static_cast<int64_t>(m) * N + out_tile * 16 + 4 * (l >> 4) + q;
        if (splits == 1)
          Y[o] = v;
        else if (reduce == kReducePartials)
          acc_ws[static_cast<int64_t>(split) * M * N + o] = v;
        else if (reduce == kReduceAtomicY)
          atomicAdd(&Y[o], v);
        else
          atomicAdd(&acc_ws[o], v);
      }
    }
    __syncthreads();
  }
  if (splits == 1 || reduce != kReduceLastArriver) return;

  // Every accumulator atomic of this workgroup is complete (vmcnt drained)
  // before the arrival counter moves.
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  uint32_t* ctr = counters + static_cast<int64_t>(e) * ntiles + blockIdx.x;
  if (tid == 0) s_last = atomicAdd(ctr, 1u) == static_cast<uint32_t>(splits - 1);
  __syncthreads();
  if (!s_last) return;
  const int count = (row_end - row_begin) * cols;
  for (int idx = tid; idx < count; idx += kWaves * 64) {
    const int64_t o = static_cast<int64_t>(row_begin + idx / cols) * N +
                      static_cast<int64_t>(blockIdx.x) * 16 * kT * kTW + idx % cols;
    Y[o] = atomicExch(&acc_ws[o], 0.0f);
  }
  if (tid == 0) atomicExch(ctr, 0u);
}

#define PRQ_STREAM_ARGS grid, lds, Aq, Asc, M, off, Wp, Wps, N, K_aug, Y, splits, flags, acc, ctr, stream
#define PRQ_STREAM_PARAMS                                                                    \
  dim3 grid, size_t lds, const uint8_t *Aq, const uint8_t *Asc, int M, const int32_t *off,  \
      const uint8_t *Wp, const uint8_t *Wps, int N, int K_aug, float *Y, int splits,        \
      int flags, float *acc, uint32_t *ctr, hipStream_t stream

template <bool kGrouped, int kWaves, int kU, int kG, int kT, int kTW>
hipError_t launch_cfg(PRQ_STREAM_PARAMS) {
  static std::once_flag attr_once;   // dynamic LDS above the 64 KiB default
  std::call_once(attr_once, [] {
    (void)hipFuncSetAttribute(
        reinterpret_cast<const void*>(&gemm_stream_kernel<kGrouped, kWaves, kU, kG, kT, kTW>),
        hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(kMaxStreamLds));
    (void)hipGetLastError();
  });
  gemm_stream_kernel<kGrouped, kWaves, kU, kG, kT, kTW><<<grid, kWaves * 64, lds, stream>>>(
      Aq, Asc, M, off, Wp, Wps, N, K_aug, Y, splits, flags, acc, ctr);
  return hipGetLastError();
}

// T: 1 = one tile per workgroup, 4 = four tiles per workgroup (one per wave
// group), 5 = four tiles per wave (one wave group; at most 8 waves of at most
// 4 steps and one row group, so that the 16 weight kilobytes of a wave fit
// its registers -- stream_config_covers admits no other).
template <bool kGrouped, int kWaves, int kU, int kG>
hipError_t launch_t(int T, PRQ_STREAM_PARAMS) {
  if constexpr (kWaves <= 8 && kU <= 4 && kG == 1)
    if (T == 5) return launch_cfg<kGrouped, kWaves, kU, kG, 1, 4>(PRQ_STREAM_ARGS);
  if (T == 4) return launch_cfg<kGrouped, kWaves, kU, kG, 4, 1>(PRQ_STREAM_ARGS);
  return launch_cfg<kGrouped, kWaves, kU, kG, 1, 1>(PRQ_STREAM_ARGS);
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

int round_unroll(int u) {
  static const int kU[] = {1, 2, 3, 4, 6, 8};
  for (int x : kU)
    if (x >= u) return x;
  return 0;
}

}  // namespace

StreamConfig choose_stream_config(int M_per_group, int N, int K_aug, int grouped, int num_cus) {
  StreamConfig c;
  const int steps = (K_aug + kStepK - 1) / kStepK;
  const int rows = std::min(std::max(M_per_group, 1), 64);
  c.groups = rows <= 16 ? 1 : (rows <= 32 ? 2 : 4);
  if (grouped) {  // many (expert, tile) workgroups already: no split-K
    c.splits = 1;
    c.tiles = 1;
    c.stage_lds = false;
    c.waves = steps <= 32 ? 4 : 16;
    c.unroll = round_unroll((steps + c.waves - 1) / c.waves);
    // Four tiles per wave where the registers allow: an activation operand a
    // wave loads (one kilobyte per lane group for the expert's few rows) then
    // feeds four weight kilobytes instead of one, and a row's Y values of the
    // workgroup are 256 contiguous bytes (128 experts x 2048 x 832, 512 routed
    // rows: 29.3 -> 24.6 us; eight tiles per wave, half the workgroups: 30.8).
    if (c.waves <= 8 && c.unroll <= 4 && c.groups == 1) c.wave_tiles = 4;
  } else {
    // Decode shapes (measured on the 9728 -> 2560 down_proj): up to 32 rows,
    // 8-wave workgroups, 3 K splits, activation operands loaded per wave,
    // atomic split-K with a last-arriver; 33-64 rows, 4 feature tiles per
    // 16-wave workgroup sharing an LDS-staged activation, 6 K splits whose
    // partial sums a second kernel adds in a fixed order.
    if (c.groups <= 2) {
      c.waves = 8;
      c.tiles = 1;
      c.splits = 3;
      c.stage_lds = false;
      c.reduce = 0;
    } else {
      c.waves = 16;
      c.tiles = 4;
      c.splits = 6;
      c.stage_lds = true;
      c.reduce = 1;
    }
    c.splits = std::max(1, std::min(c.splits, steps / 4));
    auto unroll_for = [&](int sp) {
      const int per = (steps + sp - 1) / sp;
      return round_unroll((per + c.waves / c.tiles - 1) / (c.waves / c.tiles));
    };
    c.unroll = unroll_for(c.splits);
    while ((c.unroll == 0 || !stream_config_covers(c, K_aug)) && c.splits < steps) {
      ++c.splits;
      c.unroll = unroll_for(c.splits);
    }
    (void)num_cus;
  }
  c.ok = c.unroll > 0 && stream_config_covers(c, K_aug);
  return c;
}

bool stream_config_covers(const StreamConfig& c, int K_aug) {
  const int steps = (K_aug + kStepK - 1) / kStepK;
  const bool shape = (c.waves == 4 || c.waves == 8 || c.waves == 16) &&
                     (c.unroll == 1 || c.unroll == 2 || c.unroll == 3 || c.unroll == 4 ||
                      c.unroll == 6 || c.unroll == 8) &&
                     (c.groups == 1 || c.groups == 2 || c.groups == 4) && c.splits >= 1 &&
                     c.splits <= steps;
  const bool tiles_ok = (c.tiles == 1 || (c.tiles == 4 && c.waves >= 4)) &&
                        (c.wave_tiles == 1 ||
                         (c.wave_tiles == 4 && c.tiles == 1 && c.waves <= 8 && c.unroll <= 4 &&
                          c.groups == 1));
  if (!shape || !tiles_ok || c.reduce < 0 || c.reduce > 2) return false;
  const int nst_max = (steps + c.splits - 1) / c.splits;
  return static_cast<int64_t>(c.waves / c.tiles) * c.unroll >= nst_max &&
         stream_lds_bytes(c.waves, c.groups, nst_max, c.stage_lds, c.wave_tiles) <= kMaxStreamLds;
}

int choose_variant(int M_per_group, int N, int K_aug) {
  (void)N;
  (void)K_aug;
  return M_per_group <= 64 ? PRQ_GEMM_STREAM : PRQ_GEMM_TILE;
}

size_t stream_workspace_bytes(int M, int E, int N, int splits, int reduce) {
  if (splits <= 1 || reduce == kReduceAtomicY) return 0;
  const size_t mn = static_cast<size_t>(M) * N * sizeof(float);
  if (reduce == kReducePartials) return mn * splits;
  const size_t acc = (mn + 255) & ~static_cast<size_t>(255);
  return acc + static_cast<size_t>(E) * (N / 16) * sizeof(uint32_t);
}

hipError_t launch_gemm_stream(const uint8_t* Aq, const uint8_t* Asc, int M,
                              const int32_t* group_offsets, int E, const uint8_t* Wp,
                              const uint8_t* Wps, int N, int K_aug, float* Y,
                              const StreamConfig& cfg, void* workspace, hipStream_t stream) {
  float* acc = nullptr;
  uint32_t* ctr = nullptr;
  const int64_t mn = static_cast<int64_t>(M) * N;
  if (cfg.splits > 1 && cfg.reduce != kReduceAtomicY) {
    acc = static_cast<float*>(workspace);
    const size_t a = (static_cast<size_t>(mn) * sizeof(float) + 255) & ~static_cast<size_t>(255);
    ctr = reinterpret_cast<uint32_t*>(static_cast<char*>(workspace) + a);
  }
  if (cfg.splits > 1 && cfg.reduce == kReduceAtomicY) {
    zero_kernel<<<static_cast<unsigned>((mn + 255) / 256), 256, 0, stream>>>(Y, mn);
  }
  const int flags = (cfg.stage_lds ? 0 : kDirectA) | (cfg.reduce << 1);
  const int steps = (K_aug + kStepK - 1) / kStepK;
  const size_t lds = stream_lds_bytes(cfg.waves, cfg.groups, (steps + cfg.splits - 1) / cfg.splits,
                                      cfg.stage_lds, cfg.wave_tiles);
  const int per_wg = cfg.tiles * cfg.wave_tiles;     // 16-feature tiles per workgroup
  const int T = cfg.wave_tiles == 4 ? 5 : cfg.tiles;
  const dim3 grid((N / 16 + per_wg - 1) / per_wg, cfg.splits, group_offsets ? E : 1);
  const int U = cfg.unroll, G = cfg.groups;
  const int32_t* off = group_offsets;
  const int splits = cfg.splits;
  hipError_t err;
  if (group_offsets) {
    switch (cfg.waves) {
      case 4: err = launch_u<true, 4>(U, G, T, PRQ_STREAM_ARGS); break;
      case 8: err = launch_u<true, 8>(U, G, T, PRQ_STREAM_ARGS); break;
      default: err = launch_u<true, 16>(U, G, T, PRQ_STREAM_ARGS); break;
    }
  } else {
    switch (cfg.waves) {
      case 4: err = launch_u<false, 4>(U, G, T, PRQ_STREAM_ARGS); break;
      case 8: err = launch_u<false, 8>(U, G, T, PRQ_STREAM_ARGS); break;
      default: err = launch_u<false, 16>(U, G, T, PRQ_STREAM_ARGS); break;
    }
  }
  if (err != hipSuccess || cfg.splits <= 1 || cfg.reduce != kReducePartials) return err;
  reduce_partials_kernel<<<static_cast<unsigned>((mn + 255) / 256), 256, 0, stream>>>(
      acc, cfg.splits, mn, Y);
  return hipGetLastError();
}

}  // namespace prq
