// Decode kernel of the augmented MXFP4 GEMM (arXiv 2609.22106, Eq. 3: one
// block-scaled GEMM over K_aug = K + k) for up to 64 rows per weight.
//
// The weight read dominates and the run is short, so the kernel is built to
// have everything in flight at once and to need no second pass:
//   * A workgroup owns one group of 16 activation rows and kT tiles of 16
//     output features over the WHOLE K range: no split-K, hence no partial
//     sums, atomics or reduction kernel.  The feature tiles are blockIdx.x;
//     the row groups of a dense call are dealt to blockIdx.y, a workgroup
//     looping over its row groups with its weight still in registers.
//   * Its 16 waves are kT tiles x (16 / kT) contiguous K chunks.  Each wave
//     issues the loads of its chunk of the packed weight (the MFMA A operand,
//     one contiguous kilobyte per step) first, with clamped unconditional
//     addresses; the tiles' weight scale dwords go straight to LDS.
//   * The activation operand of every K step is then copied straight into LDS
//     in MFMA lane order by direct global->LDS loads (lane l: row l % 16, K
//     part l / 16, 16 bytes at LDS offset 16 l; its scale byte into dword slot
//     l), spread over the waves -- no registers, one round trip for all of K.
//     It is read back with one conflict-free 16-byte LDS read per MFMA.
//   * One wait for all loads, one barrier, kU MFMAs per wave, and a fixed-order
//     sum of the K chunks through LDS; Y is written once.
// K parts past K_aug read the row start (a valid address) and meet zero weight
// codes; rows past the group's end are zeroed at the MFMA.
// Grouped (MoE) mode: blockIdx.z is the expert; a workgroup loops over the
// expert's 16-row groups reusing its weight registers; experts without rows
// return before reading their weight.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>

#include "mx_device.hpp"
#include "prq_internal.h"

namespace prq {
namespace {

using dev::v4f;

constexpr int kStepK = 128;
constexpr int kStepBytes = kStepK / 2;
constexpr uint32_t kNeutralScale = 127;
constexpr int kWaves = 16;
constexpr size_t kMaxDecodeLds = 160 * 1024;

#define PRQ_GPTR(p) ((const __attribute__((address_space(1))) void*)(p))
#define PRQ_LPTR(p) ((__attribute__((address_space(3))) void*)(p))

__device__ __forceinline__ void wait_all_vm() {
  // vmcnt = 0, expcnt and lgkmcnt left at their maxima
  __builtin_amdgcn_s_waitcnt((0x7 << 4) | (0xF << 8));
}

template <bool kGrouped, int kT, int kU>
__global__ __launch_bounds__(kWaves * 64) void gemm_decode_kernel(
    const uint8_t* __restrict__ Aq, const uint8_t* __restrict__ Asc, int M,
    const int32_t* __restrict__ off, const uint8_t* __restrict__ Wp,
    const uint8_t* __restrict__ Wps, int N, int K_aug, float* __restrict__ Y) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int kChunks = kWaves / kT;

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
  const int tile = blockIdx.x * kT + t_in;
  const bool tile_ok = tile < ntiles;
  const int per = (steps + kChunks - 1) / kChunks;   // <= kU (checked on the host)
  const int s0 = chunk * per;
  const int s1 = min(steps, s0 + per);

  // 1. The wave's weight chunk, before anything else.
  const int64_t et = static_cast<int64_t>(e) * ntiles + (tile_ok ? tile : 0);
  const uint8_t* Wt = Wp + et * steps * 1024 + lane * 16;
  uint4 w[kU];
#pragma unroll
  for (int j = 0; j < kU; ++j) {
    const int st = min(s0 + j, steps - 1);
    w[j] = *reinterpret_cast<const uint4*>(Wt + static_cast<int64_t>(st) * 1024);
  }

  // LDS: weight scales (kept for every pass), then the staged activation,
  // which the reduction buffer of a pass reuses.
  uint8_t* const sWs = smem;                         // [kT][sgroups][64 dwords] weight scales
  uint8_t* const sA = smem + kT * sgroups * 256;     // [steps][1024] activation codes
  uint8_t* const sAs = sA + steps * 1024;            // [steps][64 dwords] activation scales
  float* const s_red = reinterpret_cast<float*>(sA);

  // The weight scale dwords of the workgroup's tiles, straight into LDS
  // (registers are kept for the weight codes).
  for (int i = wave; i < kT * sgroups; i += kWaves) {
    const int t = i / sgroups, q = i - t * sgroups;
    const int64_t et_i = static_cast<int64_t>(e) * ntiles + min(static_cast<int>(blockIdx.x) * kT + t, ntiles - 1);
    __builtin_amdgcn_global_load_lds(PRQ_GPTR(Wps + (et_i * sgroups + q) * 256 + lane * 4),
                                     PRQ_LPTR(sWs + i * 256), 4, 0, 0);
  }

  for (int pass_row = row_begin + static_cast<int>(blockIdx.y) * 16; pass_row < row_end;
       pass_row += static_cast<int>(gridDim.y) * 16) {
    const int rows = min(16, row_end - pass_row);
    const int m = pass_row + min(lr, rows - 1);
    // 2. The activation operand of every step, straight into LDS.
    for (int s = wave; s < steps; s += kWaves) {
      const bool kin = s * kStepK + lk * 32 < K_aug;
      __builtin_amdgcn_global_load_lds(
          PRQ_GPTR(Aq + m * row_bytes + (kin ? static_cast<int64_t>(s) * kStepBytes + lk * 16 : 0)),
          PRQ_LPTR(sA + s * 1024), 16, 0, 0);
      __builtin_amdgcn_global_load_lds(
          PRQ_GPTR(Asc + static_cast<int64_t>(m) * nb + (kin ? s * 4 + lk : 0)),
          PRQ_LPTR(sAs + s * 256), 1, 0, 0);
    }
    wait_all_vm();
    __syncthreads();

    // 3. MFMAs of the wave's chunk.
    v4f acc = {0.f, 0.f, 0.f, 0.f};
    const bool row_ok = lr < rows;
#pragma unroll
    for (int j = 0; j < kU; ++j) {
      const int st = s0 + j;
      if (tile_ok && st < s1) {                       // wave-uniform
        const uint4 a = *reinterpret_cast<const uint4*>(sA + st * 1024 + lane * 16);
        const uint32_t sa = *reinterpret_cast<const uint32_t*>(sAs + st * 256 + lane * 4) & 0xFFu;
        const uint32_t sw =
            (*reinterpret_cast<const uint32_t*>(sWs + (t_in * sgroups + (st >> 2)) * 256 + lane * 4) >>
             (8 * (st & 3))) & 0xFFu;
        acc = dev::mfma_fp4_16x16x128(w[j], row_ok ? a : make_uint4(0, 0, 0, 0), sw,
                                      row_ok ? sa : kNeutralScale, acc);
      }
    }
    __syncthreads();   // the staged operand becomes the reduction buffer

    // 4. Sum the K chunks of each tile in a fixed order.  acc[q] of this lane
    //    is Y[pass_row + lr][16 tile + 4 lk + q].
#pragma unroll
    for (int q = 0; q < 4; ++q) s_red[(wave * 64 + lane) * 4 + q] = acc[q];
    __syncthreads();
    for (int idx = tid; idx < kT * 256; idx += kWaves * 64) {
      const int t = idx >> 8, l = (idx >> 2) & 63, q = idx & 3;
      const int out_tile = blockIdx.x * kT + t;
      if ((l & 15) < rows && out_tile < ntiles) {
        float v = 0.0f;
#pragma unroll
        for (int c = 0; c < kChunks; ++c) v += s_red[((c * kT + t) * 64 + l) * 4 + q];
        Y[static_cast<int64_t>(pass_row + (l & 15)) * N + out_tile * 16 + 4 * (l >> 4) + q] = v;
      }
    }
    __syncthreads();   // before the next pass overwrites LDS
  }
}

template <bool kGrouped, int kT, int kU>
hipError_t launch_cfg(dim3 grid, size_t lds, const uint8_t* Aq, const uint8_t* Asc, int M,
                      const int32_t* off, const uint8_t* Wp, const uint8_t* Wps, int N,
                      int K_aug, float* Y, hipStream_t stream) {
  static std::once_flag attr_once;   // dynamic LDS above the 64 KiB default
  std::call_once(attr_once, [] {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_decode_kernel<kGrouped, kT, kU>),
                              hipFuncAttributeMaxDynamicSharedMemorySize,
                              static_cast<int>(kMaxDecodeLds));
    (void)hipGetLastError();
  });
  gemm_decode_kernel<kGrouped, kT, kU><<<grid, kWaves * 64, lds, stream>>>(Aq, Asc, M, off, Wp, Wps,
                                                                         N, K_aug, Y);
  return hipGetLastError();
}

template <bool kGrouped, int kT>
hipError_t launch_u(int U, dim3 grid, size_t lds, const uint8_t* Aq, const uint8_t* Asc, int M,
                    const int32_t* off, const uint8_t* Wp, const uint8_t* Wps, int N, int K_aug,
                    float* Y, hipStream_t stream) {
  switch (U) {
    case 2: return launch_cfg<kGrouped, kT, 2>(grid, lds, Aq, Asc, M, off, Wp, Wps, N, K_aug, Y, stream);
    case 5: return launch_cfg<kGrouped, kT, 5>(grid, lds, Aq, Asc, M, off, Wp, Wps, N, K_aug, Y, stream);
    default: return launch_cfg<kGrouped, kT, 10>(grid, lds, Aq, Asc, M, off, Wp, Wps, N, K_aug, Y, stream);
  }
}

// Weight steps per wave: at most 10 (40 registers of codes) -- a 16-wave
// workgroup leaves each wave 128 registers in all.
int round_decode_unroll(int per) {
  static const int kU[] = {2, 5, 10};
  for (int x : kU)
    if (x >= per) return x;
  return 0;
}

}  // namespace

size_t decode_lds_bytes(int K_aug, int tiles) {
  const int steps = (K_aug + kStepK - 1) / kStepK;
  return static_cast<size_t>(tiles) * ((steps + 3) / 4) * 256 +
         std::max(static_cast<size_t>(steps) * 1280, static_cast<size_t>(kWaves) * 64 * 4 * 4);
}

DecodeConfig choose_decode_config(int M_per_group, int N, int K_aug, int grouped, int tiles,
                                  int row_splits, int num_cus) {
  DecodeConfig c;
  const int steps = (K_aug + kStepK - 1) / kStepK;
  const int groups = (std::max(M_per_group, 1) + 15) / 16;
  // Dense (measured on the 9728 -> 2560 down_proj): one tile per workgroup
  // for one row group; from two row groups on, two tiles per workgroup, and
  // each row group its own workgroup row while the launch still fits the CUs
  // in one round (a workgroup at this LDS size holds a CU) -- a second pass
  // over another row group costs ~4 us more than a workgroup of its own --
  // else two workgroup rows, each looping over its row groups with the weight
  // still in registers.  Grouped: one tile per workgroup, the expert's row
  // groups in one workgroup (the experts multiply the workgroups).
  c.tiles = tiles > 0 ? tiles : (grouped || groups <= 1 ? 1 : 2);
  const int cols = (N / 16 + c.tiles - 1) / c.tiles;
  const int auto_rows = cols * groups <= std::max(num_cus, 1) ? groups : std::min(groups, 2);
  c.row_splits = grouped ? 1 : std::min(row_splits > 0 ? row_splits : auto_rows, groups);
  if (c.tiles != 1 && c.tiles != 2 && c.tiles != 4) c.ok = false;
  c.unroll = round_decode_unroll((steps + kWaves / c.tiles - 1) / (kWaves / c.tiles));
  c.ok = c.ok && c.unroll > 0 && decode_lds_bytes(K_aug, c.tiles) <= kMaxDecodeLds &&
         (N % 16) == 0 && (!grouped || c.tiles == 1);
  return c;
}

hipError_t launch_gemm_decode(const uint8_t* Aq, const uint8_t* Asc, int M,
                              const int32_t* group_offsets, int E, const uint8_t* Wp,
                              const uint8_t* Wps, int N, int K_aug, float* Y,
                              const DecodeConfig& cfg, hipStream_t stream) {
  const int ntiles = N >> 4;
  const bool grouped = group_offsets != nullptr;
  const dim3 grid((ntiles + cfg.tiles - 1) / cfg.tiles, grouped ? 1 : cfg.row_splits,
                  grouped ? E : 1);
  const size_t lds = decode_lds_bytes(K_aug, cfg.tiles);
#define PRQ_DECODE_T(G, T)                                                                   \
  return launch_u<G, T>(cfg.unroll, grid, lds, Aq, Asc, M, group_offsets, Wp, Wps, N, K_aug, Y, \
                        stream)
  if (grouped) {
    PRQ_DECODE_T(true, 1);
  }
  switch (cfg.tiles) {
    case 1: PRQ_DECODE_T(false, 1);
    case 2: PRQ_DECODE_T(false, 2);
    default: PRQ_DECODE_T(false, 4);
  }
#undef PRQ_DECODE_T
}

}  // namespace prq
