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
//   * The group's activation rows (contiguous in the row-major quantizer
//     output) are then copied straight into LDS by direct global->LDS loads,
//     whole kilobytes of one row per copy, and its scale bytes as one
//     contiguous run -- no registers, one round trip for all of K.  Rows sit
//     at a pitch of a whole number of kilobytes plus 32 bytes, at which the
//     MFMA's operand read (lane l: row l % 16, 16 bytes of K part l / 16) is
//     free of LDS bank conflicts (measured; a pitch that is a multiple of
//     256 bytes conflicts 4- to 8-way).  Gathering the operand in MFMA lane
//     order instead (16 rows x 64 bytes and 64 scale bytes per copy) costs
//     ~2 us more per pass.
//   * One wait for all loads, one barrier; each wave reads all of its steps'
//     operands from LDS before its kU MFMAs (steps past its chunk meet zero
//     weight codes, so the reads need no branches), and a fixed-order sum of
//     the K chunks through LDS; Y is written once.
// K parts past K_aug read the row start (a valid address) and meet zero weight
// codes; rows past the group's end are zeroed at the MFMA.
// Grouped (MoE) mode: blockIdx.z is the expert; a workgroup loops over the
// expert's 16-row groups reusing its weight registers; experts without rows
// return before reading their weight.
//
// Direct variant (packed activation, two to four row groups): every operand
// loaded straight into registers, no LDS staging.  Each wave holds its K chunk
// of the weight of one or two tiles, so each activation kilobyte it loads
// feeds one or two MFMAs and no other wave needs it; the wave loads its chunk
// of the next row group's block while its MFMAs run on the current one, and
// the waves meet once, for the K-chunk sum of all groups and tiles.
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

// Pitch, in 16-byte pieces, of a staged activation row of nb pieces: whole
// kilobyte copies plus two pieces (32 bytes past a multiple of 1 KB).
__host__ __device__ inline int staged_row_pitch(int nb) { return ((nb + 63) & ~63) + 2; }

// LDS bytes of 16 staged rows, rounded up to whole kilobytes.
__host__ __device__ inline size_t staged_rows_bytes(int nb) {
  return (static_cast<size_t>(16) * staged_row_pitch(nb) * 16 + 1023) & ~static_cast<size_t>(1023);
}

__device__ __forceinline__ void wait_all_vm() {
  // vmcnt = 0, expcnt and lgkmcnt left at their maxima
  __builtin_amdgcn_s_waitcnt((0x7 << 4) | (0xF << 8));
}

template <bool kGrouped, bool kPackedA, int kT, int kU>
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

  // LDS: weight scales (kept for every pass), then the staged activation
  // rows, then their scale bytes; the reduction buffer of a pass reuses the rows.
  const int pitch = staged_row_pitch(nb);             // 16-byte pieces
  const int copies = (nb + 63) >> 6;                  // kilobyte copies per row
  uint8_t* const sWs = smem;                          // [kT][sgroups][64 dwords] weight scales
  uint8_t* const sA = smem + kT * sgroups * 256;      // [16][pitch][16 bytes] activation rows
  uint8_t* const sAs = sA + staged_rows_bytes(nb);    // the rows' scale bytes (after `shift`)
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
    // 2. The group's activation, straight into LDS.  Packed: the group's
    //    16-row block is one contiguous kilobyte per K step in MFMA lane
    //    order, plus its scale dwords.  Row-major: its rows, a kilobyte of one
    //    row per copy (lanes past the row read its start into the pad past the
    //    row's pieces, never read back), and their scale bytes as one run of
    //    16-byte pieces from the aligned address below it (each piece holds at
    //    least one byte of the run).
    int shift = 0;
    if constexpr (kPackedA) {
      const int64_t blk = pass_row >> 4;   // pass_row is a multiple of 16 (dense)
      for (int st = wave; st < steps; st += kWaves)
        __builtin_amdgcn_global_load_lds(PRQ_GPTR(Aq + (blk * steps + st) * 1024 + lane * 16),
                                         PRQ_LPTR(sA + st * 1024), 16, 0, 0);
      for (int q = wave; q < sgroups; q += kWaves)
        __builtin_amdgcn_global_load_lds(PRQ_GPTR(Asc + (blk * sgroups + q) * 256 + lane * 4),
                                         PRQ_LPTR(sAs + q * 256), 4, 0, 0);
    } else {
      const uint8_t* const ablk = Aq + static_cast<int64_t>(pass_row) * row_bytes;
      for (int i = wave; i < rows * copies; i += kWaves) {
        const int r = i / copies, c = i - r * copies;
        const int piece = c * 64 + lane;
        __builtin_amdgcn_global_load_lds(
            PRQ_GPTR(ablk + r * row_bytes + (piece < nb ? piece : 0) * 16),
            PRQ_LPTR(sA + (r * pitch + c * 64) * 16), 16, 0, 0);
      }
      const uint8_t* const sblk = Asc + static_cast<int64_t>(pass_row) * nb;
      shift = static_cast<int>(reinterpret_cast<uintptr_t>(sblk) & 15u);
      const int spieces = (rows * nb + shift + 15) >> 4;
      for (int i = wave; i < ((spieces + 63) >> 6); i += kWaves) {
        __builtin_amdgcn_global_load_lds(PRQ_GPTR(sblk - shift + min(i * 64 + lane, spieces - 1) * 16),
                                         PRQ_LPTR(sAs + i * 1024), 16, 0, 0);
      }
    }
    wait_all_vm();
    __syncthreads();

    // 3. The wave's operands from LDS, then its MFMAs, in batches of at most
    //    five steps (ten steps' operands at once do not fit beside the 40
    //    registers of weight).  Lane (lr, lk) of step s0 + j reads K part
    //    4 (s0 + j) + lk of row lr at a fixed offset from one base address per
    //    operand; the base is recomputed every pass (the empty asm), which
    //    keeps the compiler from holding ten steps' addresses in registers
    //    across passes.  Steps past the wave's chunk, rows past the group and
    //    tiles past N meet a zero activation operand, K parts past K_aug the
    //    neutral scale (their weight codes are zero), so no step branches;
    //    reads past a row land in the pad, the next row or the LDS tail.
    // (A wave with no steps reads from step 0: its operands are all masked.)
    int part0 = (s0 < steps ? s0 : 0) * 4 + lk;
    asm volatile("" : "+v"(part0));
    const int o = (part0 >> 2) & 3;   // s0 % 4
    // Packed: step s0 + j's operand is a kilobyte further on; row-major: 64
    // bytes (four K parts) further along the lane's row.
    const uint8_t* const a_at =
        kPackedA ? sA + (part0 >> 2) * 1024 + lane * 16 : sA + (lr * pitch + part0) * 16;
    const uint8_t* const sa_at = sAs + shift + lr * nb + part0;
    // Scale bytes held as dwords (four steps a dword, as in the packed
    // layouts) of steps 4 (s0 / 4) .. +4 nd - 1, realigned so that byte j % 4
    // of x[j / 4] is step s0 + j's (bytes past the tile's steps are never used).
    constexpr int nd = (kU + 6) / 4;
    uint32_t ws[nd + 1], xs[nd + 1];
    {
      const uint32_t* const ws_at = reinterpret_cast<const uint32_t*>(
          sWs + (t_in * sgroups + (part0 >> 4)) * 256 + lane * 4);
      const uint32_t* const xs_at =
          reinterpret_cast<const uint32_t*>(sAs + (part0 >> 4) * 256 + lane * 4);
#pragma unroll
      for (int i = 0; i < nd; ++i) {
        ws[i] = ws_at[i * 64];
        xs[i] = kPackedA ? xs_at[i * 64] : 0u;
      }
      ws[nd] = xs[nd] = 0;
#pragma unroll
      for (int i = 0; i < nd; ++i) {
        ws[i] = __builtin_amdgcn_alignbyte(ws[i + 1], ws[i], o);
        xs[i] = __builtin_amdgcn_alignbyte(xs[i + 1], xs[i], o);
      }
    }
    const bool row_ok = lr < rows && tile_ok;
    v4f acc = {0.f, 0.f, 0.f, 0.f};
    constexpr int kBatch = kU < 5 ? kU : 5;
#pragma unroll
    for (int j0 = 0; j0 < kU; j0 += kBatch) {
      uint4 a[kBatch];
      uint32_t sa[kBatch];
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        const int jj = j0 + j;
        if constexpr (kPackedA) {
          a[j] = *reinterpret_cast<const uint4*>(a_at + jj * 1024);
          sa[j] = (xs[jj >> 2] >> (8 * (jj & 3))) & 0xFFu;
        } else {
          a[j] = *reinterpret_cast<const uint4*>(a_at + jj * 64);
          sa[j] = sa_at[jj * 4];
        }
      }
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        const int jj = j0 + j;
        const bool step_ok = s0 + jj < s1;             // wave-uniform
        const bool use = row_ok && step_ok;
        // lane l's weight scale is feature l % 16's: masked by the step only
        const uint32_t sw = (ws[jj >> 2] >> (8 * (jj & 3))) & 0xFFu;
        acc = dev::mfma_fp4_16x16x128(w[jj], use ? a[j] : make_uint4(0, 0, 0, 0),
                                      step_ok ? sw : kNeutralScale,
                                      use && part0 + 4 * jj < nb ? sa[j] : kNeutralScale, acc);
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

// Lane (l % 16, l / 16) of step s0 + j: the packed block's kilobyte of step
// s0 + j (clamped to the last step; steps past the chunk are masked at the
// MFMA) and the nd scale dwords of steps 4 (s0 / 4) .. (clamped likewise).
template <int kU>
__device__ __forceinline__ void load_block(const uint8_t* __restrict__ Ap,
                                           const uint8_t* __restrict__ Aps, int64_t blk, int steps,
                                           int sgroups, int sbase, int lane, uint4 (&a)[kU],
                                           uint32_t (&xs)[(kU + 6) / 4 + 1]) {
  constexpr int nd = (kU + 6) / 4;
  const uint8_t* const ab = Ap + blk * steps * 1024 + lane * 16;
#pragma unroll
  for (int j = 0; j < kU; ++j)
    a[j] = *reinterpret_cast<const uint4*>(ab + static_cast<int64_t>(min(sbase + j, steps - 1)) * 1024);
  const uint32_t* const xg = reinterpret_cast<const uint32_t*>(Aps + blk * sgroups * 256) + lane;
#pragma unroll
  for (int i = 0; i < nd; ++i) xs[i] = xg[min((sbase >> 2) + i, sgroups - 1) * 64];
}

// Dense, packed activation: kTW 16-feature tiles per workgroup (tiles
// kTW blockIdx.x onward) and kP row groups (blockIdx.y + p gridDim.y), 16 waves
// of contiguous K chunks; each wave holds its chunk of the weight of every
// tile, so one load of its activation operand feeds kTW MFMAs.  Rows past M
// in the last block (zero codes as the packed quantizer writes them; whatever
// they hold only reaches their own output rows) are not stored; a second tile
// past N reloads the last one and is not stored.  The bits equal
// the staged kernel's with one tile per workgroup (same chunks, MFMA order
// and K-chunk sum).
template <int kU, int kP, int kTW>
__global__ __launch_bounds__(kWaves * 64) void gemm_decode_direct_kernel(
    const uint8_t* __restrict__ Ap, const uint8_t* __restrict__ Aps, int M,
    const uint8_t* __restrict__ Wp, const uint8_t* __restrict__ Wps, int N, int K_aug,
    float* __restrict__ Y) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int nd = (kU + 6) / 4;
  const int steps = (K_aug + kStepK - 1) / kStepK;
  const int sgroups = (steps + 3) >> 2;
  const int nb = K_aug >> 5;
  const int ntiles = N >> 4;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, lk = lane >> 4;
  const int tile0 = static_cast<int>(blockIdx.x) * kTW;
  const int per = (steps + kWaves - 1) / kWaves;   // <= kU (checked on the host)
  const int s0 = wave * per, s1 = min(steps, s0 + per);
  const int sbase = s0 < steps ? s0 : 0;          // a wave without steps reads step 0, masked
  const int o = sbase & 3;
  const int part0 = sbase * 4 + lk;

  // The weight chunks and their scale dwords (realigned after the first
  // loads of the activation are issued, so that no wait comes before them).
  uint4 w[kTW][kU];
  uint32_t ws[kTW][nd + 1];
#pragma unroll
  for (int tt = 0; tt < kTW; ++tt) {
    const int t = min(tile0 + tt, ntiles - 1);
    const uint8_t* const wt = Wp + static_cast<int64_t>(t) * steps * 1024 + lane * 16;
#pragma unroll
    for (int j = 0; j < kU; ++j)
      w[tt][j] = *reinterpret_cast<const uint4*>(wt + static_cast<int64_t>(min(sbase + j, steps - 1)) * 1024);
    const uint32_t* const wg = reinterpret_cast<const uint32_t*>(Wps + static_cast<int64_t>(t) * sgroups * 256) + lane;
#pragma unroll
    for (int i = 0; i < nd; ++i) ws[tt][i] = wg[min((sbase >> 2) + i, sgroups - 1) * 64];
    ws[tt][nd] = 0;
  }

  // Row group p's operands are loaded while group p - 1's MFMAs run (two
  // register sets); the scheduling barriers keep the compiler from sinking
  // the loads next to their MFMAs.  Groups past this workgroup's count
  // (only where the launch's rows do not divide evenly) reload the last block
  // and are not stored.
  const int nblk = (M + 15) >> 4;
  const int gy = static_cast<int>(gridDim.y), by = static_cast<int>(blockIdx.y);
  const int ngroups = (nblk - by + gy - 1) / gy;   // <= kP
  uint4 a[2][kU];
  uint32_t xs[2][nd + 1];
  load_block<kU>(Ap, Aps, by, steps, sgroups, sbase, lane, a[0], xs[0]);
  __builtin_amdgcn_sched_barrier(0);
  v4f acc[kP][kTW];
#pragma unroll
  for (int p = 0; p < kP; ++p) {
    if (p + 1 < kP)
      load_block<kU>(Ap, Aps, min(by + (p + 1) * gy, nblk - 1), steps, sgroups, sbase, lane,
                     a[(p + 1) & 1], xs[(p + 1) & 1]);
    __builtin_amdgcn_sched_barrier(0);
    if (p == 0) {
#pragma unroll
      for (int tt = 0; tt < kTW; ++tt)
#pragma unroll
        for (int i = 0; i < nd; ++i) ws[tt][i] = __builtin_amdgcn_alignbyte(ws[tt][i + 1], ws[tt][i], o);
    }
    uint32_t* const x = xs[p & 1];
    x[nd] = 0;
#pragma unroll
    for (int i = 0; i < nd; ++i) x[i] = __builtin_amdgcn_alignbyte(x[i + 1], x[i], o);
#pragma unroll
    for (int tt = 0; tt < kTW; ++tt) {
      v4f c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int jj = 0; jj < kU; ++jj) {
        const bool step_ok = s0 + jj < s1;   // wave-uniform
        const uint32_t sw = (ws[tt][jj >> 2] >> (8 * (jj & 3))) & 0xFFu;
        const uint32_t sa = (x[jj >> 2] >> (8 * (jj & 3))) & 0xFFu;
        c = dev::mfma_fp4_16x16x128(w[tt][jj], step_ok ? a[p & 1][jj] : make_uint4(0, 0, 0, 0),
                                    step_ok ? sw : kNeutralScale,
                                    step_ok && part0 + 4 * jj < nb ? sa : kNeutralScale, c);
      }
      acc[p][tt] = c;
    }
    __builtin_amdgcn_sched_barrier(0);
  }

  // The K chunks of every group and tile summed in a fixed order.
  // acc[p][tt][q] of this lane is Y[16 (by + p gy) + l % 16][16 (tile0 + tt) + 4 (l / 16) + q].
  float* const s_red = reinterpret_cast<float*>(smem);   // [kP][kTW][16 waves][64][4]
#pragma unroll
  for (int p = 0; p < kP; ++p)
#pragma unroll
    for (int tt = 0; tt < kTW; ++tt)
      *reinterpret_cast<v4f*>(s_red + (((p * kTW + tt) * kWaves + wave) * 64 + lane) * 4) = acc[p][tt];
  __syncthreads();
  for (int idx = tid; idx < ngroups * kTW * 256; idx += kWaves * 64) {
    const int pt = idx >> 8, l = (idx >> 2) & 63, q = idx & 3;
    const int p = pt / kTW, t = tile0 + (pt - p * kTW);
    const int row = (by + p * gy) * 16 + (l & 15);
    if (row < M && t < ntiles) {
      float v = 0.0f;
#pragma unroll
      for (int c = 0; c < kWaves; ++c) v += s_red[((pt * kWaves + c) * 64 + l) * 4 + q];
      Y[static_cast<int64_t>(row) * N + t * 16 + 4 * (l >> 4) + q] = v;
    }
  }
}

template <bool kGrouped, bool kPackedA, int kT, int kU>
hipError_t launch_cfg(dim3 grid, size_t lds, const uint8_t* Aq, const uint8_t* Asc, int M,
                      const int32_t* off, const uint8_t* Wp, const uint8_t* Wps, int N,
                      int K_aug, float* Y, hipStream_t stream) {
  static std::once_flag attr_once;   // dynamic LDS above the 64 KiB default
  std::call_once(attr_once, [] {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_decode_kernel<kGrouped, kPackedA, kT, kU>),
                              hipFuncAttributeMaxDynamicSharedMemorySize,
                              static_cast<int>(kMaxDecodeLds));
    (void)hipGetLastError();
  });
  gemm_decode_kernel<kGrouped, kPackedA, kT, kU><<<grid, kWaves * 64, lds, stream>>>(
      Aq, Asc, M, off, Wp, Wps, N, K_aug, Y);
  return hipGetLastError();
}

template <bool kGrouped, bool kPackedA, int kT>
hipError_t launch_u(int U, dim3 grid, size_t lds, const uint8_t* Aq, const uint8_t* Asc, int M,
                    const int32_t* off, const uint8_t* Wp, const uint8_t* Wps, int N, int K_aug,
                    float* Y, hipStream_t stream) {
  switch (U) {
    case 2:
      return launch_cfg<kGrouped, kPackedA, kT, 2>(grid, lds, Aq, Asc, M, off, Wp, Wps, N, K_aug, Y,
                                                   stream);
    case 5:
      return launch_cfg<kGrouped, kPackedA, kT, 5>(grid, lds, Aq, Asc, M, off, Wp, Wps, N, K_aug, Y,
                                                   stream);
    default:
      return launch_cfg<kGrouped, kPackedA, kT, 10>(grid, lds, Aq, Asc, M, off, Wp, Wps, N, K_aug, Y,
                                                    stream);
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
  const int nb = K_aug / 32;
  // the scale run of 16 rows: 16 nb bytes after a shift of up to 15, copied
  // in whole kilobytes of 16-byte pieces
  const size_t scale_bytes = static_cast<size_t>((((16 * nb + 15 + 15) >> 4) + 63) >> 6) * 1024;
  // + 10 KiB for the operand reads of steps past a wave's chunk (a wave reads
  // 10 steps from its first, or from step 0): in the row-major layout at most
  // 10 steps of 64 bytes past the last row, in the packed one 10 kilobyte
  // steps past the last step (the packed block of steps x 1 KB and its
  // sgroups x 256 scale bytes fit the row-major layout's room)
  return static_cast<size_t>(tiles) * ((steps + 3) / 4) * 256 +
         std::max(staged_rows_bytes(nb) + scale_bytes + 10240, static_cast<size_t>(kWaves) * 64 * 4 * 4);
}

DecodeConfig choose_decode_config(int M_per_group, int N, int K_aug, int grouped, int tiles,
                                  int row_splits, int num_cus, bool packed) {
  DecodeConfig c;
  const int steps = (K_aug + kStepK - 1) / kStepK;
  const int groups = (std::max(M_per_group, 1) + 15) / 16;
  // Dense (measured on the 9728 -> 2560 down_proj, weights rotated,
  // back-to-back launches): one tile per workgroup up to two row groups (two
  // passes of one workgroup row, M = 17 / 24 / 32 7.1 / 7.5 / 8.1 us, against
  // 7.7 / 7.8 / 8.0 for two tiles and a workgroup row per group), two tiles
  // per workgroup from three row groups on; then as many workgroup rows as
  // the launch fits in one round of the CUs (a workgroup at this LDS size
  // holds a CU), the row groups dealt to them in turn (M = 64: three rows
  // 10.6 us, two 10.7, four -- two rounds -- 12.3).  Grouped: one tile per
  // workgroup, the expert's row groups in one workgroup (the experts multiply
  // the workgroups).
  c.tiles = tiles > 0 ? tiles : (grouped || groups <= 2 ? 1 : 2);
  const int cols = (N / 16 + c.tiles - 1) / c.tiles;
  const int auto_rows = std::min(groups, std::max(1, std::max(num_cus, 1) / std::max(cols, 1)));
  c.row_splits = grouped ? 1 : std::min(row_splits > 0 ? row_splits : auto_rows, groups);
  if (c.tiles != 1 && c.tiles != 2 && c.tiles != 4) c.ok = false;
  c.unroll = round_decode_unroll((steps + kWaves / c.tiles - 1) / (kWaves / c.tiles));
  c.ok = c.ok && c.unroll > 0 && decode_lds_bytes(K_aug, c.tiles) <= kMaxDecodeLds &&
         (N % 16) == 0 && (!grouped || c.tiles == 1);
  // Packed activation from two row groups on: the direct variant.  Measured
  // on the down_proj (9728 -> 2560, weights rotated, back to back) against
  // the staged kernel's plan: two groups, one tile per wave and workgroup and
  // both groups in it, 6.8 against 7.4 us (two tiles per wave 7.0); three,
  // two tiles per wave and one group per workgroup row (240 workgroups), 6.9
  // against 7.7 (one tile per wave 7.3-7.8); four, two tiles per wave in three
  // workgroup rows, 7.9 against 9.8 (one tile, one row: 8.8).  Two tiles per
  // wave take at most two groups per workgroup (registers).
  const int per16 = (steps + kWaves - 1) / kWaves;
  if (packed && !grouped && tiles <= 0 && row_splits <= 0 && groups >= 2 && groups <= 4 &&
      per16 <= 5 && (N % 16) == 0) {
    const int cus = std::max(num_cus, 1);
    int tw = groups >= 3 ? 2 : 1;
    int cols = (N / 16 + tw - 1) / tw;
    int rows = std::min(groups, std::max(1, cus / cols));
    if (tw == 2 && (groups + rows - 1) / rows > 2) {
      tw = 1;
      cols = N / 16;
      rows = std::min(groups, std::max(1, cus / cols));
    }
    c.direct = true;
    c.tiles = tw;
    c.row_splits = rows;
    c.unroll = per16 <= 2 ? 2 : 5;
    c.ok = true;
  }
  return c;
}

size_t decode_direct_lds_bytes(int M, int tiles, int row_splits) {
  const int groups = (std::max(M, 1) + 15) / 16;
  const int kp = (groups + std::max(row_splits, 1) - 1) / std::max(row_splits, 1);
  return static_cast<size_t>(kp) * tiles * kWaves * 64 * 4 * sizeof(float);
}

hipError_t launch_gemm_decode(const uint8_t* Aq, const uint8_t* Asc, int M,
                              const int32_t* group_offsets, int E, const uint8_t* Wp,
                              const uint8_t* Wps, int N, int K_aug, float* Y,
                              const DecodeConfig& cfg, hipStream_t stream, bool packed_a) {
  if (packed_a && group_offsets) return hipErrorInvalidValue;   // dense only
  const int ntiles = N >> 4;
  if (cfg.direct) {
    const int groups = (M + 15) / 16;
    const int kp = cfg.row_splits >= 1 ? (groups + cfg.row_splits - 1) / cfg.row_splits : 0;
    if (!packed_a || groups < 1 || cfg.row_splits < 1 || cfg.row_splits > groups || kp > 4 ||
        (cfg.tiles == 2 && kp > 2) || (cfg.tiles != 1 && cfg.tiles != 2) ||
        (cfg.unroll != 2 && cfg.unroll != 5) || (N % 16) != 0)
      return hipErrorInvalidValue;
    const dim3 grid((ntiles + cfg.tiles - 1) / cfg.tiles, cfg.row_splits, 1);
    const size_t lds = decode_direct_lds_bytes(M, cfg.tiles, cfg.row_splits);   // <= 64 KiB
#define PRQ_DECODE_D(U, P, T)                                                                   \
  gemm_decode_direct_kernel<U, P, T><<<grid, kWaves * 64, lds, stream>>>(Aq, Asc, M, Wp, Wps, N, \
                                                                         K_aug, Y);             \
  return hipGetLastError()
#define PRQ_DECODE_DU(U)                       \
  if (cfg.tiles == 2) {                        \
    if (kp == 1) { PRQ_DECODE_D(U, 1, 2); }    \
    PRQ_DECODE_D(U, 2, 2);                     \
  }                                            \
  switch (kp) {                                \
    case 1: PRQ_DECODE_D(U, 1, 1);             \
    case 2: PRQ_DECODE_D(U, 2, 1);             \
    case 3: PRQ_DECODE_D(U, 3, 1);             \
    default: PRQ_DECODE_D(U, 4, 1);            \
  }
    if (cfg.unroll == 2) {
      PRQ_DECODE_DU(2)
    }
    PRQ_DECODE_DU(5)
#undef PRQ_DECODE_DU
#undef PRQ_DECODE_D
  }
  const bool grouped = group_offsets != nullptr;
  const dim3 grid((ntiles + cfg.tiles - 1) / cfg.tiles, grouped ? 1 : cfg.row_splits,
                  grouped ? E : 1);
  const size_t lds = decode_lds_bytes(K_aug, cfg.tiles);
#define PRQ_DECODE_T(G, P, T)                                                                   \
  return launch_u<G, P, T>(cfg.unroll, grid, lds, Aq, Asc, M, group_offsets, Wp, Wps, N, K_aug, Y, \
                           stream)
  if (grouped) {
    PRQ_DECODE_T(true, false, 1);
  }
  if (packed_a) {
    switch (cfg.tiles) {
      case 1: PRQ_DECODE_T(false, true, 1);
      case 2: PRQ_DECODE_T(false, true, 2);
      default: PRQ_DECODE_T(false, true, 4);
    }
  }
  switch (cfg.tiles) {
    case 1: PRQ_DECODE_T(false, false, 1);
    case 2: PRQ_DECODE_T(false, false, 2);
    default: PRQ_DECODE_T(false, false, 4);
  }
#undef PRQ_DECODE_T
}

}  // namespace prq
