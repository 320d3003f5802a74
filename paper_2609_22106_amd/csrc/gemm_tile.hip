// LDS-tiled kernel of the augmented MXFP4 GEMM (arXiv 2609.22106, Eq. 3: one
// block-scaled GEMM over K_aug = K + k) for prefill shapes, with a grouped
// (MoE expert) mode in which rows [off[e], off[e+1]) multiply expert e's weight.
//
//   Y[m, n] = sum_b 2^(Asc[m,b]-127) 2^(Wsc[n,b]-127) sum_{i<32} A[m,32b+i] W[n,32b+i]
//
// on v_mfma_scale_f32_32x32x64_f8f6f4 (FP4 operands, E8M0 scales in the
// instruction, float32 accumulation; this form issues twice the products per
// cycle of the 16x16x128 one).
//
// A workgroup computes a kBM x kBN tile with kWM x kWN waves (wave tile
// kBM/kWM x kBN/kWN).  Per 128-element K step both operands are staged in LDS
// in MFMA lane order -- for each 16-row block, 64 lanes x 16 bytes, lane l
// holding row l % 16, K part l / 16 -- so that every operand read of a wave is
// one contiguous kilobyte (conflict-free 16-byte lane reads).  The weight comes
// in that order already (packed layout, pack.hip) and is copied verbatim; the
// activation rows are transposed into it on the store.  Scales are staged the
// same way, one scale byte per lane in a dword slot.  Pipeline: kNS LDS
// stages filled by direct global->LDS loads (global_load_lds: one wave
// instruction writes one lane-ordered kilobyte), kNS - 1 K steps in flight; per
// step each wave waits for its own loads of that step with an explicit vmcnt,
// one bare barrier, the next step's loads are issued into the stage just
// freed, then the MFMAs.  Source addresses are always valid (clamped rows and
// tiles; K parts past K_aug point at the row start and meet zero weight codes).
// Workgroup ids are remapped so that each XCD (ids are dealt to the 8 XCDs in
// turn) works on a contiguous band of row tiles and its L2 serves their
// activation rows to every feature tile.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>

#include "mx_device.hpp"
#include "prq.h"
#include "prq_internal.h"

namespace prq {
namespace {

using dev::v16f;

constexpr int kStepK = 128;
constexpr int kStepBytes = kStepK / 2;
constexpr int kXcds = 8;

// Bijective remap of a linear workgroup id: ids dealt round-robin to kXcds
// XCDs become contiguous ranges per XCD.
__device__ __forceinline__ int xcd_remap(int L, int total) {
  const int q = total / kXcds, r = total % kXcds;
  const int x = L % kXcds, i = L / kXcds;
  return x * q + min(x, r) + i;
}

// Row range and expert of row tile `mt` when tiles of `tile_rows` rows are
// numbered expert after expert (prefix scan of per-expert tile counts over
// the workgroup's threads, `nthreads` at a time).
template <int kThreads>
__device__ bool grouped_tile(const int32_t* __restrict__ off, int E, int M, int mt, int tile_rows,
                             int* e_out, int* row_begin, int* row_end) {
  __shared__ int s_scan[kThreads];
  __shared__ int s_hit[3];
  const int tid = threadIdx.x;
  if (tid == 0) s_hit[0] = -1;
  int base = 0;
  for (int e0 = 0; e0 < E; e0 += kThreads) {
    const int e = e0 + tid;
    int r0 = 0, r1 = 0, t = 0;
    if (e < E) {  // offsets clamped to [0, M]: malformed offsets cannot address past A
      r0 = min(max(off[e], 0), M);
      r1 = min(max(off[e + 1], r0), M);
      t = (r1 - r0 + tile_rows - 1) / tile_rows;
    }
    s_scan[tid] = t;
    __syncthreads();
    for (int d = 1; d < kThreads; d <<= 1) {  // inclusive Hillis-Steele scan
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
    base += s_scan[kThreads - 1];
    __syncthreads();
  }
  if (s_hit[0] < 0) return false;
  *e_out = s_hit[0];
  *row_begin = s_hit[1];
  *row_end = s_hit[2];
  return true;
}

template <int v>
struct IntC {
  static constexpr int value = v;
};

template <int n, class F, int i = 0>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (i < n) {
    f(IntC<i>{});
    static_for<n, F, i + 1>(static_cast<F&&>(f));
  }
}

#define PRQ_GPTR(p) ((const __attribute__((address_space(1))) void*)(p))
#define PRQ_LPTR(p) ((__attribute__((address_space(3))) void*)(p))

// s_waitcnt immediate that waits until at most n vector-memory operations of
// this wave are outstanding and all its LDS reads are complete (expcnt left at
// its maximum).  Before a bare barrier this makes the wave's reads of the
// stage that the next direct-to-LDS loads overwrite finished, not just issued.
template <int n>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(n >= 0 && n < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((n & 0xF) | ((n >> 4) << 14) | (0x7 << 4));
}

template <int kBM, int kBN, int kWM, int kWN, int kNS, bool kGrouped>
__global__ __launch_bounds__(kWM * kWN * 64) void gemm_tile_kernel(
    const uint8_t* __restrict__ Aq, const uint8_t* __restrict__ Asc, int M,
    const int32_t* __restrict__ off, int E, int n_mtiles, const uint8_t* __restrict__ Wp,
    const uint8_t* __restrict__ Wps, int N, int K_aug, float* __restrict__ Y) {
  constexpr int kWaves = kWM * kWN;
  constexpr int kThreads = kWaves * 64;
  constexpr int kTM = kBM / kWM, kTN = kBN / kWN;    // wave tile
  constexpr int kFM = kTM / 32, kFN = kTN / 32;      // 32x32 fragments per wave
  static_assert(kTM % 32 == 0 && kTN % 32 == 0, "wave tile of whole 32x32 fragments");
  constexpr int kABlk = kBM / 16, kBBlk = kBN / 16;  // 16-row operand blocks per step
  static_assert(kABlk % kWaves == 0 && kBBlk % kWaves == 0, "blocks split evenly over waves");
  constexpr int kAPer = kABlk / kWaves, kBPer = kBBlk / kWaves;
  constexpr int kLoads = 2 * (kAPer + kBPer);        // direct-to-LDS loads per wave per step
  // Stage layout: A codes [kABlk][1 KiB] | B codes [kBBlk][1 KiB] | A scales
  // [kABlk][64 dwords] | B scales [kBBlk][64 dwords]; lane order everywhere.
  constexpr int kOffB = kABlk * 1024;
  constexpr int kOffAs = (kABlk + kBBlk) * 1024;
  constexpr int kOffBs = kOffAs + kABlk * 256;
  constexpr int kStage = (kABlk + kBBlk) * 1280;
  static_assert(kNS >= 2 && kNS <= 6, "stages");
  // One LDS object per stage: the compiler then knows which stage an
  // in-flight direct-to-LDS load writes and does not make LDS reads of the
  // other stages wait for it.
  __shared__ __align__(16) uint8_t st0[kStage];
  __shared__ __align__(16) uint8_t st1[kStage];
  __shared__ __align__(16) uint8_t st2[kNS > 2 ? kStage : 16];
  __shared__ __align__(16) uint8_t st3[kNS > 3 ? kStage : 16];
  __shared__ __align__(16) uint8_t st4[kNS > 4 ? kStage : 16];
  __shared__ __align__(16) uint8_t st5[kNS > 5 ? kStage : 16];
  auto stage = [&](auto pc) -> uint8_t* {
    constexpr int p = decltype(pc)::value;
    if constexpr (p == 0) return st0;
    else if constexpr (p == 1) return st1;
    else if constexpr (p == 2) return st2;
    else if constexpr (p == 3) return st3;
    else if constexpr (p == 4) return st4;
    else return st5;
  };

  const int ntiles = N >> 4;
  const int n_ntiles = (N + kBN - 1) / kBN;
  const int total = n_mtiles * n_ntiles;
  const int logical = xcd_remap(blockIdx.x, total);
  const int mt = logical / n_ntiles, nt = logical % n_ntiles;

  int e = 0, row_begin, row_end;
  if (kGrouped) {
    if (!grouped_tile<kThreads>(off, E, M, mt, kBM, &e, &row_begin, &row_end)) return;
  } else {
    row_begin = mt * kBM;
    row_end = min(M, row_begin + kBM);
  }
  const int t0 = nt * kBBlk;                         // first 16-feature tile
  const int64_t row_bytes = K_aug >> 1;
  const int nb = K_aug >> 5;
  const int steps = (K_aug + kStepK - 1) / kStepK;
  const int sgroups = (steps + 3) >> 2;
  const uint8_t* We = Wp + static_cast<int64_t>(e) * ntiles * steps * 1024;
  const uint8_t* Wse = Wps + static_cast<int64_t>(e) * ntiles * sgroups * 256;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave / kWN, wn = wave % kWN;
  const int lr = lane & 15, lk = lane >> 4;

  // Per-lane source rows / tiles of this wave's loads (fixed over the K loop).
  const uint8_t* a_row[kAPer];
  const uint8_t* as_row[kAPer];
  const uint8_t* b_tile[kBPer];
  const uint8_t* bs_tile[kBPer];
#pragma unroll
  for (int i = 0; i < kAPer; ++i) {
    const int rb = wave + i * kWaves;
    const int m = min(row_begin + rb * 16 + lr, row_end - 1);
    a_row[i] = Aq + m * row_bytes;
    as_row[i] = Asc + static_cast<int64_t>(m) * nb;
  }
#pragma unroll
  for (int i = 0; i < kBPer; ++i) {
    const int t = min(t0 + wave + i * kWaves, ntiles - 1);
    b_tile[i] = We + static_cast<int64_t>(t) * steps * 1024 + lane * 16;
    bs_tile[i] = Wse + static_cast<int64_t>(t) * sgroups * 256 + lane * 4;
  }

  // Step s into stage `st`: every source address is valid (parts past K_aug
  // point at the row start: they meet zero weight codes with finite scales).
  auto issue = [&](int s, uint8_t* st) {
    const bool kok = s * kStepK + lk * 32 < K_aug;
    const int64_t abyte = kok ? static_cast<int64_t>(s) * kStepBytes + lk * 16 : 0;
    const int sbyte = kok ? s * 4 + lk : 0;
#pragma unroll
    for (int i = 0; i < kAPer; ++i)
      __builtin_amdgcn_global_load_lds(PRQ_GPTR(a_row[i] + abyte),
                                       PRQ_LPTR(st + (wave + i * kWaves) * 1024), 16, 0, 0);
#pragma unroll
    for (int i = 0; i < kBPer; ++i)
      __builtin_amdgcn_global_load_lds(PRQ_GPTR(b_tile[i] + static_cast<int64_t>(s) * 1024),
                                       PRQ_LPTR(st + kOffB + (wave + i * kWaves) * 1024), 16, 0, 0);
#pragma unroll
    for (int i = 0; i < kAPer; ++i)
      __builtin_amdgcn_global_load_lds(PRQ_GPTR(as_row[i] + sbyte),
                                       PRQ_LPTR(st + kOffAs + (wave + i * kWaves) * 256), 1, 0, 0);
#pragma unroll
    for (int i = 0; i < kBPer; ++i)
      __builtin_amdgcn_global_load_lds(PRQ_GPTR(bs_tile[i] + (s >> 2) * 256 + (s & 3)),
                                       PRQ_LPTR(st + kOffBs + (wave + i * kWaves) * 256), 1, 0, 0);
  };

  v16f acc[kFM][kFN];
#pragma unroll
  for (int i = 0; i < kFM; ++i)
#pragma unroll
    for (int j = 0; j < kFN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  // A 32-row x 64-element operand of the 32x32x64 MFMA read from the staged
  // 16-row x 128-element blocks: lane l takes row l % 32 (block 2f + bit 4 of
  // l), K part 2h + l / 32 of the step -- in-block lane (l % 16) + 16 (2h + l / 32),
  // so each 16 lanes read 256 contiguous bytes (conflict-free).
  const int blk_sel = (lane >> 4) & 1;
  const int lib0 = (lane & 15) + 16 * (lane >> 5);
  auto load_half = [&](const uint8_t* st, int h, uint4 (&a)[kFM], uint4 (&b)[kFN],
                       uint32_t (&sa)[kFM], uint32_t (&sb)[kFN]) {
    const int lib = lib0 + 32 * h;
#pragma unroll
    for (int i = 0; i < kFM; ++i) {
      const int blk = wm * (kTM / 16) + 2 * i + blk_sel;
      a[i] = *reinterpret_cast<const uint4*>(st + blk * 1024 + lib * 16);
      sa[i] = *reinterpret_cast<const uint32_t*>(st + kOffAs + blk * 256 + lib * 4);
    }
#pragma unroll
    for (int j = 0; j < kFN; ++j) {
      const int blk = wn * (kTN / 16) + 2 * j + blk_sel;
      b[j] = *reinterpret_cast<const uint4*>(st + kOffB + blk * 1024 + lib * 16);
      sb[j] = *reinterpret_cast<const uint32_t*>(st + kOffBs + blk * 256 + lib * 4);
    }
  };
  auto mfma_half = [&](const uint4 (&a)[kFM], const uint4 (&b)[kFN], const uint32_t (&sa)[kFM],
                       const uint32_t (&sb)[kFN]) {
#pragma unroll
    for (int i = 0; i < kFM; ++i)
#pragma unroll
      for (int j = 0; j < kFN; ++j)
        acc[i][j] = dev::mfma_fp4_32x32x64(a[i], b[j], sa[i], sb[j], acc[i][j]);
  };
  // With one wave per SIMD (4-wave workgroups) the register budget holds both
  // K halves' operands, so all LDS reads of a step are issued before its
  // MFMAs; with two waves per SIMD the halves go one after the other.
  constexpr bool kBothHalves = kWaves <= 4;
  auto compute = [&](const uint8_t* st) {
    uint4 a0[kFM], b0[kFN];
    uint32_t sa0[kFM], sb0[kFN];
    load_half(st, 0, a0, b0, sa0, sb0);
    if constexpr (kBothHalves) {
      uint4 a1[kFM], b1[kFN];
      uint32_t sa1[kFM], sb1[kFN];
      load_half(st, 1, a1, b1, sa1, sb1);
      mfma_half(a0, b0, sa0, sb0);
      mfma_half(a1, b1, sa1, sb1);
    } else {
      mfma_half(a0, b0, sa0, sb0);
      load_half(st, 1, a0, b0, sa0, sb0);
      mfma_half(a0, b0, sa0, sb0);
    }
  };

  // Prologue: steps 0 .. kNS-2 in flight.  Every wave issues the same
  // sequence on every path: steps past the end reload the last step into a
  // stage that is never read, and the wait, barrier and issue of a stage run
  // even when its step is past the end (only its MFMAs are skipped).  Then
  // exactly kNS - 2 later steps are in flight at every wait, one constant
  // vmcnt serves every step, and the compiler sees that the stage about to be
  // read has landed (a wait count chosen at run time, or a stage skipped as a
  // whole, leaves it a path that makes it drain all loads first).
  static_for<kNS - 1>([&](auto pc) {
    issue(min(static_cast<int>(decltype(pc)::value), steps - 1), stage(pc));
  });
  // Main loop, unrolled by kNS so every stage is a known LDS object.
  for (int s0 = 0; s0 < steps; s0 += kNS) {
    static_for<kNS>([&](auto pc) {
      constexpr int p = decltype(pc)::value;
      const int s = s0 + p;
      // This wave's loads of step s have landed; the bare barrier then says
      // the same of every wave, and that every wave is done reading the stage
      // the next issue overwrites.
      wait_vmcnt<(kNS - 2) * kLoads>();
      __builtin_amdgcn_s_barrier();
      issue(min(s + kNS - 1, steps - 1), stage(IntC<(p + kNS - 1) % kNS>{}));
      if (s < steps) compute(stage(pc));
    });
  }
  wait_vmcnt<0>();   // no direct-to-LDS write outlives the workgroup

  // Element e of a lane's fragment is C[8 (e / 4) + 4 (l / 32) + e % 4][l % 32]:
  // activation row, feature column (32 lanes store 128 contiguous bytes).
#pragma unroll
  for (int i = 0; i < kFM; ++i)
#pragma unroll
    for (int j = 0; j < kFN; ++j) {
      const int n = t0 * 16 + wn * kTN + j * 32 + (lane & 31);
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int m = row_begin + wm * kTM + i * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        if (m < row_end && n < N) Y[static_cast<int64_t>(m) * N + n] = acc[i][j][e];
      }
    }
}

template <int kBM, int kBN, int kWM, int kWN, int kNS>
hipError_t launch_shape(const uint8_t* Aq, const uint8_t* Asc, int M, const int32_t* off, int E,
                        const uint8_t* Wp, const uint8_t* Wps, int N, int K_aug, float* Y,
                        hipStream_t stream) {
  const int n_ntiles = (N + kBN - 1) / kBN;
  // Grouped: an upper bound on the row tiles over all experts (extra ids exit).
  const int n_mtiles = off ? (M + kBM - 1) / kBM + E : (M + kBM - 1) / kBM;
  const int grid = n_mtiles * n_ntiles;
  if (off)
    gemm_tile_kernel<kBM, kBN, kWM, kWN, kNS, true><<<grid, kWM * kWN * 64, 0, stream>>>(
        Aq, Asc, M, off, E, n_mtiles, Wp, Wps, N, K_aug, Y);
  else
    gemm_tile_kernel<kBM, kBN, kWM, kWN, kNS, false><<<grid, kWM * kWN * 64, 0, stream>>>(
        Aq, Asc, M, nullptr, 1, n_mtiles, Wp, Wps, N, K_aug, Y);
  return hipGetLastError();
}

}  // namespace

int choose_tile_shape(int M_rows, int N, int num_cus) {
  // Estimated cost ~ rounds of workgroups over the CUs x per-tile time; the
  // per-shape factors are measured throughputs per tile area relative to
  // 256 x 256 (smaller tiles move more bytes per MFMA).
  struct Shape { int id, bm, bn; double eff; };
  const Shape shapes[] = {{0, 256, 256, 1.0}, {1, 256, 128, 0.6}, {2, 128, 128, 0.55}};
  int best = 2;
  double best_cost = 1e300;
  for (const Shape& s : shapes) {
    const int tiles = ((M_rows + s.bm - 1) / s.bm) * ((N + s.bn - 1) / s.bn);
    const int rounds = (tiles + num_cus - 1) / num_cus;
    const double cost = rounds * static_cast<double>(s.bm) * s.bn / s.eff;
    if (cost < best_cost) {
      best_cost = cost;
      best = s.id;
    }
  }
  return best;
}

hipError_t launch_gemm_tile(const uint8_t* Aq, const uint8_t* Asc, int M,
                            const int32_t* group_offsets, int E, const uint8_t* Wp,
                            const uint8_t* Wps, int N, int K_aug, float* Y, int shape,
                            hipStream_t stream) {
  switch (shape) {
    case 0: return launch_shape<256, 256, 2, 4, 3>(Aq, Asc, M, group_offsets, E, Wp, Wps, N, K_aug, Y, stream);
    case 1: return launch_shape<256, 128, 2, 2, 4>(Aq, Asc, M, group_offsets, E, Wp, Wps, N, K_aug, Y, stream);
    default: return launch_shape<128, 128, 2, 2, 6>(Aq, Asc, M, group_offsets, E, Wp, Wps, N, K_aug, Y, stream);
  }
}

}  // namespace prq
