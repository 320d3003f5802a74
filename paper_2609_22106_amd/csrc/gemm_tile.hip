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
// the workgroup's threads, `nthreads` at a time).  With kAlign16 an expert's
// tiles start at its first row rounded down to a multiple of 16 (the packed
// activation's row blocks): rows [*row_begin, *row_end) are loaded, rows
// [*row_lo, *row_end) belong to the expert and are stored.  `lds` is
// kThreads + 4 ints of LDS scratch; every thread has read it on return once a
// barrier follows the call.
template <int kThreads, bool kAlign16>
__device__ bool grouped_tile(const int32_t* __restrict__ off, int E, int M, int mt, int tile_rows,
                             int* lds, int* e_out, int* row_begin, int* row_lo, int* row_end) {
  int* const s_scan = lds;
  int* const s_hit = lds + kThreads;
  const int tid = threadIdx.x;
  if (tid == 0) s_hit[0] = -1;
  int base = 0;
  for (int e0 = 0; e0 < E; e0 += kThreads) {
    const int e = e0 + tid;
    int r0 = 0, r1 = 0, b0 = 0, t = 0;
    if (e < E) {  // offsets clamped to [0, M]: malformed offsets cannot address past A
      r0 = min(max(off[e], 0), M);
      r1 = min(max(off[e + 1], r0), M);
      b0 = kAlign16 ? (r0 & ~15) : r0;
      t = r1 > r0 ? (r1 - b0 + tile_rows - 1) / tile_rows : 0;
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
      s_hit[1] = b0 + (mt - excl) * tile_rows;
      s_hit[2] = min(r1, s_hit[1] + tile_rows);
      s_hit[3] = max(r0, s_hit[1]);
    }
    base += s_scan[kThreads - 1];
    __syncthreads();
  }
  if (s_hit[0] < 0) return false;
  *e_out = s_hit[0];
  *row_begin = s_hit[1];
  *row_end = s_hit[2];
  *row_lo = s_hit[3];
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

// Instruction order of one pipelined step: the MFMAs one after another, the
// step's direct-to-LDS loads after the first kLd of them and its LDS reads of
// the next step spread between all of them, so both are issued while the
// matrix unit is busy.
template <int kMf, int kLd, int kRd>
__device__ __forceinline__ void interleave() {
  static_for<kMf>([&](auto ic) {
    constexpr int i = decltype(ic)::value;
    constexpr int r0 = i * kRd / kMf, r1 = (i + 1) * kRd / kMf;
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);              // MFMA
    if constexpr (i < kLd) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);   // VMEM read
    if constexpr (r1 > r0) __builtin_amdgcn_sched_group_barrier(0x100, r1 - r0, 0);  // DS read
  });
}

// How the activation operand is laid out in memory: row-major Aq/Asc with the
// scales staged a byte at a time or, when K_aug % 128 == 0, one aligned dword
// per row and step; or the packed (weight) layout, staged like the weight.
enum AMode { kARowByte = 0, kARowDword = 1, kAPacked = 2 };

// LDS stage of one 128-element K step: A codes [kBM/16 blocks][1 KiB] | B codes
// [kBN/16 blocks][1 KiB] | A scales | B scales [kBN/16 tiles][64 dwords].  Codes
// are in MFMA lane order (block b, lane l: row 16b + l % 16, K part l / 16, 16
// bytes).  A scales: row dwords -- one dword per row (the row's four scale bytes
// of the step); row bytes -- one byte per lane-order slot of each 16-row block
// (dword slots); packed -- as B.  B scales are the packed weight's dwords of the
// step's group of four steps (byte j = step 4q+j).
template <int kBM, int kBN, int kAMode>
struct TileStage {
  static constexpr int kABlk = kBM / 16, kBBlk = kBN / 16;
  static constexpr int kOffB = kABlk * 1024;
  static constexpr int kOffAs = (kABlk + kBBlk) * 1024;
  static constexpr int kAsBytes = kAMode == kARowDword ? kBM * 4 : kABlk * 256;
  static constexpr int kOffBs = kOffAs + kAsBytes;
  static constexpr int kBytes = kOffBs + kBBlk * 256;
};


template <int kBM, int kBN, int kWM, int kWN, int kNS, bool kGrouped, int kAMode>
__global__ __launch_bounds__(kWM * kWN * 64) void gemm_tile_kernel(
    const uint8_t* __restrict__ Aq, const uint8_t* __restrict__ Asc, int M,
    const int32_t* __restrict__ off, int E, int n_mtiles, int tile_base, int region_tiles,
    const uint8_t* __restrict__ Wp,
    const uint8_t* __restrict__ Wps, int N, int K_aug, float* __restrict__ Y, int splits,
    int split_steps, float* __restrict__ ws, int group_rows) {
  using L = TileStage<kBM, kBN, kAMode>;
  constexpr bool kScaleDword = kAMode == kARowDword;
  constexpr bool kPackedA = kAMode == kAPacked;
  constexpr int kWaves = kWM * kWN;
  constexpr int kThreads = kWaves * 64;
  constexpr int kTM = kBM / kWM, kTN = kBN / kWN;    // wave tile
  constexpr int kFM = kTM / 32, kFN = kTN / 32;      // 32x32 fragments per wave
  static_assert(kTM % 32 == 0 && kTN % 32 == 0, "wave tile of whole 32x32 fragments");
  constexpr int kABlk = L::kABlk, kBBlk = L::kBBlk;
  static_assert(kABlk % kWaves == 0, "A code blocks split evenly over waves");
  static_assert(kBBlk % 4 == 0, "B scales move four tile entries per instruction");
  // B blocks are dealt to the waves in turn; when they do not divide evenly
  // (256 x 320: 20 blocks, 8 waves) the last block is loaded again into its own
  // place (the same bytes), so that every wave issues the same loads.
  constexpr int kAPer = kABlk / kWaves, kBPer = (kBBlk + kWaves - 1) / kWaves;
  // Scale instructions per step: A as 64 row dwords, one per 16-row block
  // (bytes), or four block entries of 256 bytes (packed); B as four tile
  // entries.  When there are fewer than waves, several waves load the same
  // chunk (identical bytes).
  constexpr int kAsChunks = kScaleDword ? kBM / 64 : (kPackedA ? kABlk / 4 : kABlk);
  constexpr int kBsChunks = kBBlk / 4;
  constexpr int kAsPer = (kAsChunks + kWaves - 1) / kWaves;
  constexpr int kBsPer = (kBsChunks + kWaves - 1) / kWaves;
  // Packed activations: the A and B scale chunks (a kilobyte each) are one list
  // dealt to the waves in turn, so no wave reloads a chunk another wave loads.
  constexpr int kScChunks = kAsChunks + kBsChunks;
  constexpr int kScPer = (kScChunks + kWaves - 1) / kWaves;
  // direct-to-LDS loads per wave per step
  constexpr int kLoads = kAPer + kBPer + (kPackedA ? kScPer : kAsPer + kBsPer);
  static_assert(kNS >= 2 && kNS <= 4, "stages");
  static_assert(kNS * L::kBytes <= 160 * 1024, "LDS");
  static_assert(L::kBytes >= kThreads * 4 + 16, "the expert scan borrows a stage");
  constexpr int kU = kNS;         // main-loop unroll: the stage index is known
  constexpr int kMfmas = 2 * kFM * kFN;                                  // per step
  constexpr int kReads = 4 * (kFM + kFN);                                // LDS reads per step
  // One LDS object per stage: the compiler then knows which stage an in-flight
  // direct-to-LDS load writes and does not make LDS reads of the other stages
  // wait for it.
  __shared__ __align__(16) uint8_t st0[L::kBytes];
  __shared__ __align__(16) uint8_t st1[L::kBytes];
  __shared__ __align__(16) uint8_t st2[kNS > 2 ? L::kBytes : 16];
  __shared__ __align__(16) uint8_t st3[kNS > 3 ? L::kBytes : 16];
  auto stage = [&](auto pc) -> uint8_t* {
    constexpr int p = decltype(pc)::value % kNS;
    if constexpr (p == 0) return st0;
    else if constexpr (p == 1) return st1;
    else if constexpr (p == 2) return st2;
    else return st3;
  };

  const int ntiles = N >> 4;
  const int n_ntiles = (region_tiles + kBBlk - 1) / kBBlk;   // column tiles of the region
  // Split-K: workgroup id = split * tiles + tile; split p takes K steps
  // [p * split_steps, (p + 1) * split_steps) (the host makes every range
  // non-empty) and writes its partial sum to Y (p = 0) or ws[p - 1].
  // Grouped launches keep the hardware's round-robin order: their grid is an
  // upper bound, and contiguous per-XCD bands would hand the surplus ids (all
  // at the end) to the last XCDs, idling them (146 against 170 us on the
  // expert prefill shape).  An expert's weight column tile still stays on one
  // XCD (id mod 8 fixes the column tile when the column tiles are a multiple
  // of 8).
  const int n_tiles = n_mtiles * n_ntiles;
  const int logical = kGrouped ? static_cast<int>(blockIdx.x) : xcd_remap(blockIdx.x, n_tiles * splits);
  const int split = logical / n_tiles;
  const int tl = logical - split * n_tiles;
  // Tile order within a launch: row-major (an XCD's contiguous range is a band
  // of row tiles), or groups of group_rows row tiles, column-major inside each
  // group, so that an XCD's range is a block of row and column tiles and its
  // L2 holds fewer operand bytes per step (the host's choice per launch).
  int mt, nt;
  if (!kGrouped && group_rows > 0) {                  // uniform
    const int grp = tl / (group_rows * n_ntiles), first_m = grp * group_rows;
    const int gm = min(n_mtiles - first_m, group_rows);
    const int in_g = tl - grp * group_rows * n_ntiles;
    mt = first_m + in_g % gm;
    nt = in_g / gm;
  } else {
    mt = tl / n_ntiles;
    nt = tl % n_ntiles;
  }

  int e = 0, row_begin, row_lo, row_end;
  if (kGrouped) {
    // (the scan's scratch is stage 0, free until the first load is issued)
    if (!grouped_tile<kThreads, kPackedA>(off, E, M, mt, kBM, reinterpret_cast<int*>(st0), &e,
                                          &row_begin, &row_lo, &row_end))
      return;
    __syncthreads();
  } else {
    row_begin = row_lo = mt * kBM;
    row_end = min(M, row_begin + kBM);
  }
  const int t0 = tile_base + nt * kBBlk;             // first 16-feature tile
  const int n_end = min(N, (tile_base + region_tiles) * 16);   // the region's columns
  const int64_t row_bytes = K_aug >> 1;
  const int nb = K_aug >> 5;
  const int steps = (K_aug + kStepK - 1) / kStepK;
  const int sgroups = (steps + 3) >> 2;
  const int s_lo = split * split_steps;
  const int s_hi = min(steps, s_lo + split_steps);
  const int nblk = (M + 15) >> 4;                    // packed activation row blocks
  const uint8_t* We = Wp + static_cast<int64_t>(e) * ntiles * steps * 1024;
  const uint8_t* Wse = Wps + static_cast<int64_t>(e) * ntiles * sgroups * 256;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: scalar registers
  const int wm = wave / kWN, wn = wave % kWN;
  const int lr = lane & 15, lk = lane >> 4;

  // Per-lane byte offsets of this wave's loads from uniform bases (fixed over
  // the K loop; rows and tiles clamped into the operands; the host checks that
  // the operands fit 32-bit offsets).
  // Scale kilobytes (four 256-byte blocks of 64 dwords, dword = row + 16 K
  // part) land in LDS with the K parts of every odd block swapped in pairs
  // (0 <-> 1, 2 <-> 3).  A wave's scale read covers two blocks, 16 lanes per
  // (block, K part); the LDS serves dword reads half a wave at a time over 32
  // banks, so without the swap lanes 0-15 and 16-31 (same K part, two blocks)
  // hit the same 16 banks; with it they take the other 16.  A lane's global
  // source is its own piece's swap partner.
  uint32_t a_off[kAPer], as_off[kAsPer], b_off[kBPer], bs_off[kBsPer], sc_off[kScPer];
  const int swz = ((lane & 15) ^ (((lane >> 4) & 1) << 2)) * 16;
#pragma unroll
  for (int i = 0; i < kAPer; ++i) {
    if constexpr (kPackedA) {
      const int rb = min((row_begin >> 4) + wave + i * kWaves, nblk - 1);
      a_off[i] = static_cast<uint32_t>(rb) * steps * 1024 + lane * 16;
    } else {
      const int m = min(row_begin + (wave + i * kWaves) * 16 + lr, row_end - 1);
      a_off[i] = static_cast<uint32_t>(m) * static_cast<uint32_t>(row_bytes) + lk * 16;
    }
  }
#pragma unroll
  for (int i = 0; i < kAsPer; ++i) {
    const int c = (wave + i * kWaves) % kAsChunks;
    const int m = kScaleDword ? min(row_begin + c * 64 + lane, row_end - 1)
                              : min(row_begin + c * 16 + lr, row_end - 1);
    as_off[i] = static_cast<uint32_t>(m) * nb;
  }
#pragma unroll
  for (int i = 0; i < kScPer; ++i) {   // packed: A chunks first, then B chunks
    const int c = (wave + i * kWaves) % kScChunks;
    const int blk = c < kAsChunks ? min((row_begin >> 4) + c * 4 + (lane >> 4), nblk - 1)
                                  : min(t0 + (c - kAsChunks) * 4 + (lane >> 4), ntiles - 1);
    sc_off[i] = static_cast<uint32_t>(blk) * sgroups * 256 + swz;
  }
#pragma unroll
  for (int i = 0; i < kBPer; ++i) {
    const int t = min(t0 + min(wave + i * kWaves, kBBlk - 1), ntiles - 1);
    b_off[i] = static_cast<uint32_t>(t) * steps * 1024 + lane * 16;
  }
#pragma unroll
  for (int i = 0; i < kBsPer; ++i) {
    const int c = (wave + i * kWaves) % kBsChunks;
    const int t = min(t0 + c * 4 + (lane >> 4), ntiles - 1);
    bs_off[i] = static_cast<uint32_t>(t) * sgroups * 256 + swz;
  }

  // Step s into stage `st`.  Every source address is valid: with K_aug not a
  // multiple of 128, K parts of the last step past K_aug point at the row start
  // (they meet zero weight codes with finite scales).
  auto issue = [&](int s, uint8_t* st) {
    const bool kok = kScaleDword || s * kStepK + lk * 32 < K_aug;
#pragma unroll
    for (int i = 0; i < kAPer; ++i) {
      if constexpr (kPackedA)   // padded past K_aug and M: whole steps, whole blocks
        __builtin_amdgcn_global_load_lds(PRQ_GPTR(Aq + (a_off[i] + s * 1024u)),
                                         PRQ_LPTR(st + (wave + i * kWaves) * 1024), 16, 0, 0);
      else
        __builtin_amdgcn_global_load_lds(
            PRQ_GPTR(Aq + (kok ? a_off[i] + s * kStepBytes : a_off[i] - lk * 16)),
            PRQ_LPTR(st + (wave + i * kWaves) * 1024), 16, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < kBPer; ++i)
      __builtin_amdgcn_global_load_lds(PRQ_GPTR(We + (b_off[i] + s * 1024u)),
                                       PRQ_LPTR(st + L::kOffB + min(wave + i * kWaves, kBBlk - 1) * 1024), 16,
                                       0, 0);
    if constexpr (kPackedA) {
#pragma unroll
      for (int i = 0; i < kScPer; ++i) {   // four blocks' entries of the step's group
        const int c = (wave + i * kWaves) % kScChunks;   // uniform: the source is a select
        const uint8_t* src = c < kAsChunks ? Asc : Wse;
        const int dst = c < kAsChunks ? L::kOffAs + c * 1024 : L::kOffBs + (c - kAsChunks) * 1024;
        __builtin_amdgcn_global_load_lds(PRQ_GPTR(src + (sc_off[i] + (s >> 2) * 256u)),
                                         PRQ_LPTR(st + dst), 16, 0, 0);
      }
    } else {
#pragma unroll
      for (int i = 0; i < kAsPer; ++i) {
        const int c = (wave + i * kWaves) % kAsChunks;
        if constexpr (kScaleDword)   // K_aug % 128 == 0: the row's 4 bytes of step s, aligned
          __builtin_amdgcn_global_load_lds(PRQ_GPTR(Asc + (as_off[i] + s * 4)),
                                           PRQ_LPTR(st + L::kOffAs + c * 256), 4, 0, 0);
        else {   // block c: the lane's K part (swapped in odd blocks); past K_aug the row start
          const int kp = lk ^ (c & 1);
          __builtin_amdgcn_global_load_lds(
              PRQ_GPTR(Asc + (as_off[i] + (s * kStepK + kp * 32 < K_aug ? s * 4 + kp : 0))),
              PRQ_LPTR(st + L::kOffAs + c * 256), 1, 0, 0);
        }
      }
#pragma unroll
      for (int i = 0; i < kBsPer; ++i) {
        const int c = (wave + i * kWaves) % kBsChunks;
        __builtin_amdgcn_global_load_lds(PRQ_GPTR(Wse + (bs_off[i] + (s >> 2) * 256u)),
                                         PRQ_LPTR(st + L::kOffBs + c * 1024), 16, 0, 0);
      }
    }
  };

  v16f acc[kFM][kFN];
#pragma unroll
  for (int i = 0; i < kFM; ++i)
#pragma unroll
    for (int j = 0; j < kFN; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.f;

  // Operands of one half of a step in registers: for half h (K elements
  // [64h, 64h+64) of the step), the 32-row x 64-element MFMA operand of
  // fragment i: lane l takes row l % 32 (block 2i + bit 4 of l) and K part
  // 2h + l / 32, i.e. in-block lane (l % 16) + 16 (2h + l / 32); each 16 lanes
  // read 256 contiguous bytes (conflict-free).
  struct Half {
    uint4 a[kFM], b[kFN];
    uint32_t sa[kFM], sb[kFN];
  };
  // Per-lane LDS byte offsets of the reads within a stage; fragment and half
  // add compile-time constants (the instruction's immediate offset).
  const int blk_sel = (lane >> 4) & 1;
  const int lib0 = (lane & 15) + 16 * (lane >> 5);
  const uint32_t a_lb = (wm * (kTM / 16) + blk_sel) * 1024 + lib0 * 16;
  const uint32_t b_lb = L::kOffB + (wn * (kTN / 16) + blk_sel) * 1024 + lib0 * 16;
  // Scale dwords: half h of a step reads K part 2h + l / 32, found in an odd
  // block (blk_sel = 1) at part 2h + (l / 32 ^ 1).
  static_assert((kTM / 16) % 2 == 0 && (kTN / 16) % 2 == 0, "blk_sel is the block parity");
  const uint32_t lsc = (lane & 15) * 4 + (((lane >> 5) ^ blk_sel) * 64);
  const uint32_t as_lb = kScaleDword ? L::kOffAs + (wm * kTM + (lane & 31)) * 4
                                     : L::kOffAs + (wm * (kTM / 16) + blk_sel) * 256 + lsc;
  const uint32_t bs_lb = L::kOffBs + (wn * (kTN / 16) + blk_sel) * 256 + lsc;
  const uint32_t a_shift = 8 * (lane >> 5);   // row dword: part l / 32 to byte 0, 2 + l / 32 to byte 2
  auto read = [&](const uint8_t* st, auto hc, Half& o) {
    constexpr int h = decltype(hc)::value;
#pragma unroll
    for (int i = 0; i < kFM; ++i) {
      o.a[i] = *reinterpret_cast<const uint4*>(st + a_lb + (2 * i * 1024 + h * 512));
      o.sa[i] = *reinterpret_cast<const uint32_t*>(
          st + as_lb + (kScaleDword ? 32 * i * 4 : 2 * i * 256 + h * 128));
    }
#pragma unroll
    for (int j = 0; j < kFN; ++j) {
      o.b[j] = *reinterpret_cast<const uint4*>(st + b_lb + (2 * j * 1024 + h * 512));
      o.sb[j] = *reinterpret_cast<const uint32_t*>(st + bs_lb + (2 * j * 256 + h * 128));
    }
  };
  // The MFMAs of half h of step s.  Packed scale dwords hold four K steps:
  // byte s mod 4 is shifted down to byte 0 (one shift per fragment and step;
  // a compile-time byte select would force a 4-step unroll).
  auto mfma = [&](const Half& o, auto hc, int s) {
    constexpr int h = decltype(hc)::value;
    const uint32_t qshift = 8u * static_cast<uint32_t>(s & 3);
    uint32_t sb[kFN];
#pragma unroll
    for (int j = 0; j < kFN; ++j) sb[j] = o.sb[j] >> qshift;
#pragma unroll
    for (int i = 0; i < kFM; ++i) {
      const uint32_t sa = kScaleDword ? (o.sa[i] >> a_shift) : (kPackedA ? (o.sa[i] >> qshift) : o.sa[i]);
#pragma unroll
      for (int j = 0; j < kFN; ++j)
        acc[i][j] = dev::mfma_fp4_32x32x64_sel<kScaleDword ? 2 * h : 0, 0>(o.a[i], o.b[j], sa,
                                                                          sb[j], acc[i][j]);
    }
  };

  // Pipeline, kNS stages of one K step each.  Prologue: steps 0 .. kNS-1 into
  // every stage; wait for step 0; read its first half.  Iteration s:
  //   MFMAs of half 0 of step s, while half 1 of step s is read from LDS;
  //   wait until this wave's loads of step s+1 have landed and its LDS reads
  //   are complete, one bare barrier (the same then holds for every wave, so
  //   step s's stage is free), issue step s+kNS into it;
  //   MFMAs of half 1 of step s, while half 0 of step s+1 is read.
  // Every wave issues the same sequence on every path -- steps past the end
  // reload the last step, and the wait, barrier, issue and reads of a step run
  // even past the end (only its MFMAs are skipped) -- so one constant vmcnt
  // serves every iteration and the compiler sees that the stage about to be
  // read has landed (a wait count chosen at run time leaves it a path on which
  // it drains every load first).  Scheduling barriers keep each wait and
  // barrier between the MFMAs it separates.
  static_for<kNS>([&](auto pc) {
    issue(min(s_lo + static_cast<int>(decltype(pc)::value), s_hi - 1), stage(pc));
  });
  wait_vmcnt<(kNS - 1) * kLoads>();
  __builtin_amdgcn_s_barrier();
  Half h0, h1;
  read(st0, IntC<0>{}, h0);
  auto body = [&](int s0, auto pc, auto gc) {
    constexpr int p = decltype(pc)::value;
    constexpr bool kGuard = decltype(gc)::value;
    const int s = s0 + p;
    const bool live = !kGuard || s < s_hi;
    __builtin_amdgcn_sched_barrier(0);
    if (live) mfma(h0, IntC<0>{}, s);
    read(stage(pc), IntC<1>{}, h1);
    if constexpr (!kGuard) interleave<kMfmas / 2, 0, kReads / 2>();
    __builtin_amdgcn_sched_barrier(0);
    wait_vmcnt<(kNS - 2) * kLoads>();
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    issue(min(s + kNS, s_hi - 1), stage(pc));
    if (live) mfma(h1, IntC<1>{}, s);
    read(stage(IntC<p + 1>{}), IntC<0>{}, h0);
    if constexpr (!kGuard) interleave<kMfmas / 2, kLoads, kReads / 2>();
    __builtin_amdgcn_sched_barrier(0);
  };
  // Whole groups of kU steps without guards (so the scheduler can interleave
  // the LDS reads with the MFMAs), then one guarded group for the rest.
  int s0 = s_lo;
  for (; s0 + kU <= s_hi; s0 += kU)
    static_for<kU>([&](auto pc) { body(s0, pc, IntC<0>{}); });
  if (s0 < s_hi) static_for<kU>([&](auto pc) { body(s0, pc, IntC<1>{}); });
  wait_vmcnt<0>();   // no direct-to-LDS write outlives the workgroup

  // Element q of a lane's fragment is C[8 (q / 4) + 4 (l / 32) + q % 4][l % 32]:
  // activation row, feature column (32 lanes store 128 contiguous bytes).
  float* const dst = split == 0 ? Y : ws + static_cast<int64_t>(split - 1) * M * N;
#pragma unroll
  for (int i = 0; i < kFM; ++i)
#pragma unroll
    for (int j = 0; j < kFN; ++j) {
      const int n = t0 * 16 + wn * kTN + j * 32 + (lane & 31);
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int m = row_begin + wm * kTM + i * 32 + 8 * (q >> 2) + 4 * (lane >> 5) + (q & 3);
        if (m >= row_lo && m < row_end && n < n_end) dst[static_cast<int64_t>(m) * N + n] = acc[i][j][q];
      }
    }
}

// Grouped (MoE) tile GEMM on a packed activation, persistent and pipelined
// across tiles.  XCD x (workgroup ids are dealt to the XCDs in turn) owns
// experts x, x + 8, x + 16, ... and its workgroups stride over that list's
// tiles (expert-major, row tiles then column tiles), so each expert's weight
// and rows are fetched into one L2.  Lane j of every wave holds expert x + 8 j
// (up to 512 experts) and the inclusive prefix of the list's row-tile counts
// (a wave scan: no LDS, no barrier); a tile's expert is the number of lanes
// whose prefix ends at or before it.
//
// A tile takes P = ceil(steps / kNS) * kNS pipeline slots (slots past the K
// steps compute nothing), so every tile starts on stage 0; slot s issues slot
// s + kNS, which from slot P - kNS on is the first steps of the workgroup's
// next tile.  The next tile's loads are therefore in flight while the current
// tile finishes and stores, and its first half step is already in registers
// when its MFMAs start.  The same per-step wait, barrier and load sequence as
// gemm_tile_kernel; the first slots of a tile also wait for the previous
// tile's Y stores (they share the memory counter), which is conservative.
template <int kBM, int kBN, int kWM, int kWN, int kNS>
__global__ __launch_bounds__(kWM * kWN * 64) void gemm_grouped_persist_kernel(
    const uint8_t* __restrict__ Ap, const uint8_t* __restrict__ Aps, int M,
    const int32_t* __restrict__ off, int E, const uint8_t* __restrict__ Wp,
    const uint8_t* __restrict__ Wps, int N, int K_aug, float* __restrict__ Y) {
  using L = TileStage<kBM, kBN, kAPacked>;
  constexpr int kWaves = kWM * kWN;
  constexpr int kTM = kBM / kWM, kTN = kBN / kWN;
  constexpr int kFM = kTM / 32, kFN = kTN / 32;
  static_assert(kTM % 32 == 0 && kTN % 32 == 0, "wave tile of whole 32x32 fragments");
  constexpr int kABlk = L::kABlk, kBBlk = L::kBBlk;
  static_assert(kABlk % kWaves == 0 && kBBlk % kWaves == 0, "code blocks split evenly over waves");
  static_assert(kABlk % 4 == 0 && kBBlk % 4 == 0, "scales move four block entries per instruction");
  constexpr int kAPer = kABlk / kWaves, kBPer = kBBlk / kWaves;
  constexpr int kAsChunks = kABlk / 4, kBsChunks = kBBlk / 4;
  constexpr int kScChunks = kAsChunks + kBsChunks;   // one list dealt to the waves
  constexpr int kScPer = (kScChunks + kWaves - 1) / kWaves;
  constexpr int kLoads = kAPer + kBPer + kScPer;
  static_assert(kNS >= 2 && kNS <= 4, "stages");
  static_assert(kNS * L::kBytes <= 160 * 1024, "LDS");
  constexpr int kU = kNS;
  constexpr int kMfmas = 2 * kFM * kFN;
  constexpr int kReads = 4 * (kFM + kFN);
  __shared__ __align__(16) uint8_t st0[L::kBytes];
  __shared__ __align__(16) uint8_t st1[L::kBytes];
  __shared__ __align__(16) uint8_t st2[kNS > 2 ? L::kBytes : 16];
  __shared__ __align__(16) uint8_t st3[kNS > 3 ? L::kBytes : 16];
  auto stage = [&](auto pc) -> uint8_t* {
    constexpr int p = decltype(pc)::value % kNS;
    if constexpr (p == 0) return st0;
    else if constexpr (p == 1) return st1;
    else if constexpr (p == 2) return st2;
    else return st3;
  };

  const int ntiles = N >> 4;
  const int n_ntiles = (ntiles + kBBlk - 1) / kBBlk;
  const int steps = (K_aug + kStepK - 1) / kStepK;
  const int sgroups = (steps + 3) >> 2;
  const int nblk = (M + 15) >> 4;
  const int slots = (steps + kNS - 1) / kNS * kNS;   // P: pipeline slots per tile
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / kWN, wn = wave % kWN;

  // This XCD's experts, one per lane.
  const int xcd = static_cast<int>(blockIdx.x) % kXcds;
  int px_r0 = 0, px_r1 = 0, px_b0 = 0, px_t = 0;
  {
    const int ex = xcd + kXcds * lane;
    if (ex < E) {   // offsets clamped to [0, M]: malformed offsets cannot address past A
      px_r0 = min(max(off[ex], 0), M);
      px_r1 = min(max(off[ex + 1], px_r0), M);
      px_b0 = px_r0 & ~15;
      px_t = px_r1 > px_r0 ? (px_r1 - px_b0 + kBM - 1) / kBM : 0;
    }
  }
  int px_incl = px_t;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int u = __shfl_up(px_incl, d, 64);
    if (lane >= d) px_incl += u;
  }
  const int n_tiles = __builtin_amdgcn_readlane(px_incl, 63) * n_ntiles;
  const int q_step = static_cast<int>(gridDim.x) / kXcds;
  int q = static_cast<int>(blockIdx.x) / kXcds;
  if (q >= n_tiles) return;

  struct Tile {
    int row_begin, row_lo, row_end, t0;
    const uint8_t* W;    // the expert's packed weight codes
    const uint8_t* Ws;   // and scales
  };
  // Tile q of this XCD's list (q < n_tiles).
  auto tile_at = [&](int tq) {
    const int mtl = tq / n_ntiles;
    const int j = __popcll(__ballot(px_incl <= mtl));
    const int e = xcd + kXcds * j;
    const int first = __builtin_amdgcn_readlane(px_incl, j) - __builtin_amdgcn_readlane(px_t, j);
    Tile t;
    t.row_begin = __builtin_amdgcn_readlane(px_b0, j) + (mtl - first) * kBM;
    t.row_end = min(__builtin_amdgcn_readlane(px_r1, j), t.row_begin + kBM);
    t.row_lo = max(__builtin_amdgcn_readlane(px_r0, j), t.row_begin);
    t.t0 = (tq - mtl * n_ntiles) * kBBlk;
    t.W = Wp + static_cast<int64_t>(e) * ntiles * steps * 1024;
    t.Ws = Wps + static_cast<int64_t>(e) * ntiles * sgroups * 256;
    return t;
  };
  // Per-lane byte offsets of a tile's loads (rows and feature tiles clamped
  // into the operands; 32-bit offsets checked on the host).
  struct Offs {
    uint32_t a[kAPer], b[kBPer], sc[kScPer];
  };
  const int swz = ((lane & 15) ^ (((lane >> 4) & 1) << 2)) * 16;
  auto offsets = [&](const Tile& t) {
    Offs o;
#pragma unroll
    for (int i = 0; i < kAPer; ++i) {
      const int rb = min((t.row_begin >> 4) + wave + i * kWaves, nblk - 1);
      o.a[i] = static_cast<uint32_t>(rb) * steps * 1024 + lane * 16;
    }
#pragma unroll
    for (int i = 0; i < kBPer; ++i) {
      const int ft = min(t.t0 + wave + i * kWaves, ntiles - 1);
      o.b[i] = static_cast<uint32_t>(ft) * steps * 1024 + lane * 16;
    }
#pragma unroll
    for (int i = 0; i < kScPer; ++i) {   // A scale chunks first, then B
      const int c = (wave + i * kWaves) % kScChunks;
      const int blk = c < kAsChunks ? min((t.row_begin >> 4) + c * 4 + (lane >> 4), nblk - 1)
                                    : min(t.t0 + (c - kAsChunks) * 4 + (lane >> 4), ntiles - 1);
      o.sc[i] = static_cast<uint32_t>(blk) * sgroups * 256 + swz;   // odd blocks' K parts swapped in pairs
    }
    return o;
  };

  Tile cur = tile_at(q);
  bool has_next = q + q_step < n_tiles;
  Tile nxt = has_next ? tile_at(q + q_step) : cur;
  Offs oc = offsets(cur), on = offsets(nxt);

  // Slot `slot` of the current tile into stage `st`: slots past the tile are
  // the next tile's first slots (or, after the last tile, reload its last step).
  // The operand selection is branch-free: every wave issues the same loads.
  auto issue = [&](int slot, uint8_t* st) {
    const bool use_next = has_next && slot >= slots;
    const int s = use_next ? min(slot - slots, steps - 1) : min(slot, steps - 1);
    const uint8_t* W = use_next ? nxt.W : cur.W;
    const uint8_t* Ws = use_next ? nxt.Ws : cur.Ws;
#pragma unroll
    for (int i = 0; i < kAPer; ++i)
      __builtin_amdgcn_global_load_lds(PRQ_GPTR(Ap + ((use_next ? on.a[i] : oc.a[i]) + s * 1024u)),
                                       PRQ_LPTR(st + (wave + i * kWaves) * 1024), 16, 0, 0);
#pragma unroll
    for (int i = 0; i < kBPer; ++i)
      __builtin_amdgcn_global_load_lds(PRQ_GPTR(W + ((use_next ? on.b[i] : oc.b[i]) + s * 1024u)),
                                       PRQ_LPTR(st + L::kOffB + (wave + i * kWaves) * 1024), 16,
                                       0, 0);
#pragma unroll
    for (int i = 0; i < kScPer; ++i) {
      const int c = (wave + i * kWaves) % kScChunks;   // uniform: the source is a select
      const uint8_t* src = c < kAsChunks ? Aps : Ws;
      const int dst = c < kAsChunks ? L::kOffAs + c * 1024 : L::kOffBs + (c - kAsChunks) * 1024;
      __builtin_amdgcn_global_load_lds(
          PRQ_GPTR(src + ((use_next ? on.sc[i] : oc.sc[i]) + (s >> 2) * 256u)),
          PRQ_LPTR(st + dst), 16, 0, 0);
    }
  };

  // Operand registers and LDS reads as in gemm_tile_kernel (packed layout).
  struct Half {
    uint4 a[kFM], b[kFN];
    uint32_t sa[kFM], sb[kFN];
  };
  const int blk_sel = (lane >> 4) & 1;
  const int lib0 = (lane & 15) + 16 * (lane >> 5);
  const uint32_t a_lb = (wm * (kTM / 16) + blk_sel) * 1024 + lib0 * 16;
  const uint32_t b_lb = L::kOffB + (wn * (kTN / 16) + blk_sel) * 1024 + lib0 * 16;
  static_assert((kTM / 16) % 2 == 0 && (kTN / 16) % 2 == 0, "blk_sel is the block parity");
  const uint32_t lsc = (lane & 15) * 4 + (((lane >> 5) ^ blk_sel) * 64);   // odd blocks swapped
  const uint32_t as_lb = L::kOffAs + (wm * (kTM / 16) + blk_sel) * 256 + lsc;
  const uint32_t bs_lb = L::kOffBs + (wn * (kTN / 16) + blk_sel) * 256 + lsc;
  auto read = [&](const uint8_t* st, auto hc, Half& o) {
    constexpr int h = decltype(hc)::value;
#pragma unroll
    for (int i = 0; i < kFM; ++i) {
      o.a[i] = *reinterpret_cast<const uint4*>(st + a_lb + (2 * i * 1024 + h * 512));
      o.sa[i] = *reinterpret_cast<const uint32_t*>(st + as_lb + (2 * i * 256 + h * 128));
    }
#pragma unroll
    for (int j = 0; j < kFN; ++j) {
      o.b[j] = *reinterpret_cast<const uint4*>(st + b_lb + (2 * j * 1024 + h * 512));
      o.sb[j] = *reinterpret_cast<const uint32_t*>(st + bs_lb + (2 * j * 256 + h * 128));
    }
  };
  v16f acc[kFM][kFN];
  auto mfma = [&](const Half& o, int s) {
    const uint32_t qshift = 8u * static_cast<uint32_t>(s & 3);
#pragma unroll
    for (int i = 0; i < kFM; ++i) {
      const uint32_t sa = o.sa[i] >> qshift;
#pragma unroll
      for (int j = 0; j < kFN; ++j)
        acc[i][j] = dev::mfma_fp4_32x32x64_sel<0, 0>(o.a[i], o.b[j], sa, o.sb[j] >> qshift,
                                                     acc[i][j]);
    }
  };

  // Prologue of the first tile: slots 0 .. kNS-1, all landed, half 0 of slot 0 read.
  static_for<kNS>([&](auto pc) { issue(static_cast<int>(decltype(pc)::value), stage(pc)); });
  wait_vmcnt<0>();
  __builtin_amdgcn_s_barrier();
  Half h0, h1;
  read(st0, IntC<0>{}, h0);
  auto body = [&](int s0, auto pc, auto gc) {
    constexpr int p = decltype(pc)::value;
    constexpr bool kGuard = decltype(gc)::value;
    const int s = s0 + p;
    const bool live = !kGuard || s < steps;
    __builtin_amdgcn_sched_barrier(0);
    if (live) mfma(h0, s);
    read(stage(pc), IntC<1>{}, h1);
    if constexpr (!kGuard) interleave<kMfmas / 2, 0, kReads / 2>();
    __builtin_amdgcn_sched_barrier(0);
    wait_vmcnt<(kNS - 2) * kLoads>();
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    issue(s + kNS, stage(pc));
    if (live) mfma(h1, s);
    read(stage(IntC<p + 1>{}), IntC<0>{}, h0);
    if constexpr (!kGuard) interleave<kMfmas / 2, kLoads, kReads / 2>();
    __builtin_amdgcn_sched_barrier(0);
  };

  for (;;) {
#pragma unroll
    for (int i = 0; i < kFM; ++i)
#pragma unroll
      for (int j = 0; j < kFN; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
    int s0 = 0;
    for (; s0 + kU <= steps; s0 += kU)
      static_for<kU>([&](auto pc) { body(s0, pc, IntC<0>{}); });
    if (s0 < steps) static_for<kU>([&](auto pc) { body(s0, pc, IntC<1>{}); });

    // Y rows [row_lo, row_end) of the tile (element e of a lane's fragment is
    // C[8 (e / 4) + 4 (l / 32) + e % 4][l % 32]).
#pragma unroll
    for (int i = 0; i < kFM; ++i)
#pragma unroll
      for (int j = 0; j < kFN; ++j) {
        const int n = cur.t0 * 16 + wn * kTN + j * 32 + (lane & 31);
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int m = cur.row_begin + wm * kTM + i * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
          if (m >= cur.row_lo && m < cur.row_end && n < N)
            Y[static_cast<int64_t>(m) * N + n] = acc[i][j][e];
        }
      }
    if (!has_next) break;
    q += q_step;
    cur = nxt;
    oc = on;
    has_next = q + q_step < n_tiles;
    if (has_next) {
      nxt = tile_at(q + q_step);
      on = offsets(nxt);
    }
  }
  wait_vmcnt<0>();   // no direct-to-LDS write outlives the workgroup
}

// Split-K sum: Y[i] = ((Y[i] + P_0[i]) + P_1[i]) + ... over `parts` partial
// arrays of n4 float4 each, in that fixed order.
__global__ __launch_bounds__(256) void splitk_reduce_kernel(float4* __restrict__ Y,
                                                          const float4* __restrict__ P,
                                                          int64_t n4, int parts) {
  for (int64_t i = blockIdx.x * 256 + threadIdx.x; i < n4; i += static_cast<int64_t>(gridDim.x) * 256) {
    float4 v = Y[i];
    for (int p = 0; p < parts; ++p) {
      const float4 w = P[p * n4 + i];
      v.x += w.x;
      v.y += w.y;
      v.z += w.z;
      v.w += w.w;
    }
    Y[i] = v;
  }
}

template <int kBM, int kBN, int kWM, int kWN, int kNS, int kAMode>
hipError_t launch_shape_scales(const uint8_t* Aq, const uint8_t* Asc, int M, const int32_t* off,
                               int E, const uint8_t* Wp, const uint8_t* Wps, int N, int K_aug,
                               float* Y, int tile_base, int region_tiles, int splits, float* ws,
                               hipStream_t stream) {
  // The kernel addresses A and one expert's weight with 32-bit byte offsets.
  const int64_t steps = (K_aug + kStepK - 1) / kStepK;
  if (static_cast<int64_t>((M + 15) / 16) * steps * 1024 >= (int64_t{1} << 31) ||
      static_cast<int64_t>(N / 16) * steps * 1024 >= (int64_t{1} << 31))
    return hipErrorInvalidValue;
  if (region_tiles <= 0) return hipSuccess;
  const int n_ntiles = (region_tiles + kBN / 16 - 1) / (kBN / 16);
  // Grouped: an upper bound on the row tiles over all experts (extra ids exit):
  // expert e takes ceil((c_e + a) / kBM) <= (c_e + a + kBM - 1) / kBM tiles for
  // its c_e rows, a = 15 with the packed layout (tiles start on the expert's
  // first 16-row block), else 0; summed over the experts and floored.
  const int64_t lead = kAMode == kAPacked ? 15 : 0;
  const int n_mtiles = off ? static_cast<int>((M + static_cast<int64_t>(E) * (kBM - 1 + lead)) / kBM)
                           : (M + kBM - 1) / kBM;
  // Split-K (dense, whole-width calls only): every split a non-empty K range.
  int split_steps = static_cast<int>(steps);
  if (splits > 1) {
    if (off || !ws || tile_base != 0 || region_tiles != N / 16) return hipErrorInvalidValue;
    split_steps = static_cast<int>((steps + splits - 1) / splits);
    splits = static_cast<int>((steps + split_steps - 1) / split_steps);
  } else {
    splits = 1;
  }
  const int grid = n_mtiles * n_ntiles * splits;
  if (off) {
    gemm_tile_kernel<kBM, kBN, kWM, kWN, kNS, true, kAMode><<<grid, kWM * kWN * 64, 0, stream>>>(
        Aq, Asc, M, off, E, n_mtiles, tile_base, region_tiles, Wp, Wps, N, K_aug, Y, 1,
        split_steps, nullptr, 0);
  } else {
    // Grouped tile order (measured, weights rotated, M x N x (K + k)): for 256-row
    // tiles always -- 4096 x 9728 x 2624 in 256 x 320, 77.0 -> 73.6 us; 4096 x
    // 2560 x 4192 in 256 x 256, 40.3 -> 35.0; 2048 x 2560 x 9984 in 256 x 128,
    // 52.5 -> 44.8 -- and for 128 x 128 tiles up to 8 row tiles (1024 x 2560 x
    // 9984: 31.6 -> 28.8 us; 2048 x 2560 went 44.4 -> 51.5, 512 and 4096 x 1024
    // unchanged).
    const int group_rows = kBM == 256 || n_mtiles <= 8 ? 4 : 0;
    gemm_tile_kernel<kBM, kBN, kWM, kWN, kNS, false, kAMode><<<grid, kWM * kWN * 64, 0, stream>>>(
        Aq, Asc, M, nullptr, 1, n_mtiles, tile_base, region_tiles, Wp, Wps, N, K_aug, Y, splits,
        split_steps, ws, group_rows);
  }
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || splits == 1) return err;
  // Y += ws[0] + ws[1] + ... in that order (deterministic).
  const int64_t n4 = static_cast<int64_t>(M) * N / 4;
  const int blocks = static_cast<int>(std::min<int64_t>((n4 + 255) / 256, 2048));
  splitk_reduce_kernel<<<blocks, 256, 0, stream>>>(reinterpret_cast<float4*>(Y),
                                                    reinterpret_cast<const float4*>(ws), n4,
                                                    splits - 1);
  return hipGetLastError();
}

// Activation scale rows are dword-aligned when K_aug is a multiple of 128
// (K_aug / 32 scale bytes per row) and Asc is; otherwise they are staged a
// byte at a time.
template <int kBM, int kBN, int kWM, int kWN, int kNSDword, int kNSByte>
hipError_t launch_shape(const uint8_t* Aq, const uint8_t* Asc, int M, const int32_t* off, int E,
                        const uint8_t* Wp, const uint8_t* Wps, int N, int K_aug, float* Y,
                        bool packed, int tile_base, int region_tiles, int splits, float* ws,
                        hipStream_t stream) {
  if (packed)
    return launch_shape_scales<kBM, kBN, kWM, kWN, kNSDword, kAPacked>(
        Aq, Asc, M, off, E, Wp, Wps, N, K_aug, Y, tile_base, region_tiles, splits, ws, stream);
  if (K_aug % 128 == 0 && (reinterpret_cast<uintptr_t>(Asc) & 3u) == 0)
    return launch_shape_scales<kBM, kBN, kWM, kWN, kNSDword, kARowDword>(
        Aq, Asc, M, off, E, Wp, Wps, N, K_aug, Y, tile_base, region_tiles, splits, ws, stream);
  return launch_shape_scales<kBM, kBN, kWM, kWN, kNSByte, kARowByte>(
      Aq, Asc, M, off, E, Wp, Wps, N, K_aug, Y, tile_base, region_tiles, splits, ws, stream);
}

// Columns [16 tile_base, 16 (tile_base + region_tiles)) of Y with one tile shape
// (split along K into `splits` ranges when > 1: whole-width dense calls, ws of
// (splits - 1) * M * N floats).
hipError_t launch_region(const uint8_t* Aq, const uint8_t* Asc, int M, const int32_t* off, int E,
                         const uint8_t* Wp, const uint8_t* Wps, int N, int K_aug, float* Y,
                         int shape, bool packed, int tile_base, int region_tiles,
                         hipStream_t stream, int splits = 1, float* ws = nullptr) {
  switch (shape) {
    case 0: return launch_shape<256, 256, 2, 4, 4, 3>(Aq, Asc, M, off, E, Wp, Wps, N, K_aug, Y, packed, tile_base, region_tiles, splits, ws, stream);
    case 1: return launch_shape<256, 128, 2, 2, 4, 4>(Aq, Asc, M, off, E, Wp, Wps, N, K_aug, Y, packed, tile_base, region_tiles, splits, ws, stream);
    case 3: return launch_shape<256, 320, 4, 2, 3, 3>(Aq, Asc, M, off, E, Wp, Wps, N, K_aug, Y, packed, tile_base, region_tiles, splits, ws, stream);
    default: return launch_shape<128, 128, 2, 2, 4, 4>(Aq, Asc, M, off, E, Wp, Wps, N, K_aug, Y, packed, tile_base, region_tiles, splits, ws, stream);
  }
}

struct Shape {
  int id, bm, bn;
  double eff_rows;      // measured throughput per tile area relative to 256 x 256 (row-major A)
  // Packed A, by the most tiles any CU runs (1, 2, 3 or more), relative to one
  // 256 x 256 tile per CU; fitted to the down_proj sweep (M = 1024 .. 8192, N =
  // 2560, K + k = 9984, weights rotated): 128 x 128 workgroups fit two to a CU
  // and hide each other's latency, so two per CU run far better than one.
  double eff_packed[3];
};
// 256 x 320 (8 waves, 64 x 160 each, 3 stages): where it fills the CUs evenly
// it beats every other plan -- 8192 x 2560 x 9984 in one round of 256 tiles,
// 106 against 120 us for 256 x 256 over 2048 columns and 128 x 128 over the
// rest; 4096 x 9728 x 2624, 80 against 93 us -- and loses elsewhere (half-empty
// rounds); its factors are set to pick it exactly there.
constexpr Shape kShapes[] = {{0, 256, 256, 1.0, {1.0, 0.92, 0.92}},
                             {1, 256, 128, 0.63, {0.73, 0.87, 0.80}},
                             {2, 128, 128, 0.5, {0.58, 0.81, 0.68}},
                             {3, 256, 320, 0.5, {0.9, 0.9, 0.85}}};

// Cost of `tiles` tiles of shape s on `cus` CUs in tile-area units (one
// 256 x 256 tile alone on its CU = 65536): the busiest CU's tiles over the
// shape's efficiency at that load.
double shape_cost(const Shape& s, bool packed, long tiles, int cus) {
  const long per_cu = (tiles + cus - 1) / cus;
  const double eff = packed ? s.eff_packed[std::min<long>(per_cu, 3) - 1] : s.eff_rows;
  return per_cu * static_cast<double>(s.bm) * s.bn / eff;
}

// Plan of a dense tile GEMM: one shape over all N columns (optionally split
// along K), or a main region of whole column tiles in one shape and the
// remaining columns in another, so that each launch fills the CUs in whole
// rounds (M = 8192, N = 2560: 256 tiles of 256 x 256 over 2048 columns, then
// 256 tiles of 128 x 128).  Modelled time: workgroup rounds x (K steps per
// workgroup + a fixed pipeline fill and store cost) x the shape's measured
// time per step, plus a fixed cost for a second launch, or for split-K the
// reduction (a launch plus the partial sums written, read and added).
struct TilePlan {
  int shape[2] = {2, 2};
  int tiles[2] = {0, 0};   // 16-column tiles of each region
  int parts = 1;
  int splits = 1;          // K ranges (single region only)
};

constexpr double kStepUs256 = 0.9;      // one K step of a 256 x 256 tile in a full round
constexpr double kFillSteps = 3.0;      // pipeline fill, drain and Y store, in steps
constexpr double kLaunchUs = 3.0;       // a second launch
constexpr double kReduceBytesPerUs = 5.0e6;

TilePlan plan_tile_gemm(int M, int N, int K_aug, int num_cus, bool packed, bool allow_split) {
  const int cus = std::max(num_cus, 1);
  const int ntiles = N / 16;
  const int steps = (K_aug + kStepK - 1) / kStepK;
  auto cost = [&](const Shape& s, int cols16, int splits) {
    if (cols16 <= 0) return 0.0;
    const long tiles = static_cast<long>((M + s.bm - 1) / s.bm) * ((cols16 * 16 + s.bn - 1) / s.bn);
    const int per = (steps + splits - 1) / splits;
    const long wgs = tiles * ((steps + per - 1) / per);
    // per-step time of the busiest CU: kStepUs256 per 256 x 256 tile alone
    const double step_us = kStepUs256 * shape_cost(s, packed, wgs, cus) / 65536.0;
    double c = (per + kFillSteps) * step_us;
    if (splits > 1)   // partials written, then Y and the partials read and Y written
      c += kLaunchUs + 2.0 * ((steps + per - 1) / per) * 4.0 * M * N / kReduceBytesPerUs;
    return c;
  };
  TilePlan best;
  double best_cost = 1e300;
  static const int kSplits[] = {1, 2, 3, 4, 6, 8};
  for (const Shape& s : kShapes)
    for (int sp : kSplits) {
      if (sp > 1 && (!allow_split || sp > steps)) break;
      const double c = cost(s, ntiles, sp);
      if (c < best_cost) {
        best_cost = c;
        best = TilePlan{};
        best.shape[0] = s.id;
        best.tiles[0] = ntiles;
        best.splits = sp;
      }
    }
  for (const Shape& a : kShapes)
    for (int main16 = a.bn / 16; main16 < ntiles; main16 += a.bn / 16)
      for (const Shape& b : kShapes) {
        const double c = cost(a, main16, 1) + cost(b, ntiles - main16, 1) + kLaunchUs;
        if (c < best_cost) {
          best_cost = c;
          best = TilePlan{};
          best.shape[0] = a.id;
          best.shape[1] = b.id;
          best.tiles[0] = main16;
          best.tiles[1] = ntiles - main16;
          best.parts = 2;
        }
      }
  if (best.splits > 1) {   // the launcher's normalisation: every range non-empty
    const int per = (steps + best.splits - 1) / best.splits;
    best.splits = (steps + per - 1) / per;
  }
  return best;
}

hipError_t launch_plan(const uint8_t* Aq, const uint8_t* Asc, int M, const uint8_t* Wp,
                       const uint8_t* Wps, int N, int K_aug, float* Y, bool packed,
                       const TilePlan& plan, float* ws, hipStream_t stream) {
  int base = 0;
  for (int p = 0; p < plan.parts; ++p) {
    const hipError_t e = launch_region(Aq, Asc, M, nullptr, 1, Wp, Wps, N, K_aug, Y,
                                       plan.shape[p], packed, base, plan.tiles[p], stream,
                                       plan.splits, ws);
    if (e != hipSuccess) return e;
    base += plan.tiles[p];
  }
  return hipSuccess;
}

}  // namespace

int choose_tile_shape(int M_rows, int N, int num_cus, bool packed) {
  // One shape over all columns (grouped calls and the tuning entry).
  int best = 2;
  double best_cost = 1e300;
  for (const Shape& s : kShapes) {
    const long tiles = static_cast<long>((M_rows + s.bm - 1) / s.bm) * ((N + s.bn - 1) / s.bn);
    const double c = shape_cost(s, packed, tiles, std::max(num_cus, 1));
    if (c < best_cost) {
      best_cost = c;
      best = s.id;
    }
  }
  return best;
}

hipError_t launch_gemm_tile(const uint8_t* Aq, const uint8_t* Asc, int M,
                            const int32_t* group_offsets, int E, const uint8_t* Wp,
                            const uint8_t* Wps, int N, int K_aug, float* Y, int shape,
                            hipStream_t stream) {
  return launch_region(Aq, Asc, M, group_offsets, E, Wp, Wps, N, K_aug, Y, shape, false, 0, N / 16,
                       stream);
}

hipError_t launch_gemm_tile_packed(const uint8_t* Ap, const uint8_t* Aps, int M,
                                   const uint8_t* Wp, const uint8_t* Wps, int N, int K_aug,
                                   float* Y, int shape, hipStream_t stream) {
  return launch_region(Ap, Aps, M, nullptr, 1, Wp, Wps, N, K_aug, Y, shape, true, 0, N / 16,
                       stream);
}

// The persistent grouped kernel (128 x 128 tiles) over num_cus CUs: as many
// workgroups as fit on them at once, a multiple of the XCD count.
hipError_t launch_grouped_persist(const uint8_t* Ap, const uint8_t* Aps, int M,
                                  const int32_t* off, int E, const uint8_t* Wp,
                                  const uint8_t* Wps, int N, int K_aug, float* Y, int num_cus,
                                  hipStream_t stream) {
  const int64_t steps = (K_aug + kStepK - 1) / kStepK;
  if (!off || E < 1 || E > 64 * kXcds || num_cus < 1 ||
      static_cast<int64_t>((M + 15) / 16) * steps * 1024 >= (int64_t{1} << 31) ||
      static_cast<int64_t>(N / 16) * steps * 1024 >= (int64_t{1} << 31))
    return hipErrorInvalidValue;
  constexpr int kThreads = 256;
  auto kernel = gemm_grouped_persist_kernel<128, 128, 2, 2, 4>;
  static int per_cu = 0;   // the kernel's occupancy (gfx950 only: the same on every device)
  if (per_cu == 0) {
    int n = 0;
    const hipError_t err = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, kThreads, 0);
    if (err != hipSuccess) return err;
    per_cu = std::max(n, 1);
  }
  const int grid = std::max(kXcds, num_cus * per_cu / kXcds * kXcds);
  kernel<<<grid, kThreads, 0, stream>>>(Ap, Aps, M, off, E, Wp, Wps, N, K_aug, Y);
  return hipGetLastError();
}

// Shape of the grouped packed GEMM.  128 x 128 throughout: on the expert
// shape (~256 rows per expert, N = 2048, K + k = 832) it measured 158 us
// against 167 (256 x 256) and 220 (256 x 128), and smaller row tiles waste
// less on experts with fewer rows.
int choose_grouped_packed_shape(int rows_per_expert, int N, int K_aug, int E) {
  (void)rows_per_expert;
  (void)N;
  (void)K_aug;
  return E <= 64 * kXcds ? kShapePersist : 2;
}

hipError_t launch_grouped_gemm_tile_packed(const uint8_t* Ap, const uint8_t* Aps, int M_total,
                                           const int32_t* group_offsets, int E, const uint8_t* Wp,
                                           const uint8_t* Wps, int N, int K_aug, float* Y,
                                           int shape, int num_cus, hipStream_t stream) {
  if (shape == kShapePersist)
    return launch_grouped_persist(Ap, Aps, M_total, group_offsets, E, Wp, Wps, N, K_aug, Y,
                                  num_cus, stream);
  return launch_region(Ap, Aps, M_total, group_offsets, E, Wp, Wps, N, K_aug, Y, shape, true, 0,
                       N / 16, stream);
}

size_t tile_workspace_bytes(int M, int N, int K_aug, bool packed, int num_cus) {
  const TilePlan plan = plan_tile_gemm(M, N, K_aug, num_cus, packed, true);
  return plan.splits > 1 ? static_cast<size_t>(plan.splits - 1) * M * N * sizeof(float) : 0;
}

hipError_t launch_gemm_tile_planned(const uint8_t* Aq, const uint8_t* Asc, int M,
                                    const uint8_t* Wp, const uint8_t* Wps, int N, int K_aug,
                                    float* Y, bool packed, int num_cus, void* workspace,
                                    size_t workspace_bytes, hipStream_t stream) {
  // Split-K only with room for its partial sums and 16-byte aligned Y and
  // workspace (the reduction moves float4s); otherwise the best plan without.
  const bool aligned = (reinterpret_cast<uintptr_t>(Y) & 15u) == 0 &&
                       (reinterpret_cast<uintptr_t>(workspace) & 15u) == 0;
  const size_t need = tile_workspace_bytes(M, N, K_aug, packed, num_cus);
  const bool split = workspace && aligned && need > 0 && workspace_bytes >= need;
  return launch_plan(Aq, Asc, M, Wp, Wps, N, K_aug, Y, packed,
                     plan_tile_gemm(M, N, K_aug, num_cus, packed, split),
                     static_cast<float*>(workspace), stream);
}

hipError_t launch_gemm_tile_split(const uint8_t* Aq, const uint8_t* Asc, int M, const uint8_t* Wp,
                                  const uint8_t* Wps, int N, int K_aug, float* Y, bool packed,
                                  int shape, int splits, float* ws, hipStream_t stream) {
  return launch_region(Aq, Asc, M, nullptr, 1, Wp, Wps, N, K_aug, Y, shape, packed, 0, N / 16,
                       stream, splits, ws);
}

}  // namespace prq
