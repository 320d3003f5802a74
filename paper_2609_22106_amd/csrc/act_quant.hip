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
//     workgroups; perm and d of its 8 positions live in registers (d is given
//     in position order); the workgroup's rows are copied whole into LDS
//     while those entries load, and gathered from LDS.
//   * LDS kernel (many rows, prefill): a workgroup takes a contiguous range of
//     rows; a thread keeps the perm and d of its units in registers; each row
//     is staged into LDS with coalesced 16-byte loads (double-buffered, the
//     next row already loading into registers) and gathered from LDS.
// E2M1 encoding uses the hardware FP32->FP4 converter on exactly scaled values.
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

// Positions of a unit with their source channels packed two per register
// (K <= 16384 fits 16 bits) and their inverse scales.
struct PackedUnit {
  uint32_t src2[4];
  float d[8];
};

// rot (0-3): the pairs stored rotated, pair j = the unit's pair (j + rot) % 4
// (selects only: a run-time index into a private array would be moved to
// memory by the compiler).
__device__ __forceinline__ void load_packed_unit(const int32_t* __restrict__ perm,
                                                 const float* __restrict__ inv, int g, int K,
                                                 int u, PackedUnit* out, int rot = 0) {
  Unit t;
  load_unit(perm, inv, g, K, u, &t);
  uint32_t p[4];
  float2 q[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    p[j] = static_cast<uint32_t>(t.src[2 * j]) | (static_cast<uint32_t>(t.src[2 * j + 1]) << 16);
    q[j] = make_float2(t.d[2 * j], t.d[2 * j + 1]);
  }
  const bool r2 = rot & 2, r1 = rot & 1;
  const uint32_t a0 = r2 ? p[2] : p[0], a1 = r2 ? p[3] : p[1], a2 = r2 ? p[0] : p[2], a3 = r2 ? p[1] : p[3];
  const float2 b0 = r2 ? q[2] : q[0], b1 = r2 ? q[3] : q[1], b2 = r2 ? q[0] : q[2], b3 = r2 ? q[1] : q[3];
  out->src2[0] = r1 ? a1 : a0;
  out->src2[1] = r1 ? a2 : a1;
  out->src2[2] = r1 ? a3 : a2;
  out->src2[3] = r1 ? a0 : a3;
  const float2 c0 = r1 ? b1 : b0, c1 = r1 ? b2 : b1, c2 = r1 ? b3 : b2, c3 = r1 ? b0 : b3;
  out->d[0] = c0.x; out->d[1] = c0.y; out->d[2] = c1.x; out->d[3] = c1.y;
  out->d[4] = c2.x; out->d[5] = c2.y; out->d[6] = c3.x; out->d[7] = c3.y;
}

// Where a row's codes and scales go.  Row-major: Aq [M][K_aug/2], Asc
// [M][K_aug/32].  Packed: the MFMA-ordered layout of the packed weights with the
// rows in the place of the output features -- Ap [ceil(M/16)][S][64][16] bytes,
// entry (row block, step s, lane l) the 16 code bytes of row 16 rb + l % 16,
// K elements [128 s + 32 (l / 16), +32); Aps [ceil(M/16)][ceil(S/4)][64] uint32,
// byte j of entry (rb, q, l) the scale of the same row, 32-block
// 4 (4 q + j) + l / 16 -- so the GEMM copies both operands in whole kilobytes.
struct RowSink {
  uint8_t* arow;
  uint8_t* srow;
  __device__ void word(int v, uint32_t w) const { *reinterpret_cast<uint32_t*>(arow + 4 * v) = w; }
  __device__ void scale(int b, uint32_t c) const { srow[b] = static_cast<uint8_t>(c); }
};

struct PackedSink {
  uint8_t* code;    // Ap + (r / 16) S 1024 + (r % 16) 16
  uint8_t* sc;      // Aps + (r / 16) ceil(S/4) 256 + (r % 16) 4
  __device__ PackedSink(uint8_t* Ap, uint8_t* Aps, int r, int steps, int sgroups)
      : code(Ap + static_cast<int64_t>(r >> 4) * steps * 1024 + (r & 15) * 16),
        sc(Aps + static_cast<int64_t>(r >> 4) * sgroups * 256 + (r & 15) * 4) {}
  // unit v = 8 positions: block v / 4 (step b / 4, K part b % 4), quarter v % 4
  __device__ void word(int v, uint32_t w) const {
    const int b = v >> 2;
    *reinterpret_cast<uint32_t*>(code + (b >> 2) * 1024 + (b & 3) * 256 + (v & 3) * 4) = w;
  }
  __device__ void scale(int b, uint32_t c) const {
    const int s = b >> 2;
    sc[(s >> 2) * 256 + (b & 3) * 64 + (s & 3)] = static_cast<uint8_t>(c);
  }
};

// One row of an 8-row window of the packed layout staged in LDS: the window's
// codes as [S][4 K parts][8 slots][16 bytes] and then its scales as
// [ceil(S/4)][4 K parts][8 rows][4 bytes] -- the packed layout with the row
// block cut to the window's 8 rows, so that every (step, K part) of the window
// is 128 contiguous bytes in LDS and in global memory (its 32-byte scale runs
// likewise).  Row j's 16 bytes of code line L = 4 step + K part sit in slot
// (j + L) % 8: the 32 words a half wave writes (8 lines x 4 words of one row)
// then fall on 32 distinct banks instead of the row's 4.
struct LdsPackedSink {
  uint8_t* code;    // window codes
  uint8_t* sc;      // window scales + j 4
  int j;            // the row's place in the window
  __device__ void word(int v, uint32_t w) const {
    const int line = v >> 2;
    *reinterpret_cast<uint32_t*>(code + line * 128 + (((j + line) & 7) << 4) + (v & 3) * 4) = w;
  }
  __device__ void scale(int b, uint32_t c) const {
    const int s = b >> 2;
    sc[(s >> 2) * 128 + (b & 3) * 32 + (s & 3)] = static_cast<uint8_t>(c);
  }
};

// Quantize 8 values of a quarter block (the quad holds the whole block) and
// write the word, the scale and, for tail blocks, their copies.  t = z * 2^-e
// is exact (a power-of-two product whose magnitude stays below 8, or a
// signed zero/denormal that encodes as a signed zero either way); its E2M1
// code comes from the hardware converter at scale 1, which rounds to nearest
// even and saturates at 6 exactly like the software rule on every float32
// (checked exhaustively on the GPU).
// rs: z holds the unit's values with their pairs rotated by 4 - rs (pair j =
// pair (j + 4 - rs) % 4); the code word is rotated back by rs bytes.
template <class Sink>
__device__ __forceinline__ void quantize_store(const float (&z)[8], int u, int tail_unit0,
                                               int copy_units, int copy_blocks, const Sink& out,
                                               int rs = 0) {
  float amax = 0.0f;
#pragma unroll
  for (int j = 0; j < 8; ++j) amax = fmaxf(amax, fabsf(z[j]));
  amax = dev::quad_max(amax);
  const uint32_t code = dev::e8m0_code(amax);
  const float mul = dev::e8m0_reciprocal(code);
  // four converts, each writing its pair into one byte of the word
  uint32_t w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, z[0] * mul, z[1] * mul, 1.0f, 0);
  w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w, z[2] * mul, z[3] * mul, 1.0f, 1);
  w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w, z[4] * mul, z[5] * mul, 1.0f, 2);
  w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w, z[6] * mul, z[7] * mul, 1.0f, 3);
  if (rs) w = __builtin_amdgcn_alignbyte(w, w, rs);   // byte i -> byte (i - rs) mod 4
  out.word(u, w);
  if ((u & 3) == 0) out.scale(u >> 2, code);
  if (u >= tail_unit0) {  // online copy of the quantized tail and its scales
    out.word(u + copy_units, w);
    if ((u & 3) == 0) out.scale((u >> 2) + copy_blocks, code);
  }
}

// Packed layout padding of one row past K_aug: zero codes up to the end of
// the last K step, scale byte 127 up to the end of the last group of four
// steps (fewer than 16 blocks; the row's thread with unit u0 writes blocks
// nb + u0, nb + u0 + units, ...).
template <class Sink>
__device__ __forceinline__ void pad_row_tail(const Sink& out, int u0, int units, int nb,
                                             int steps, int sgroups) {
  for (int t = u0; t < 16; t += units) {
    const int b = nb + t;
    if (b < sgroups * 16) {
      out.scale(b, 127u);
      if (b < steps * 4)
#pragma unroll
        for (int q = 0; q < 4; ++q) out.word(4 * b + q, 0u);
    }
  }
}

#define PRQ_ROWS_GPTR(p) ((const __attribute__((address_space(1))) void*)(p))
#define PRQ_ROWS_LPTR(p) ((__attribute__((address_space(3))) void*)(p))

// Few rows (decode).  A workgroup owns kRowsThreads units (quarter blocks) of
// `rows_per_wg` rows.  Its rows are copied whole into LDS by direct
// global->LDS copies issued at once, in flight together with the units'
// permutation entries and inverse scales (the copies do not depend on them),
// so a cold call pays one memory round trip before the gather instead of
// two (permutation, then the rows at the permuted channels); the gather then
// reads LDS.
template <bool kGrouped, bool kPacked>
__global__ __launch_bounds__(kRowsThreads) void act_quant_rows_kernel(
    const uint16_t* __restrict__ X, int64_t ld_x, int M, int K, int k_tail,
    const float* __restrict__ inv, const int32_t* __restrict__ perm,
    const int32_t* __restrict__ offsets, int G, int rows_per_wg, uint8_t* __restrict__ Aq,
    uint8_t* __restrict__ Asc) {
  extern __shared__ __align__(16) unsigned char rows_lds[];   // [rows_per_wg][pitch]
  const int units = K >> 3;
  const int u = blockIdx.x * kRowsThreads + threadIdx.x;
  const int r0 = blockIdx.y * rows_per_wg;
  const int r1 = min(M, r0 + rows_per_wg);
  const int n = r1 - r0;
  const int k_aug = K + k_tail;
  const int64_t row_bytes = k_aug >> 1;
  const int nb = k_aug >> 5;
  const int steps = (k_aug + 127) >> 7;
  const int sgroups = (steps + 3) >> 2;
  if (kPacked && n <= 0) {
    // Workgroup rows past M (packed output, up to the end of the last 16-row
    // block): zero codes and scale byte 127 over the whole padded row.
    if (u >= units) return;
    for (int r = r0; r < r0 + rows_per_wg; ++r) {
      const PackedSink ps(Aq, Asc, r, steps, sgroups);
      ps.word(u, 0u);
      if ((u & 3) == 0) ps.scale(u >> 2, 127u);
      if (u >= (K - k_tail) >> 3) {
        ps.word(u + (k_tail >> 3), 0u);
        if ((u & 3) == 0) ps.scale((u >> 2) + (k_tail >> 5), 127u);
      }
      pad_row_tail(ps, u, units, nb, steps, sgroups);
    }
    return;
  }
  const int xb = 2 * K;                               // bytes of a row of X
  const int chunks = (xb + 1023) >> 10;
  const int pitch = chunks * 1024;
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  const int lane = threadIdx.x & 63;
  // 1. The rows, 1 KB per wave copy (lanes past the row copy its start into
  //    the pad, never read).
  for (int i = wave; i < n * chunks; i += kRowsThreads / 64) {
    const int rr = i / chunks, c = i - rr * chunks;
    const int off = c * 1024 + lane * 16;
    const uint8_t* src = reinterpret_cast<const uint8_t*>(X + static_cast<int64_t>(r0 + rr) * ld_x);
    __builtin_amdgcn_global_load_lds(PRQ_ROWS_GPTR(src + (off < xb ? off : 0)),
                                     PRQ_ROWS_LPTR(rows_lds + rr * pitch + c * 1024), 16, 0, 0);
  }
  // 2. The unit's permutation entries and inverse scales meanwhile.
  const bool active = u < units;                      // K/8 is a multiple of 4: quads agree
  const int uc = active ? u : units - 1;
  // Pairs rotated by (lane / 8) % 4 dwords against LDS bank conflicts, as in
  // the copy kernel below.
  const int rot = (threadIdx.x >> 3) & 3;
  const int rs = (4 - rot) & 3;
  PackedUnit un;
  int cur_g = kGrouped ? dev::find_group(offsets, G, r0) : 0;
  load_packed_unit(perm, inv, cur_g, K, uc, &un, rot);
  __builtin_amdgcn_s_waitcnt((0x7 << 4) | (0xF << 8));   // vmcnt(0): copies and entries
  __syncthreads();
  if (!active) return;
  // 3. Gather from LDS, quantize, store.
  for (int rr = 0; rr < n; ++rr) {
    const int r = r0 + rr;
    if (kGrouped) {
      const int g = dev::find_group(offsets, G, r);
      if (g != cur_g) {
        load_packed_unit(perm, inv, g, K, uc, &un, rot);
        cur_g = g;
      }
    }
    const uint16_t* xr = reinterpret_cast<const uint16_t*>(rows_lds + rr * pitch);
    float z[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t sp = un.src2[e];
      z[2 * e] = __uint_as_float(static_cast<uint32_t>(xr[sp & 0xFFFFu]) << 16) * un.d[2 * e];
      z[2 * e + 1] = __uint_as_float(static_cast<uint32_t>(xr[sp >> 16]) << 16) * un.d[2 * e + 1];
    }
    if constexpr (kPacked) {
      const PackedSink ps(Aq, Asc, r, steps, sgroups);
      quantize_store(z, u, (K - k_tail) >> 3, k_tail >> 3, k_tail >> 5, ps, rs);
      pad_row_tail(ps, u, units, nb, steps, sgroups);
    } else {
      quantize_store(z, u, (K - k_tail) >> 3, k_tail >> 3, k_tail >> 5,
                     RowSink{Aq + static_cast<int64_t>(r) * row_bytes, Asc + static_cast<int64_t>(r) * nb},
                     rs);
    }
  }
}

// Rows handled together by one pass of the LDS kernel: one when a row has at
// least as many units as the workgroup has threads, else as many whole rows
// as fit (a thread then owns one unit of one of them).
__host__ __device__ inline int lds_rows_per_pass(int units) {
  return units >= kLdsThreads ? 1 : kLdsThreads / units;
}

inline size_t lds_kernel_bytes(int K) {
  const int units = K >> 3;
  return static_cast<size_t>(lds_rows_per_pass(units)) * units * 16 * 2;   // two staged passes
}

// Many rows.  A workgroup takes a contiguous range of rows, a pass of
// lds_rows_per_pass(K/8) rows at a time.  Thread t owns the units t + 512 j
// of the pass (kUnits of them; with several rows per pass, one): flat index f
// -> row f / units, unit f % units, the same row for all of a thread's units.
// Their source channels and inverse scales stay in registers, reloaded only
// when the thread's row enters another expert.  Passes are staged in LDS with
// coalesced 16-byte loads into two alternating buffers: pass i+1 is loaded
// into registers while pass i is quantized, and one barrier per pass suffices
// -- a thread writes pass i into buffer i&1 only after the barrier of pass
// i-1, which every thread passes only after it finished reading pass i-2 from
// that buffer.
template <bool kGrouped, int kUnits, bool kPacked>
__global__ __launch_bounds__(kLdsThreads) void act_quant_lds_kernel(
    const uint16_t* __restrict__ X, int64_t ld_x, int M, int K, int k_tail,
    const float* __restrict__ inv, const int32_t* __restrict__ perm,
    const int32_t* __restrict__ offsets, int G, int rows_per_wg, uint8_t* __restrict__ Aq,
    uint8_t* __restrict__ Asc) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x;
  const int units = K >> 3;                       // units (= uint4 vectors) per row
  const int rpp = lds_rows_per_pass(units);
  const int pass_vecs = rpp * units;              // <= max(units, 512) <= 2048
  uint4* const buf0 = reinterpret_cast<uint4*>(smem);
  uint4* const buf1 = buf0 + pass_vecs;
  const int r0 = blockIdx.x * rows_per_wg;
  const int r1 = min(M, r0 + rows_per_wg);
  const int k_aug = K + k_tail;
  const int64_t row_bytes = k_aug >> 1;
  const int nb = k_aug >> 5;
  const int tail_unit0 = (K - k_tail) >> 3;
  const int steps = (k_aug + 127) >> 7;
  const int sgroups = (steps + 3) >> 2;

  // Staged vectors of this thread: v = tid + 512 i -> (row offset, vector),
  // as named registers (an array here ends up in scratch when its copy loop is
  // not fully unrolled).
  static_assert(kMaxRowVec == 4, "four named row vectors");
  int vro[4];
  int64_t voff[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int v = tid + i * kLdsThreads;
    vro[i] = v < pass_vecs ? v / units : rpp;     // rpp: never a valid row offset
    voff[i] = v < pass_vecs ? static_cast<int64_t>(vro[i]) * ld_x + (v - vro[i] * units) * 8 : 0;
  }
  // A pass holds at most max(units, 512) vectors, kUnits (= ceil(units / 512))
  // per thread: vectors past kUnits are never loaded (short rows then hold one
  // vector register set instead of four: 96 -> 72 VGPRs, packed).
  uint4 p0 = {}, p1 = {}, p2 = {}, p3 = {};
  auto prefetch = [&](int rb) {
    const int lim = min(rpp, r1 - rb);           // rows of this pass
    const uint16_t* xb = X + static_cast<int64_t>(rb) * ld_x;
    if (vro[0] < lim) p0 = *reinterpret_cast<const uint4*>(xb + voff[0]);
    if (kUnits > 1 && vro[1] < lim) p1 = *reinterpret_cast<const uint4*>(xb + voff[1]);
    if (kUnits > 2 && vro[2] < lim) p2 = *reinterpret_cast<const uint4*>(xb + voff[2]);
    if (kUnits > 3 && vro[3] < lim) p3 = *reinterpret_cast<const uint4*>(xb + voff[3]);
  };
  if (r0 < r1) prefetch(r0);

  const int ro = tid / units;                     // this thread's row within a pass
  const int u0 = tid - ro * units;                // its first unit
  // Pairs rotated by (lane / 8) % 4 dwords against LDS bank conflicts (the
  // rows of a pass lie back to back: lanes still read consecutive 16-byte
  // stretches), as in the copy kernel below.
  const int rot = (tid >> 3) & 3;
  const int rs = (4 - rot) & 3;
  PackedUnit un[kUnits];
  int cur_g = -1;
  dev::GroupCursor gc;   // this thread's rows only increase
  int pass = 0;
  for (int rb = r0; rb < r1; rb += rpp, ++pass) {
    uint4* const sb = (pass & 1) ? buf1 : buf0;
    if (tid < pass_vecs) sb[tid] = p0;
    if (kUnits > 1 && tid + kLdsThreads < pass_vecs) sb[tid + kLdsThreads] = p1;
    if (kUnits > 2 && tid + 2 * kLdsThreads < pass_vecs) sb[tid + 2 * kLdsThreads] = p2;
    if (kUnits > 3 && tid + 3 * kLdsThreads < pass_vecs) sb[tid + 3 * kLdsThreads] = p3;
    if (rb + rpp < r1) prefetch(rb + rpp);       // in flight while this pass is quantized
    __syncthreads();

    const int r = rb + ro;
    if (ro < rpp && r < r1) {                     // quad-uniform: units is a multiple of 4
      const int g = kGrouped ? gc.at(offsets, G, r) : 0;
      if (g != cur_g) {
#pragma unroll
        for (int j = 0; j < kUnits; ++j) {
          const int u = u0 + j * kLdsThreads;
          if (u < units) load_packed_unit(perm, inv, g, K, u, &un[j], rot);
        }
        cur_g = g;
      }
      const uint16_t* row = reinterpret_cast<const uint16_t*>(sb) + static_cast<int64_t>(ro) * K;
      const RowSink rsink{Aq + static_cast<int64_t>(r) * row_bytes, Asc + static_cast<int64_t>(r) * nb};
      const PackedSink psink(Aq, Asc, r, steps, sgroups);
      if constexpr (kPacked) pad_row_tail(psink, u0, units, nb, steps, sgroups);
#pragma unroll
      for (int j = 0; j < kUnits; ++j) {
        const int u = u0 + j * kLdsThreads;
        if (u < units) {
          float z[8];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const uint32_t sp = un[j].src2[e];
            z[2 * e] = __uint_as_float(static_cast<uint32_t>(row[sp & 0xFFFFu]) << 16) * un[j].d[2 * e];
            z[2 * e + 1] = __uint_as_float(static_cast<uint32_t>(row[sp >> 16]) << 16) * un[j].d[2 * e + 1];
          }
          if constexpr (kPacked)
            quantize_store(z, u, tail_unit0, k_tail >> 3, k_tail >> 5, psink, rs);
          else
            quantize_store(z, u, tail_unit0, k_tail >> 3, k_tail >> 5, rsink, rs);
        }
      }
    }
  }
  // Packed layout: the workgroup with the last row also fills the rows of the
  // last 16-row block past M (zero codes, scale byte 127).
  if constexpr (kPacked) {
    if (r0 < r1 && r1 == M) {
      for (int r = M; r < ((M + 15) & ~15); ++r) {
        const PackedSink psink(Aq, Asc, r, steps, sgroups);
        for (int v = tid; v < steps * 16; v += kLdsThreads) psink.word(v, 0u);
        for (int b = tid; b < sgroups * 16; b += kLdsThreads) psink.scale(b, 127u);
      }
    }
  }
}

// Many rows, rows copied by direct global->LDS loads.  A workgroup takes a
// contiguous range of rows and runs them through kNS LDS stages (one row each).
// Two copy waves issue the row copies, kNS - 2 rows in flight beyond the one
// being quantized, with one constant wait per row; eight compute waves hold
// their units' source channels and inverse scales in registers and quantize the
// staged row.  Stores count in the same memory counter as loads, so the waves
// that store the output are not the ones that wait for the copies.  Per row i:
// the copy waves wait for their copies of row i, every wave passes one bare
// barrier (the compute waves having finished reading row i-1, whose stage the
// copy waves then refill with row i+kNS-1), the compute waves quantize row i.
// The copies are issued as inline assembly: the compiler then sees no
// direct-to-LDS write that the compute waves' stage reads could alias (it would
// make them wait for all their outstanding stores); their ordering is the copy
// waves' explicit wait and the barrier.
// Packed output with kOut > 0: a row's 16-byte code pieces lie 256 bytes apart
// in the packed layout, so written straight away each 128-byte line takes eight
// partial writes.  The compute waves instead quantize into an LDS window of 8
// rows (LdsPackedSink) and, once a row opens the next window (after the row
// barrier, so every wave's writes are in), copy the window out in whole lines
// and pass a second barrier (every wave in step) before they refill it.
#define PRQ_LPTR(p) ((__attribute__((address_space(3))) void*)(p))

constexpr int kCopyWaves = 2;
constexpr int kComputeThreads = 512;
constexpr int kDmaThreads = kComputeThreads + kCopyWaves * 64;

// s_waitcnt: vmcnt(n) with lgkmcnt(0) (n = 63: LDS only).
template <int n>
__device__ __forceinline__ void wait_vmcnt_lgkm0() {
  static_assert(n >= 0 && n < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((n & 0xF) | ((n >> 4) << 14) | (0x7 << 4));
}

// One direct global->LDS copy of 16 bytes per lane: lane l's 16 bytes at src
// land at LDS byte lds + 16 l (lds: wave-uniform LDS address, through M0).
__device__ __forceinline__ void lds_copy16(const void* src, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(src), "s"(lds)
               : "memory", "m0");
}

template <bool kGrouped, bool kPacked, int kStage, int kNS, int kUnits, int kOut>
__global__ __launch_bounds__(kDmaThreads) void act_quant_dma_kernel(
    const uint16_t* __restrict__ X, int64_t ld_x, int M, int K, int k_tail,
    const float* __restrict__ inv, const int32_t* __restrict__ perm,
    const int32_t* __restrict__ offsets, int G, int rows_per_wg, uint8_t* __restrict__ Aq,
    uint8_t* __restrict__ Asc) {
  static_assert(kNS >= 3 && kNS <= 8, "stages");
  constexpr int kCpw = kStage / 1024 / kCopyWaves;   // copies per copy wave per row
  static_assert(kCpw * kCopyWaves * 1024 == kStage, "stage of whole copy rounds");
  static_assert((kNS - 2) * kCpw < 64, "vmcnt");
  constexpr bool kWindow = kPacked && kOut > 0;   // host check: 512 S + 128 ceil(S/4) <= kOut
  __shared__ __align__(16) uint8_t stg[kNS * kStage];
  __shared__ __align__(16) uint8_t win[kWindow ? kOut : 16];
  const int r0 = blockIdx.x * rows_per_wg;
  const int r1 = min(M, r0 + rows_per_wg);
  if (r0 >= r1) return;                            // uniform
  const int n = r1 - r0;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const bool copier = wave >= kComputeThreads / 64;
  const int cw = wave - kComputeThreads / 64;      // copy wave index (copiers)
  const int row_bytes_x = 2 * K;
  const int chunks = (row_bytes_x + 1023) >> 10;   // <= kStage / 1024 (host check)
  const int k_aug = K + k_tail;
  const int64_t row_bytes = k_aug >> 1;
  const int nb = k_aug >> 5;
  const int tail_unit0 = (K - k_tail) >> 3;
  const int steps = (k_aug + 127) >> 7;
  const int sgroups = (steps + 3) >> 2;
  const int units = K >> 3;
  const uint32_t stg_lds = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(PRQ_LPTR(stg)));

  // Row i of the range into its stage (copy waves; i clamped into the range,
  // lanes past the row read its start into the stage's pad).
  auto copy_row = [&](int i) {
    const uint8_t* src = reinterpret_cast<const uint8_t*>(X + static_cast<int64_t>(r0 + min(i, n - 1)) * ld_x);
    const uint32_t st = stg_lds + static_cast<uint32_t>(i % kNS) * kStage;
#pragma unroll
    for (int j = 0; j < kCpw; ++j) {
      const int c = min(cw + j * kCopyWaves, chunks - 1);
      const int off = c * 1024 + lane * 16;
      lds_copy16(src + (off < row_bytes_x ? off : 0), __builtin_amdgcn_readfirstlane(st + c * 1024));
    }
  };

  PackedUnit un[kUnits];
  int cur_g = -1;
  // A unit's 8 values are gathered two bytes at a time from its 16-byte
  // stretch of the row; the LDS serves half a wave per pass over 32 banks, so
  // lanes 8 units apart (128 bytes) would hit the same banks (4 lanes per
  // bank).  Each lane instead takes its pairs rotated by rot = (lane / 8) % 4
  // dwords (fixed when the units are loaded; the code word rotated back by one
  // byte-align): a half wave's reads then cover 32 distinct banks.  (Rotating
  // by the unit's first channel instead, which follows the shifts the
  // selected channels cause, measured no better.)
  const int rot = (lane >> 3) & 3;
  const int rs = (4 - rot) & 3;
  // (Re)load the units' permutation entries and inverse scales, then wait for
  // them right here: later uses then see nothing outstanding.
  auto load_units = [&](int g) {
#pragma unroll
    for (int j = 0; j < kUnits; ++j) {
      const int u = min(tid + j * kComputeThreads, units - 1);
      load_packed_unit(perm, inv, g, K, u, &un[j], rot);
    }
    __builtin_amdgcn_s_waitcnt((0x7 << 4) | (0xF << 8));   // vmcnt(0)
    cur_g = g;
  };
  dev::GroupCursor gc;
  if (!copier) load_units(kGrouped ? gc.at(offsets, G, r0) : 0);

  // Rows [lo, hi) of the window of rows [w0, w0 + 8) from LDS to the packed
  // layout (compute waves): 16-byte code pieces, consecutive threads on
  // consecutive pieces of one 128-byte line; 4-byte scale pieces likewise.
  uint8_t* const win_sc = win + steps * 512;
  auto flush = [&](int w0, int lo, int hi) {
    const int j = tid & 7;                          // the thread's row in the window, fixed
    if (j < lo - w0 || j >= hi - w0) return;
    uint8_t* const gcode = Aq + static_cast<int64_t>(w0 >> 4) * steps * 1024 + (w0 & 8) * 16;
    for (int c = tid; c < steps * 32; c += kComputeThreads)   // line c / 8, row j (slot rotated)
      *reinterpret_cast<uint4*>(gcode + (c >> 3) * 256 + j * 16) =
          *reinterpret_cast<const uint4*>(win + (c >> 3) * 128 + (((j + (c >> 3)) & 7) << 4));
    uint8_t* const gsc = Asc + static_cast<int64_t>(w0 >> 4) * sgroups * 256 + (w0 & 8) * 4;
    for (int e = tid; e < sgroups * 32; e += kComputeThreads)
      *reinterpret_cast<uint32_t*>(gsc + (e >> 3) * 64 + j * 4) =
          *reinterpret_cast<const uint32_t*>(win_sc + e * 4);
  };

  if (copier)
    for (int i = 0; i < kNS - 1; ++i) copy_row(i);
  for (int i = 0; i < n; ++i) {
    const int r = r0 + i;
    const bool window_out = kWindow && i > 0 && (r & 7) == 0;   // uniform
    if (copier) {
      wait_vmcnt_lgkm0<(kNS - 2) * kCpw>();         // row i has landed
      __builtin_amdgcn_s_barrier();
      copy_row(i + kNS - 1);                        // into the stage of row i-1
      if (window_out) __builtin_amdgcn_s_barrier();
      continue;
    }
    wait_vmcnt_lgkm0<63>();                         // this wave's LDS reads of row i-1 (and writes)
    __builtin_amdgcn_s_barrier();
    if (window_out) {                               // the window of rows r-8..r-1 is complete
      flush(r - 8, max(r0, r - 8), r);
      wait_vmcnt_lgkm0<63>();
      __builtin_amdgcn_s_barrier();
    }
    if (kGrouped) {   // a load only when the row leaves its group
      const int g = gc.at(offsets, G, r);
      if (g != cur_g) load_units(g);
    }
    const uint16_t* row = reinterpret_cast<const uint16_t*>(stg + (i % kNS) * kStage);
    const RowSink rsink{Aq + static_cast<int64_t>(r) * row_bytes, Asc + static_cast<int64_t>(r) * nb};
    const PackedSink psink(Aq, Asc, r, steps, sgroups);
    const LdsPackedSink wsink{win, win_sc + (r & 7) * 4, r & 7};
    if constexpr (kWindow) pad_row_tail(wsink, tid, units, nb, steps, sgroups);
    else if constexpr (kPacked) pad_row_tail(psink, tid, units, nb, steps, sgroups);
    // Units below the last always exist (the host picks kUnits = ceil(units /
    // kComputeThreads)): no guard, so their LDS gathers can all be in flight
    // together; the last unit is guarded (quad-uniform: units % 4 == 0).
#pragma unroll
    for (int j = 0; j < kUnits; ++j) {
      const int u = tid + j * kComputeThreads;
      if (j + 1 < kUnits || u < units) {
        float z[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t sp = un[j].src2[e];
          z[2 * e] = __uint_as_float(static_cast<uint32_t>(row[sp & 0xFFFFu]) << 16) * un[j].d[2 * e];
          z[2 * e + 1] = __uint_as_float(static_cast<uint32_t>(row[sp >> 16]) << 16) * un[j].d[2 * e + 1];
        }
        if constexpr (kWindow)
          quantize_store(z, u, tail_unit0, k_tail >> 3, k_tail >> 5, wsink, rs);
        else if constexpr (kPacked)
          quantize_store(z, u, tail_unit0, k_tail >> 3, k_tail >> 5, psink, rs);
        else
          quantize_store(z, u, tail_unit0, k_tail >> 3, k_tail >> 5, rsink, rs);
      }
    }
  }
  if (copier) __builtin_amdgcn_s_waitcnt((0x7 << 4) | (0xF << 8));   // no copy outlives the workgroup
  if constexpr (kWindow) {   // the last (possibly partial) window: every wave passes the barrier
    if (!copier) wait_vmcnt_lgkm0<63>();
    __builtin_amdgcn_s_barrier();
    const int w0 = (r1 - 1) & ~7;
    if (!copier) flush(w0, max(r0, w0), r1);
  }

  // Packed layout: the workgroup with the last row also fills the rows of the
  // last 16-row block past M (zero codes, scale byte 127).
  if constexpr (kPacked) {
    if (r1 == M && !copier) {
      for (int r = M; r < ((M + 15) & ~15); ++r) {
        const PackedSink psink(Aq, Asc, r, steps, sgroups);
        for (int v = tid; v < steps * 16; v += kComputeThreads) psink.word(v, 0u);
        for (int b = tid; b < sgroups * 16; b += kComputeThreads) psink.scale(b, 127u);
      }
    }
  }
}

template <bool kGrouped, int kUnits, bool kPacked = false>
void launch_lds(dim3 grid, size_t lds, hipStream_t stream, const uint16_t* X, int64_t ld_x,
                int M, int K, int k_tail, const float* inv, const int32_t* perm,
                const int32_t* offsets, int G, int rows_per_wg, uint8_t* Aq, uint8_t* Asc) {
  act_quant_lds_kernel<kGrouped, kUnits, kPacked><<<grid, kLdsThreads, lds, stream>>>(
      X, ld_x, M, K, k_tail, inv, perm, offsets, G, rows_per_wg, Aq, Asc);
}

// Rows per workgroup of the LDS kernel: two workgroups per CU, a whole number
// of passes each, contiguous row ranges (inside one expert for most rows).
int lds_rows_per_wg(int M, int units, int num_cus) {
  const int rpp = lds_rows_per_pass(units);
  const int target = std::max(1, num_cus * 2);
  int rows_per_wg = std::max(1, (M + target - 1) / target);
  return (rows_per_wg + rpp - 1) / rpp * rpp;
}

// Stage classes of the copy kernel by row length (2K bytes): stage bytes, stages,
// units per compute thread (K/8 units over 512 threads), LDS bytes of the packed
// output window (each workgroup's LDS within 160 KiB / workgroups per CU; the
// window holds K + k up to 2K in the first three classes, up to 14336 in the
// fourth, 15360 in the fifth, never in the last).  window: 0 = where it pays,
// 1 = where it fits, 2 = never (packed output stored directly).  It pays on
// rows long enough for one workgroup per CU with many rows per workgroup: a
// row block's lines then stay partial in L2 too long (cold, M = 8192 x 9728:
// 56.5 -> 42.5 us, M = 4096: 29.5 -> 23.7; M = 8192 x 6144: 32.3 -> 28.7);
// with short rows they complete in L2 anyway and the window's last flush is
// pure latency (M = 4096 x 2560: 8.5 -> 12.3 us, x 4096: 10.4 -> 13.9; M =
// 512 x 9728, two rows each: 6.8 -> 8.1).  The 20480-byte class (five stages)
// fits the 19456-byte down_proj row; against 24576-byte stages (four) it
// measured the same.
static_assert(kComputeThreads == 512, "stage classes assume 512 compute threads");
constexpr int kWindowBytes[6] = {17408, 34816, 69632, 61440, 65536, 0};
constexpr int cls_of(int stage) {
  return stage <= 4096 ? 0 : stage <= 8192 ? 1 : stage <= 16384 ? 2 : stage <= 20480 ? 3 : stage <= 24576 ? 4 : 5;
}

int packed_window_bytes(int K_aug) {
  const int steps = (K_aug + 127) / 128;
  return steps * 512 + (steps + 3) / 4 * 128;
}

template <bool kGrouped, bool kPacked>
hipError_t launch_dma(const uint16_t* X, int64_t ld_x, int M, int K, int k_tail, const float* inv,
                      const int32_t* perm, const int32_t* offsets, int G, uint8_t* Aq, uint8_t* Asc,
                      int num_cus, hipStream_t stream, int window = 0) {
  const int rb = 2 * K;
  const int per_cu = rb <= 8192 ? 2 : 1;           // workgroups a CU holds (LDS)
  const int target = std::max(1, num_cus * per_cu);
  const int rows_per_wg = std::max(1, (M + target - 1) / target);
  const dim3 grid((M + rows_per_wg - 1) / rows_per_wg);
  const int cls = cls_of(rb);
  const bool pays = per_cu == 1 && rows_per_wg >= 16;
  const bool win = kPacked && window != 2 && (window == 1 || pays) &&
                   packed_window_bytes(K + k_tail) <= kWindowBytes[cls];
#define PRQ_DMA_OUT(STAGE, NS, U, OUT)                                                            \
  act_quant_dma_kernel<kGrouped, kPacked, STAGE, NS, U, OUT><<<grid, kDmaThreads, 0, stream>>>(  \
      X, ld_x, M, K, k_tail, inv, perm, offsets, G, rows_per_wg, Aq, Asc)
#define PRQ_DMA(STAGE, NS, U)                                                                     \
  do {                                                                                            \
    if (kPacked && win)                                                                           \
      PRQ_DMA_OUT(STAGE, NS, U, (kPacked ? kWindowBytes[cls_of(STAGE)] : 0));                     \
    else                                                                                          \
      PRQ_DMA_OUT(STAGE, NS, U, 0);                                                               \
  } while (0)
  // kUnits = ceil(K / 8 / 512) exactly: every unit but the last exists.
  // Four stages in every class but 20480 bytes (five): with all of a
  // workgroup's rows requested at once (up to 8 stages) the copies of the
  // whole launch exceed X itself and the short-row cases ran a third slower
  // (M = 4096: K = 2560 11.8 -> 8.4 us, K = 4096 14.4 -> 11.1 us packed; K =
  // 9728 unchanged).
  if (rb <= 4096) PRQ_DMA(4096, 4, 1);
  else if (rb <= 8192) PRQ_DMA(8192, 4, 1);
  else if (rb <= 16384) PRQ_DMA(16384, 4, 2);
  else if (rb <= 20480) PRQ_DMA(20480, 5, 3);
  else if (rb <= 24576) PRQ_DMA(24576, 4, 3);
  else PRQ_DMA_OUT(32768, 4, 4, 0);
#undef PRQ_DMA
#undef PRQ_DMA_OUT
  return hipGetLastError();
}

}  // namespace

hipError_t launch_act_quant(const uint16_t* X, int64_t ld_x, int M, int K, int k_tail,
                            const float* inv_scale_pos, const int32_t* perm,
                            const int32_t* group_offsets, int G, uint8_t* Aq, uint8_t* Asc,
                            int num_cus, hipStream_t stream) {
  return launch_act_quant_kernel(X, ld_x, M, K, k_tail, inv_scale_pos, perm, group_offsets, G, Aq,
                                 Asc, num_cus, 0, stream);
}

// Dynamic LDS of the few-rows kernel above the 64 KiB default (up to four
// staged rows of K = 16384), set once per instantiation.
template <bool kGrouped, bool kPacked>
void set_rows_lds_limit() {
  static std::once_flag once;
  std::call_once(once, [] {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&act_quant_rows_kernel<kGrouped, kPacked>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, 4 * 32768);
    (void)hipGetLastError();
  });
}

// Few rows into the packed layout: one row per workgroup row, and workgroup
// rows up to the end of the last 16-row block that write its padding rows.
hipError_t launch_rows_packed(const uint16_t* X, int64_t ld_x, int M, int K, int k_tail,
                              const float* inv, const int32_t* perm, const int32_t* off, int G,
                              uint8_t* Ap, uint8_t* Aps, hipStream_t stream) {
  const int units = K >> 3;
  const int pitch = (2 * K + 1023) / 1024 * 1024;
  const dim3 grid((units + kRowsThreads - 1) / kRowsThreads, (M + 15) / 16 * 16);
  if (off) {
    set_rows_lds_limit<true, true>();
    act_quant_rows_kernel<true, true><<<grid, kRowsThreads, pitch, stream>>>(
        X, ld_x, M, K, k_tail, inv, perm, off, G, 1, Ap, Aps);
  } else {
    set_rows_lds_limit<false, true>();
    act_quant_rows_kernel<false, true><<<grid, kRowsThreads, pitch, stream>>>(
        X, ld_x, M, K, k_tail, inv, perm, nullptr, 1, 1, Ap, Aps);
  }
  return hipGetLastError();
}

hipError_t launch_act_quant_kernel(const uint16_t* X, int64_t ld_x, int M, int K, int k_tail,
                                   const float* inv_scale_pos, const int32_t* perm,
                                   const int32_t* group_offsets, int G, uint8_t* Aq, uint8_t* Asc,
                                   int num_cus, int kernel, hipStream_t stream) {
  const bool grouped = group_offsets && G > 1;
  const int units = K >> 3;
  if (kernel == 1 || (kernel == 0 && M <= 64)) {
    // Few rows: spread the positions over workgroups, one row per workgroup
    // row up to 64 rows (measured on the 9728 -> 9984 down_proj row against 16
    // row chunks: M = 32 3.36 -> 2.77 us, M = 64 4.67 -> 3.22 warm, 3.90 -> 3.24
    // and 5.23 -> 3.82 after an L2-evicting fill; M = 1 and 8 unchanged), else
    // (forced for more rows) at most ~16 row chunks; a workgroup's rows are
    // staged whole in LDS (at most 4 rows of 32 KiB).
    const int pitch = (2 * K + 1023) / 1024 * 1024;
    const int rows_per_wg = M <= 64 ? 1 : std::max(1, std::min((M + 15) / 16, 4 * 32768 / pitch));
    const dim3 grid((units + kRowsThreads - 1) / kRowsThreads, (M + rows_per_wg - 1) / rows_per_wg);
    const size_t lds = static_cast<size_t>(std::min(rows_per_wg, M)) * pitch;
    if (grouped) {
      set_rows_lds_limit<true, false>();
      act_quant_rows_kernel<true, false><<<grid, kRowsThreads, lds, stream>>>(
          X, ld_x, M, K, k_tail, inv_scale_pos, perm, group_offsets, G, rows_per_wg, Aq, Asc);
    } else {
      set_rows_lds_limit<false, false>();
      act_quant_rows_kernel<false, false><<<grid, kRowsThreads, lds, stream>>>(
          X, ld_x, M, K, k_tail, inv_scale_pos, perm, nullptr, 1, rows_per_wg, Aq, Asc);
    }
    return hipGetLastError();
  }
  const int32_t* goff = grouped ? group_offsets : nullptr;
  // Long rows (K >= 2048): rows copied into LDS stages; shorter rows: several
  // rows per pass of the register-staged kernel (measured faster at K = 768).
  if (kernel == 3 || (kernel == 0 && K >= 2048)) {
    if (grouped)
      return launch_dma<true, false>(X, ld_x, M, K, k_tail, inv_scale_pos, perm, goff, G, Aq, Asc,
                                     num_cus, stream);
    return launch_dma<false, false>(X, ld_x, M, K, k_tail, inv_scale_pos, perm, nullptr, 1, Aq, Asc,
                                    num_cus, stream);
  }
  // At most 2 * 2048 * 16 bytes = 64 KiB of LDS: within the default limit.
  const size_t lds = lds_kernel_bytes(K);
  const int per_thread = (units + kLdsThreads - 1) / kLdsThreads;   // 1..4 (K <= 16384)
  const int rows_per_wg = lds_rows_per_wg(M, units, num_cus);
  const dim3 grid((M + rows_per_wg - 1) / rows_per_wg);
  const int32_t* off = grouped ? group_offsets : nullptr;
  const int g = grouped ? G : 1;
#define PRQ_LDS_CASE(n)                                                                     \
  case n:                                                                                   \
    if (grouped)                                                                            \
      launch_lds<true, n>(grid, lds, stream, X, ld_x, M, K, k_tail, inv_scale_pos, perm, off, \
                          g, rows_per_wg, Aq, Asc);                                         \
    else                                                                                    \
      launch_lds<false, n>(grid, lds, stream, X, ld_x, M, K, k_tail, inv_scale_pos, perm,   \
                           off, g, rows_per_wg, Aq, Asc);                                   \
    break;
  switch (per_thread) {
    PRQ_LDS_CASE(1)
    PRQ_LDS_CASE(2)
    PRQ_LDS_CASE(3)
    default:
      PRQ_LDS_CASE(4)
  }
#undef PRQ_LDS_CASE
  return hipGetLastError();
}

hipError_t launch_act_quant_packed(const uint16_t* X, int64_t ld_x, int M, int K, int k_tail,
                                   const float* inv_scale_pos, const int32_t* perm,
                                   const int32_t* group_offsets, int G, uint8_t* Ap, uint8_t* Aps,
                                   int num_cus, hipStream_t stream) {
  return launch_act_quant_packed_kernel(X, ld_x, M, K, k_tail, inv_scale_pos, perm, group_offsets,
                                        G, Ap, Aps, num_cus, 0, stream);
}

hipError_t launch_act_quant_packed_kernel(const uint16_t* X, int64_t ld_x, int M, int K,
                                          int k_tail, const float* inv_scale_pos,
                                          const int32_t* perm, const int32_t* group_offsets,
                                          int G, uint8_t* Ap, uint8_t* Aps, int num_cus,
                                          int kernel, hipStream_t stream) {
  const bool grouped = group_offsets && G > 1;
  const int32_t* off = grouped ? group_offsets : nullptr;
  // Few rows (decode): the few-rows kernel, as for the row-major output (the
  // whole-K decode GEMM then copies each 16-row group's operand in whole
  // kilobytes).
  if (kernel == 1 || (kernel == 0 && M <= 64))
    return launch_rows_packed(X, ld_x, M, K, k_tail, inv_scale_pos, perm, off, G, Ap, Aps, stream);
  if (kernel == 3 || kernel == 4 || (kernel == 0 && K >= 2048)) {
    const int window = kernel == 3 ? 1 : kernel == 4 ? 2 : 0;
    if (grouped)
      return launch_dma<true, true>(X, ld_x, M, K, k_tail, inv_scale_pos, perm, off, G, Ap, Aps,
                                    num_cus, stream, window);
    return launch_dma<false, true>(X, ld_x, M, K, k_tail, inv_scale_pos, perm, nullptr, 1, Ap, Aps,
                                   num_cus, stream, window);
  }
  const int units = K >> 3;
  const size_t lds = lds_kernel_bytes(K);
  const int per_thread = (units + kLdsThreads - 1) / kLdsThreads;
  const int rows_per_wg = lds_rows_per_wg(M, units, num_cus);
  const dim3 grid((M + rows_per_wg - 1) / rows_per_wg);
#define PRQ_LDS_PACKED_CASE(n)                                                                  \
  if (grouped)                                                                                 \
    launch_lds<true, n, true>(grid, lds, stream, X, ld_x, M, K, k_tail, inv_scale_pos, perm, off, \
                              G, rows_per_wg, Ap, Aps);                                        \
  else                                                                                         \
    launch_lds<false, n, true>(grid, lds, stream, X, ld_x, M, K, k_tail, inv_scale_pos, perm,   \
                               nullptr, 1, rows_per_wg, Ap, Aps);                              \
  break;
  switch (per_thread) {
    case 1: PRQ_LDS_PACKED_CASE(1)
    case 2: PRQ_LDS_PACKED_CASE(2)
    case 3: PRQ_LDS_PACKED_CASE(3)
    default: PRQ_LDS_PACKED_CASE(4)
  }
#undef PRQ_LDS_PACKED_CASE
  return hipGetLastError();
}

namespace {

// Offline copy, producer side (Sec. Method, "Activation tail construction";
// Eq. 1 with sigma = SiLU): the expanded up/gate projections emit gate and up
// outputs K_aug = C + k wide whose product SiLU(gate) * up is already
// [Z~, Z~_tail], so the down-projection's MXFP4 input is that product
// quantized -- no gather, no scaling, no tail copy.  The product is formed in
// float32 and never rounded to bf16.  SiLU(g) = g / (1 + e^-g) with e^x by a
// fixed sequence, one IEEE float32 operation per step (contraction off), so
// the result does not depend on the device's own exp: x clamped to [-104, 89];
// n = rint(x log2 e); r = (x - n ln2_hi) - n ln2_lo with ln 2 split into a
// 15-bit head (n ln2_hi exact) and a tail; e^r by its degree-6 Taylor
// polynomial in Horner form; e^x = r's polynomial scaled by 2^n (exact).
__device__ __forceinline__ float silu_seq(float g) {
#pragma clang fp contract(off)
  const float x = fminf(fmaxf(-g, -104.0f), 89.0f);
  const float n = rintf(x * 0x1.715476p+0f);                // log2 e
  const float r = (x - n * 0x1.62e4p-1f) - n * 0x1.7f7d1cp-20f;   // ln 2 head, tail
  float p = 0x1.6c16c2p-10f;                                // 1/6!
  p = p * r + 0x1.111112p-7f;                               // 1/5!
  p = p * r + 0x1.555556p-5f;                               // 1/4!
  p = p * r + 0x1.555556p-3f;                               // 1/3!
  p = p * r + 0.5f;
  p = p * r + 1.0f;
  p = p * r + 1.0f;
  const float e = ldexpf(p, static_cast<int>(n));
  return __fdiv_rn(g, 1.0f + e);
}

// One thread per unit (8 consecutive outputs of a row); the 4 units of a
// 32-block are consecutive lanes (K_aug % 32 == 0).  Packed output: the rows of
// the last 16-row block past M and the K positions past K_aug get zero codes
// and scale byte 127, as the packed quantizer writes them.
template <bool kPacked>
__global__ __launch_bounds__(256) void swiglu_quant_kernel(const uint16_t* __restrict__ G,
                                                           const uint16_t* __restrict__ U,
                                                           int64_t ld, int M, int K_aug,
                                                           uint8_t* __restrict__ Aq,
                                                           uint8_t* __restrict__ Asc) {
#pragma clang fp contract(off)
  const int units = K_aug >> 3;
  const int nb = K_aug >> 5;
  const int64_t row_bytes = K_aug >> 1;
  const int steps = (K_aug + 127) >> 7;
  const int sgroups = (steps + 3) >> 2;
  const int rows = kPacked ? (M + 15) & ~15 : M;
  const int64_t total = static_cast<int64_t>(rows) * units;   // a multiple of 4: whole quads
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < total;
       i += static_cast<int64_t>(gridDim.x) * 256) {
    const int r = static_cast<int>(i / units);
    const int u = static_cast<int>(i - static_cast<int64_t>(r) * units);
    if (kPacked && r >= M) {                       // quad-uniform
      const PackedSink psink(Aq, Asc, r, steps, sgroups);
      psink.word(u, 0u);
      if ((u & 3) == 0) psink.scale(u >> 2, 127u);
      pad_row_tail(psink, u, units, nb, steps, sgroups);
      continue;
    }
    const int64_t at = static_cast<int64_t>(r) * ld + u * 8;
    const uint4 gv = *reinterpret_cast<const uint4*>(G + at);
    const uint4 uv = *reinterpret_cast<const uint4*>(U + at);
    const uint32_t gw[4] = {gv.x, gv.y, gv.z, gv.w};
    const uint32_t uw[4] = {uv.x, uv.y, uv.z, uv.w};
    float z[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float g0 = __uint_as_float(gw[j] << 16), g1 = __uint_as_float(gw[j] & 0xFFFF0000u);
      const float u0 = __uint_as_float(uw[j] << 16), u1 = __uint_as_float(uw[j] & 0xFFFF0000u);
      z[2 * j] = silu_seq(g0) * u0;
      z[2 * j + 1] = silu_seq(g1) * u1;
    }
    if constexpr (kPacked) {
      const PackedSink psink(Aq, Asc, r, steps, sgroups);
      quantize_store(z, u, units, 0, 0, psink);
      pad_row_tail(psink, u, units, nb, steps, sgroups);
    } else {
      quantize_store(z, u, units, 0, 0,
                     RowSink{Aq + static_cast<int64_t>(r) * row_bytes, Asc + static_cast<int64_t>(r) * nb});
    }
  }
}

}  // namespace

hipError_t launch_swiglu_quant(const uint16_t* G, const uint16_t* U, int64_t ld, int M, int K_aug,
                               uint8_t* Aq, uint8_t* Asc, bool packed, int num_cus,
                               hipStream_t stream) {
  // One thread per unit (a thread's two 16-byte loads are its only memory
  // round trip; with a grid capped at a few workgroups per CU each thread
  // looped over ~20 units, one round trip after another: 132 against 64 us at
  // M = 8192 x 9984); the loop only covers grids past the launch limit.
  (void)num_cus;
  const int rows = packed ? (M + 15) & ~15 : M;
  const int64_t total = static_cast<int64_t>(rows) * (K_aug >> 3);
  const dim3 grid(static_cast<unsigned>(std::max<int64_t>(1, std::min<int64_t>((total + 255) / 256, int64_t{1} << 30))));
  if (packed)
    swiglu_quant_kernel<true><<<grid, 256, 0, stream>>>(G, U, ld, M, K_aug, Aq, Asc);
  else
    swiglu_quant_kernel<false><<<grid, 256, 0, stream>>>(G, U, ld, M, K_aug, Aq, Asc);
  return hipGetLastError();
}

}  // namespace prq
