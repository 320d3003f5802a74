// Packed weight layout for the block-scaled FP4 MFMA (an invertible byte
// permutation of the exported Q([W~, R_W]) of Eq. 3, applied once per weight).
//
// Canonical (prq_prepare output): Wq [E][N][K_aug/2], Wsc [E][N][K_aug/32].
// Packed, with S = ceil(K_aug / 128) K steps and T = N / 16 feature tiles:
//   Wp  [E][T][S][64 lanes][16 bytes]: lane l of block (t, s) holds the 16
//       code bytes of weight row 16t + (l % 16), K elements
//       [128 s + 32 (l / 16), +32), i.e. exactly what lane l feeds to the
//       v_mfma_scale_f32_16x16x128_f8f6f4 A/B operand; zero past K_aug.
//   Wps [E][T][ceil(S/4)][64 lanes][4 bytes]: byte j of lane l's dword in
//       group (t, q) is the E8M0 scale of row 16t + (l % 16), 32-block
//       4 (4q + j) + l / 16; 127 past K_aug.
// So one wave reads one contiguous kilobyte per MFMA operand and one dword of
// scales per four K steps.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "prq_internal.h"

namespace prq {
namespace {

constexpr int kPackThreads = 256;

// One thread per (e, t, s, lane): copies 16 bytes (4 dwords of one row).
__global__ __launch_bounds__(kPackThreads) void pack_codes_kernel(
    const uint8_t* __restrict__ Wq, int N, int K_aug, int E, uint8_t* __restrict__ Wp) {
  const int S = (K_aug + 127) / 128;
  const int T = N / 16;
  const int64_t total = static_cast<int64_t>(E) * T * S * 64;
  const int64_t i = static_cast<int64_t>(blockIdx.x) * kPackThreads + threadIdx.x;
  if (i >= total) return;
  const int l = static_cast<int>(i & 63);
  const int64_t blk = i >> 6;                 // (e * T + t) * S + s
  const int s = static_cast<int>(blk % S);
  const int64_t et = blk / S;                 // e * T + t
  const int64_t row = et * 16 + (l & 15);     // row within [E * N]
  const int kel = s * 128 + (l >> 4) * 32;
  uint4 v = make_uint4(0, 0, 0, 0);
  if (kel < K_aug)
    v = *reinterpret_cast<const uint4*>(Wq + row * (K_aug / 2) + kel / 2);
  *reinterpret_cast<uint4*>(Wp + i * 16) = v;
}

// One thread per (e, t, q, lane): gathers 4 scale bytes into a dword.
__global__ __launch_bounds__(kPackThreads) void pack_scales_kernel(
    const uint8_t* __restrict__ Wsc, int N, int K_aug, int E, uint32_t* __restrict__ Wps) {
  const int S = (K_aug + 127) / 128;
  const int Q = (S + 3) / 4;
  const int T = N / 16;
  const int nb = K_aug / 32;
  const int64_t total = static_cast<int64_t>(E) * T * Q * 64;
  const int64_t i = static_cast<int64_t>(blockIdx.x) * kPackThreads + threadIdx.x;
  if (i >= total) return;
  const int l = static_cast<int>(i & 63);
  const int64_t grp = i >> 6;                 // (e * T + t) * Q + q
  const int q = static_cast<int>(grp % Q);
  const int64_t row = (grp / Q) * 16 + (l & 15);
  uint32_t d = 0;
  for (int j = 0; j < 4; ++j) {
    const int b = 4 * (4 * q + j) + (l >> 4);
    const uint32_t sc = b < nb ? Wsc[row * nb + b] : 127u;
    d |= sc << (8 * j);
  }
  Wps[i] = d;
}

}  // namespace

size_t packed_code_bytes(int N, int K_aug, int E) {
  return static_cast<size_t>(E) * (N / 16) * ((K_aug + 127) / 128) * 1024;
}

size_t packed_scale_bytes(int N, int K_aug, int E) {
  return static_cast<size_t>(E) * (N / 16) * (((K_aug + 127) / 128 + 3) / 4) * 256;
}

hipError_t launch_pack_weight(const uint8_t* Wq, const uint8_t* Wsc, int N, int K_aug, int E,
                              uint8_t* Wp, uint8_t* Wps, hipStream_t stream) {
  const int64_t nc = static_cast<int64_t>(packed_code_bytes(N, K_aug, E) / 16);
  const int64_t ns = static_cast<int64_t>(packed_scale_bytes(N, K_aug, E) / 4);
  pack_codes_kernel<<<static_cast<unsigned>((nc + kPackThreads - 1) / kPackThreads), kPackThreads, 0,
                      stream>>>(Wq, N, K_aug, E, Wp);
  pack_scales_kernel<<<static_cast<unsigned>((ns + kPackThreads - 1) / kPackThreads), kPackThreads, 0,
                       stream>>>(Wsc, N, K_aug, E, reinterpret_cast<uint32_t*>(Wps));
  return hipGetLastError();
}

}  // namespace prq
