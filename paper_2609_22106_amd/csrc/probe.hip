// Test-only probes of gfx950 instruction semantics (libprq_probe.so; not part
// of libprq.so).  Every kernel is in bounds by construction: one wave for the
// MFMA probe, a fixed 2^32-pattern sweep with no memory traffic except an
// atomic mismatch counter for the conversion probe.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "mx_device.hpp"
#include "prq_internal.h"

namespace {

using prq::dev::v4f;

// One wave: lane l passes a[l] (16 bytes of FP4), b[l], sa[l], sb[l] to a single
// block-scaled 16x16x128 FP4 MFMA and writes its 4 accumulator values.
__global__ __launch_bounds__(64) void mfma16_probe(const uint4* a, const uint4* b,
                                                   const uint32_t* sa, const uint32_t* sb,
                                                   float* out) {
  const int l = threadIdx.x;
  v4f c = {0.f, 0.f, 0.f, 0.f};
  c = prq::dev::mfma_fp4_16x16x128(a[l], b[l], sa[l], sb[l], c);
  for (int q = 0; q < 4; ++q) out[l * 4 + q] = c[q];
}

// Exhaustive comparison of the hardware FP32 -> FP4 conversion (scale 1.0)
// with the software rounding rule of mx_device.hpp over every finite float32
// bit pattern.  result[0] counts mismatches, result[1..2*kRec] records the
// first bit patterns and hardware bytes.
constexpr int kRec = 8;

__global__ __launch_bounds__(256) void cvt_sweep(uint32_t* result) {
  const uint64_t t = static_cast<uint64_t>(blockIdx.x) * 256 + threadIdx.x;
  for (uint32_t i = 0; i < 256; ++i) {
    const uint32_t bits = static_cast<uint32_t>(t * 256 + i);
    if (((bits >> 23) & 0xFFu) == 0xFFu) continue;  // Inf / NaN
    const float x = __uint_as_float(bits);
    const uint32_t hw = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, x, -x, 1.0f, 0) & 0xFFu;
    const uint32_t sw = prq::dev::e2m1_code(x, x) | (prq::dev::e2m1_code(-x, -x) << 4);
    if (hw != sw) {
      const uint32_t k = atomicAdd(&result[0], 1u);
      if (k < kRec) {
        result[1 + 2 * k] = bits;
        result[2 + 2 * k] = hw;
      }
    }
  }
}

// Convert (x[i], y[i]) with scale s[i] into byte i (x in the low nibble slot).
__global__ void cvt_pairs(const float* x, const float* y, const float* s, int n, uint8_t* out) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) out[i] = static_cast<uint8_t>(__builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, x[i], y[i], s[i], 0) & 0xFFu);
}

// The FP32 -> FP4 pair conversion with each destination byte select: lane l
// converts (x[l], y[l]) at scale 1 into byte `sel` of old = 0x89ABCDEF for
// sel = 0..3; out[4 l + sel] is the whole result word.
__global__ __launch_bounds__(64) void cvt_sel_probe(const float* x, const float* y, uint32_t* out) {
  const int l = threadIdx.x;
  const uint32_t old = 0x89ABCDEFu;
  out[4 * l + 0] = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(old, x[l], y[l], 1.0f, 0);
  out[4 * l + 1] = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(old, x[l], y[l], 1.0f, 1);
  out[4 * l + 2] = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(old, x[l], y[l], 1.0f, 2);
  out[4 * l + 3] = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(old, x[l], y[l], 1.0f, 3);
}

// Direct global->LDS loads (one wave): 16 bytes per lane from g16 into LDS at
// byte 0, one byte per lane from g1 into LDS at byte 4096; the 8 KiB LDS image
// (zeroed first) is copied out so the host can see where each lane's data went.
__global__ __launch_bounds__(64) void lds_dma_probe(const uint8_t* g16, const uint8_t* g1,
                                                    uint8_t* out) {
  __shared__ __align__(16) uint8_t s[8192];
  const int l = threadIdx.x;
  for (int i = l; i < 8192 / 16; i += 64) reinterpret_cast<uint4*>(s)[i] = make_uint4(0, 0, 0, 0);
  __syncthreads();
  __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)(g16 + l * 16),
                                   (__attribute__((address_space(3))) void*)(s), 16, 0, 0);
  __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)(g1 + l),
                                   (__attribute__((address_space(3))) void*)(s + 4096), 1, 0, 0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  for (int i = l; i < 8192 / 16; i += 64) reinterpret_cast<uint4*>(out)[i] = reinterpret_cast<uint4*>(s)[i];
}

// The weight-read floor: the kilobytes [0, kib1) of p1 and then [0, kib2) of
// p2 read with `wgs` workgroups of 8 waves, each an equal contiguous share of
// the kilobytes, every load issued before any is consumed (the memory side of
// a weight-streaming decode GEMM, with no arithmetic and no output but a
// never-taken store that keeps the loads).
__global__ __launch_bounds__(512) void read_floor_kernel(const uint8_t* __restrict__ p1, int kib1,
                                                         const uint8_t* __restrict__ p2, int kib2,
                                                         uint32_t* __restrict__ out) {
  const int total = kib1 + kib2;
  const int wgs = gridDim.x, wg = blockIdx.x;
  const int u0 = static_cast<int>(static_cast<int64_t>(total) * wg / wgs);
  const int u1 = static_cast<int>(static_cast<int64_t>(total) * (wg + 1) / wgs);
  const int nu = u1 - u0, wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int v0 = u0 + nu * wave / 8, cnt = nu * (wave + 1) / 8 - nu * wave / 8;   // <= 8 (host)
  uint4 w[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int u = cnt > 0 ? v0 + min(j, cnt - 1) : u0;
    const uint8_t* src = u < kib1 ? p1 + static_cast<int64_t>(u) * 1024
                                  : p2 + static_cast<int64_t>(u - kib1) * 1024;
    w[j] = *reinterpret_cast<const uint4*>(src + lane * 16);
  }
  uint32_t x = 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) x ^= w[j].x ^ w[j].y ^ w[j].z ^ w[j].w;
  if (x == 0x9E3779B9u && lane == 0) out[wg] = x;
}

// LDS read patterns (reference points for the bank-conflict counters): each
// workgroup of 4 waves fills 16 KiB of LDS, then every wave reads, `iters`
// times, one kilobyte (rotating over the 16) in pattern kMode:
//   0  16 bytes per lane at 16 l: the tile GEMM's operand reads;
//   1  4 bytes per lane at 256 ((l / 16) % 2) + 4 ((l % 16) + 16 (l / 32)):
//      the tile GEMM's scale reads (two 16-row blocks, half a step each);
//   2  4 bytes per lane at 4 l (one dword per bank);
//   4  pattern 1 with the tile GEMM's staging swap: lanes of the odd block
//      (l / 16 odd) read K part (l / 32) ^ 1, 4 ((l % 16) + 16 ((l / 32) ^ 1));
//   3  eight 2-byte reads per lane at 16 l + 2 j: the quantizer's gather of a
//      unit of 8 consecutive channels (the element stride `elem` = 2 is a
//      run-time value, so the reads stay eight separate 2-byte reads as in
//      the quantizer, whose addresses come from the permutation).
// Every address is inside the 16 KiB; lane results are folded and stored.
template <int kMode>
__global__ __launch_bounds__(256) void lds_pattern_kernel(int iters, int elem, uint32_t* __restrict__ out) {
  __shared__ __align__(16) uint8_t s[16384];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int i = tid; i < 16384 / 4; i += 256) reinterpret_cast<uint32_t*>(s)[i] = i * 2654435761u;
  __syncthreads();
  uint32_t acc = 0;
  for (int it = 0; it < iters; ++it) {
    const int base = ((it + wave) & 15) * 1024;
    if constexpr (kMode == 0) {
      const uint4 v = *reinterpret_cast<const uint4*>(s + base + lane * 16);
      acc ^= v.x ^ v.y ^ v.z ^ v.w;
    } else if constexpr (kMode == 1) {
      acc ^= *reinterpret_cast<const uint32_t*>(
          s + base + ((lane >> 4) & 1) * 256 + ((lane & 15) + 16 * (lane >> 5)) * 4);
    } else if constexpr (kMode == 2) {
      acc ^= *reinterpret_cast<const uint32_t*>(s + base + lane * 4);
    } else if constexpr (kMode == 4) {
      const int odd = (lane >> 4) & 1;
      acc ^= *reinterpret_cast<const uint32_t*>(
          s + base + odd * 256 + ((lane & 15) + 16 * ((lane >> 5) ^ odd)) * 4);
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j)
        acc += *reinterpret_cast<const uint16_t*>(s + base + lane * 16 + elem * j);
    }
    asm volatile("" ::: "memory");   // one read (set) per iteration, none hoisted
  }
  out[blockIdx.x * 256 + tid] = acc;
}

}  // namespace

extern "C" {

// Weight-read floor (context for the decode GEMM): out needs wgs dwords;
// kib1, kib2 >= 0 kilobytes, at most 64 kilobytes per workgroup.
int prq_probe_read_floor(const uint8_t* p1, int kib1, const uint8_t* p2, int kib2, int wgs,
                         uint32_t* out, hipStream_t stream) {
  if (wgs <= 0 || kib1 < 0 || kib2 < 0 || kib1 + kib2 < wgs ||
      (static_cast<int64_t>(kib1) + kib2 + wgs - 1) / wgs > 64 || !out || (kib1 && !p1) ||
      (kib2 && !p2))
    return -1;
  read_floor_kernel<<<wgs, 512, 0, stream>>>(p1, kib1, p2, kib2, out);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}


// The LDS read-pattern kernel of `mode` (0-4): `blocks` workgroups, `iters`
// reads per wave; out holds blocks * 256 uint32 (their folded values).
int prq_probe_lds_pattern(int mode, int blocks, int iters, uint32_t* out, hipStream_t stream) {
  if (mode < 0 || mode > 4 || blocks <= 0 || iters < 0 || !out) return -1;
  const int elem = 2;   // mode 3: 8 reads of 2 bytes, 16 l + 14 + 2 < 1024
  switch (mode) {
    case 0: lds_pattern_kernel<0><<<blocks, 256, 0, stream>>>(iters, elem, out); break;
    case 1: lds_pattern_kernel<1><<<blocks, 256, 0, stream>>>(iters, elem, out); break;
    case 2: lds_pattern_kernel<2><<<blocks, 256, 0, stream>>>(iters, elem, out); break;
    case 4: lds_pattern_kernel<4><<<blocks, 256, 0, stream>>>(iters, elem, out); break;
    default: lds_pattern_kernel<3><<<blocks, 256, 0, stream>>>(iters, elem, out); break;
  }
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

int prq_probe_mfma16(const void* a, const void* b, const uint32_t* sa, const uint32_t* sb,
                     float* out, hipStream_t stream) {
  mfma16_probe<<<1, 64, 0, stream>>>(static_cast<const uint4*>(a), static_cast<const uint4*>(b), sa,
                                     sb, out);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

// result: device uint32[1 + 2*8], zero-filled by the caller.
int prq_probe_cvt_sweep(uint32_t* result, hipStream_t stream) {
  cvt_sweep<<<65536, 256, 0, stream>>>(result);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

// x, y: 64 floats each, out: 256 uint32 (device).
int prq_probe_cvt_sel(const float* x, const float* y, uint32_t* out, hipStream_t stream) {
  cvt_sel_probe<<<1, 64, 0, stream>>>(x, y, out);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

int prq_probe_cvt_pairs(const float* x, const float* y, const float* s, int n, uint8_t* out,
                        hipStream_t stream) {
  if (n <= 0) return 0;
  cvt_pairs<<<(n + 255) / 256, 256, 0, stream>>>(x, y, s, n, out);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

// Tuning entry: the weight-streaming GEMM with an explicit configuration.
// Returns -1 when the configuration does not cover K_aug (nothing launched).
int prq_tune_gemm_stream(const uint8_t* Aq, const uint8_t* Asc, int M, const int32_t* off, int E,
                         const uint8_t* Wq, const uint8_t* Wsc, int N, int K_aug, float* Y,
                         int splits, int waves, int unroll, int groups, int tiles,
                         int stage_lds, int reduce, int wave_tiles, void* workspace,
                         hipStream_t stream) {
  prq::StreamConfig c;
  c.tiles = tiles;
  c.wave_tiles = wave_tiles;
  c.stage_lds = stage_lds != 0;
  c.reduce = reduce;
  c.splits = splits;
  c.waves = waves;
  c.unroll = unroll;
  c.groups = groups;
  if (!prq::stream_config_covers(c, K_aug) || N % 16 || K_aug % 32 || M <= 0) return -1;
  if (splits > 1 && reduce != 2 && !workspace) return -1;
  if (reduce < 0 || reduce > 2) return -1;
  return prq::launch_gemm_stream(Aq, Asc, M, off, E, Wq, Wsc, N, K_aug, Y, c, workspace, stream) ==
                 hipSuccess
             ? 0
             : -3;
}

typedef float v16f_t __attribute__((ext_vector_type(16)));

// One 32x32x64 block-scaled FP4 MFMA on lane-supplied operands: a, b are
// [64 lanes][16 bytes], sa, sb one E8M0 byte per lane; out [64 lanes][16].
__global__ __launch_bounds__(64) void mfma32_probe(const uint4* a, const uint4* b,
                                                   const uint32_t* sa, const uint32_t* sb,
                                                   float* out) {
  const int l = threadIdx.x;
  const uint4 x = a[l], y = b[l];
  const prq::dev::v8i av = {static_cast<int>(x.x), static_cast<int>(x.y), static_cast<int>(x.z),
                            static_cast<int>(x.w), 0, 0, 0, 0};
  const prq::dev::v8i bv = {static_cast<int>(y.x), static_cast<int>(y.y), static_cast<int>(y.z),
                            static_cast<int>(y.w), 0, 0, 0, 0};
  v16f_t c;
#pragma unroll
  for (int j = 0; j < 16; ++j) c[j] = 0.f;
  c = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av, bv, c, 4, 4, 0, static_cast<int>(sa[l]), 0,
                                                      static_cast<int>(sb[l]));
#pragma unroll
  for (int j = 0; j < 16; ++j) out[l * 16 + j] = c[j];
}

int prq_probe_mfma32(const void* a, const void* b, const void* sa, const void* sb, float* out,
                     hipStream_t stream) {
  mfma32_probe<<<1, 64, 0, stream>>>(static_cast<const uint4*>(a), static_cast<const uint4*>(b),
                                     static_cast<const uint32_t*>(sa),
                                     static_cast<const uint32_t*>(sb), out);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

// Activation quantization with a forced kernel (1 few-rows, 2 many-rows with
// register-staged rows, 3 many-rows with rows copied into LDS stages).
int prq_tune_act_quant(const void* X, int64_t ld_x, int M, int K, int k_tail, const float* inv,
                       const int32_t* perm, uint8_t* Aq, uint8_t* Asc, int kernel,
                       hipStream_t stream) {
  if (M <= 0 || K <= 0 || K % 32 || k_tail % 32 || k_tail > K || K > 16384 || ld_x < K) return -1;
  return prq::launch_act_quant_kernel(static_cast<const uint16_t*>(X), ld_x, M, K, k_tail, inv, perm,
                                      nullptr, 1, Aq, Asc, 256, kernel, stream) == hipSuccess
             ? 0
             : -3;
}

// The same into the packed activation layout (0 automatic, 1 one row per workgroup row,
// 2 register-staged, 3 LDS stages
// with the output through an LDS window where it fits, 4 LDS stages with the
// output stored directly), its workgroups sized for num_cus CUs.
int prq_tune_act_quant_packed(const void* X, int64_t ld_x, int M, int K, int k_tail,
                              const float* inv, const int32_t* perm, const int32_t* off, int G,
                              uint8_t* Ap, uint8_t* Aps, int kernel, int num_cus,
                              hipStream_t stream) {
  if (M <= 0 || K <= 0 || K % 32 || k_tail % 32 || k_tail > K || K > 16384 || ld_x < K ||
      kernel < 0 || kernel > 4 || num_cus <= 0)
    return -1;
  return prq::launch_act_quant_packed_kernel(static_cast<const uint16_t*>(X), ld_x, M, K, k_tail,
                                             inv, perm, off, G, Ap, Aps, num_cus, kernel,
                                             stream) == hipSuccess
             ? 0
             : -3;
}

// The decode GEMM with forced tile / row-split counts (0 = automatic); -1 when the shape
// is not covered.
int prq_tune_gemm_decode(const uint8_t* Aq, const uint8_t* Asc, int M, const int32_t* off, int E,
                         const uint8_t* Wq, const uint8_t* Wsc, int N, int K_aug, float* Y,
                         int tiles, int row_splits, hipStream_t stream) {
  if (N % 16 || K_aug % 32 || M <= 0) return -1;
  const prq::DecodeConfig c = prq::choose_decode_config(off ? (M + E - 1) / E : M, N, K_aug,
                                                        off ? 1 : 0, tiles, row_splits, 256);
  if (!c.ok || (off && c.tiles != 1)) return -1;
  return prq::launch_gemm_decode(Aq, Asc, M, off, E, Wq, Wsc, N, K_aug, Y, c, stream) == hipSuccess
             ? 0
             : -3;
}

// Tuning entry: the stream-K decode GEMM planned for `num_cus` CUs with
// `workgroups` workgroups (0: the planner's choice; the workspace sized for
// that plan).  Returns -1 when the kernel does not apply (nothing launched).
int prq_tune_gemm_streamk(const uint8_t* Aq, const uint8_t* Asc, int M, const uint8_t* Wp,
                          const uint8_t* Wps, int N, int K_aug, float* Y, int num_cus,
                          int workgroups, void* workspace, size_t workspace_bytes,
                          hipStream_t stream) {
  if (N % 16 || K_aug % 32 || M <= 0 || num_cus <= 0) return -1;
  const prq::StreamKConfig c = prq::choose_streamk_config(M, N, K_aug, num_cus, workgroups);
  if (!c.ok) return -1;
  const size_t need = c.shared ? prq::kWorkspaceStateBytes +
                                     static_cast<size_t>(c.workgroups) * 2 * M * 16 * sizeof(float)
                               : 0;
  if (workspace_bytes < need) return -1;
  return prq::launch_gemm_streamk(Aq, Asc, M, Wp, Wps, N, K_aug, Y, c, workspace, stream) ==
                 hipSuccess
             ? 0
             : -3;
}

// Workspace bytes of prq_tune_gemm_streamk (0 when the kernel does not apply).
size_t prq_tune_streamk_workspace_bytes(int M, int N, int K_aug, int num_cus, int workgroups) {
  const prq::StreamKConfig c = prq::choose_streamk_config(M, N, K_aug, num_cus, workgroups);
  return c.ok && c.shared ? prq::kWorkspaceStateBytes +
                               static_cast<size_t>(c.workgroups) * 2 * M * 16 * sizeof(float)
                         : 0;
}

// Tuning entry: the tile GEMM with an explicit tile shape (0, 1 or 2).
int prq_tune_gemm_tile(const uint8_t* Aq, const uint8_t* Asc, int M, const int32_t* off, int E,
                       const uint8_t* Wp, const uint8_t* Wps, int N, int K_aug, float* Y, int shape,
                       hipStream_t stream) {
  if (shape < 0 || shape > 3 || N % 16 || K_aug % 32 || M <= 0) return -1;
  return prq::launch_gemm_tile(Aq, Asc, M, off, E, Wp, Wps, N, K_aug, Y, shape, stream) == hipSuccess
             ? 0
             : -3;
}

// Tuning entry: the tile GEMM on a packed activation with an explicit tile shape.
int prq_tune_gemm_tile_packed(const uint8_t* Ap, const uint8_t* Aps, int M, const uint8_t* Wp,
                              const uint8_t* Wps, int N, int K_aug, float* Y, int shape,
                              hipStream_t stream) {
  if (shape < 0 || shape > 3 || N % 16 || K_aug % 32 || M <= 0) return -1;
  return prq::launch_gemm_tile_packed(Ap, Aps, M, Wp, Wps, N, K_aug, Y, shape, stream) == hipSuccess
             ? 0
             : -3;
}

// The dense tile GEMM with a forced shape and split count along K (packed or
// row-major activation); ws: (splits - 1) * M * N floats (ws_bytes checked),
// 16-byte aligned.
int prq_tune_gemm_tile_split(const uint8_t* A, const uint8_t* As, int M, const uint8_t* Wp,
                             const uint8_t* Wps, int N, int K_aug, float* Y, int shape,
                             int splits, int packed, float* ws, size_t ws_bytes,
                             hipStream_t stream) {
  if (shape < 0 || shape > 3 || N % 16 || K_aug % 32 || M <= 0 || splits < 1) return -1;
  if (splits > 1 &&
      (!ws || static_cast<size_t>(splits - 1) * M * N * sizeof(float) > ws_bytes))
    return -2;   // the partial sums would not fit
  return prq::launch_gemm_tile_split(A, As, M, Wp, Wps, N, K_aug, Y, packed != 0, shape, splits,
                                     ws, stream) == hipSuccess
             ? 0
             : -3;
}

// The grouped tile GEMM on a packed activation with a forced shape (0-3: a
// workgroup per tile; 4: the persistent kernel over num_cus CUs).
int prq_tune_grouped_gemm_tile_packed(const uint8_t* Ap, const uint8_t* Aps, int M,
                                      const int32_t* off, int E, const uint8_t* Wp,
                                      const uint8_t* Wps, int N, int K_aug, float* Y, int shape,
                                      int num_cus, hipStream_t stream) {
  if (shape < 0 || shape > prq::kShapePersist || N % 16 || K_aug % 32 || M <= 0 || E < 1 ||
      !off || num_cus < 0 || (shape == prq::kShapePersist && (num_cus < 1 || E > 512)))
    return -1;
  return prq::launch_grouped_gemm_tile_packed(Ap, Aps, M, off, E, Wp, Wps, N, K_aug, Y, shape,
                                              num_cus, stream) == hipSuccess
             ? 0
             : -3;
}

// g16: 1024 bytes, g1: 64 bytes, out: 8192 bytes (device).
int prq_probe_lds_dma(const uint8_t* g16, const uint8_t* g1, uint8_t* out, hipStream_t stream) {
  lds_dma_probe<<<1, 64, 0, stream>>>(g16, g1, out);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

}  // extern "C"
