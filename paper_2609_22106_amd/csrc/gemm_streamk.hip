// Stream-K decode kernel of the augmented MXFP4 GEMM (arXiv 2609.22106,
// Eq. 3: one block-scaled GEMM over K_aug = K + k) for up to 64 activation
// rows, where the call is bound by reading W_aug once from HBM.
//
// The packed weight is a sequence of U = T * S units, a unit being one
// 16-feature tile at one 128-element K step (one contiguous kilobyte of codes
// plus a byte of each of its 64 lanes' scale dwords), ordered tile-major.
// The launch has one workgroup per CU and workgroup w owns the contiguous
// unit range [U w / P, U (w + 1) / P): every CU streams an equal share of the
// weight whatever N / 16 is (N = 2560 has 160 tiles for 256 CUs).  Because a
// range is at most one tile long (T <= P, checked on the host), it touches at
// most two tiles, and a tile is shared by at most a few neighbouring
// workgroups.
//
//   * The workgroup's range is split into contiguous runs of its waves; a wave
//     issues, for each of its units in order, the weight codes (the MFMA A
//     operand: 16 features x 128 K), the tile's scale dword, and the
//     activation operand of that step for each 16-row group (the MFMA B
//     operand, read from the row-major quantizer output: 16 rows x 64 bytes,
//     rows past M clamped to the last row and never stored) with its scale
//     bytes -- every load of the wave before its first MFMA, and the MFMAs in
//     load order, so the wave waits only for the unit it needs next.
//   * A wave keeps one accumulator per row group for each of the (at most two)
//     tiles of the workgroup; the waves' accumulators are summed through LDS
//     in wave order.
//   * A tile covered whole by one workgroup is written to Y.  Otherwise each
//     covering workgroup writes its partial tile into its own slot of the
//     caller's workspace with device-scope stores, waits for them to complete,
//     and increments the tile's arrival counter (in the workspace's state
//     head, ahead of the partial slots); the last to arrive adds the
//     covering workgroups' partials in workgroup order (a fixed order: the
//     result does not depend on which arrives last), writes Y and resets the
//     counter, so the counters are zero between calls.  No workgroup waits for
//     another.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>

#include "mx_device.hpp"
#include "prq_internal.h"

namespace prq {
namespace {

using dev::v4f;

constexpr int kStepK = 128;
constexpr uint32_t kNeutralScale = 127;
constexpr int kMaxRows = 64;
constexpr int kMaxFrags = 4;   // workgroups sharing one tile

__device__ __forceinline__ void wait_all_vm() {
  // vmcnt = 0 (stores included), expcnt and lgkmcnt left at their maxima
  __builtin_amdgcn_s_waitcnt((0x7 << 4) | (0xF << 8));
}

// First unit of workgroup wg's range (units * wgs < 2^31, checked on the host).
__device__ __forceinline__ int range_begin(int units, int wg, int wgs) {
  return static_cast<int>(static_cast<uint32_t>(units * wg) / static_cast<uint32_t>(wgs));
}

// Waves given to the first of a range's two parts (a of nu units in tile
// t0, the rest in tile t0 + 1): the count, at least one per non-empty part,
// that minimizes the most units any wave gets (the first such count).
__host__ __device__ inline int wave_split(int a, int nu, int waves) {
  if (a >= nu) return waves;
  int best = 1, best_units = 0x7fffffff;
  for (int n = 1; n < waves; ++n) {
    const int x = (a + n - 1) / n, y = (nu - a + waves - n - 1) / (waves - n);
    const int most = x > y ? x : y;
    if (most < best_units) {
      best_units = most;
      best = n;
    }
  }
  return best;
}

template <int kWaves, int kU, int kG>
__global__ __launch_bounds__(kWaves * 64) void gemm_streamk_kernel(
    const uint8_t* __restrict__ Aq, const uint8_t* __restrict__ Asc, int M,
    const uint8_t* __restrict__ Wp, const uint8_t* __restrict__ Wps, int N, int K_aug,
    float* __restrict__ Y, float* __restrict__ part, uint32_t* __restrict__ ctr) {
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ int s_last[2];

  const int S = (K_aug + kStepK - 1) / kStepK;
  const int SG = (S + 3) >> 2;
  const int T = N >> 4;
  const int U = T * S;
  const int wgs = static_cast<int>(gridDim.x);
  const int wg = static_cast<int>(blockIdx.x);
  const int u0 = range_begin(U, wg, wgs), u1 = range_begin(U, wg + 1, wgs);
  const int t0 = u0 / S;
  const int t_last = (u1 - 1) / S;                   // t0 or t0 + 1

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 15, lk = lane >> 4;
  const int64_t row_bytes = K_aug >> 1;
  const int nb = K_aug >> 5;

  // The range's units in tile t0 (a) and in tile t0 + 1 (b); the first nA
  // waves split the first part, the others the second, so a wave's units lie
  // in one tile.  v counts steps from tile t0's first step.
  const int base = u0 - t0 * S;
  const int nu = u1 - u0;
  const int a_units = min(nu, S - base);
  const int nA = wave_split(a_units, nu, kWaves);
  const int slot = wave < nA ? 0 : 1;
  const int fw = slot == 0 ? wave : wave - nA;                 // wave within its part
  const int fn = slot == 0 ? nA : kWaves - nA;                 // waves of its part
  const int flen = slot == 0 ? a_units : nu - a_units;
  const int v0 = base + (slot == 0 ? 0 : a_units) + flen * fw / fn;
  const int cnt = flen * (fw + 1) / fn - flen * fw / fn;       // <= kU (host check)
  const int t = t0 + slot;

  // 1. Every load of the wave, unit by unit in the order the MFMAs consume
  //    them (the memory counter drains in issue order, so the wave waits only
  //    for the unit it needs next).  Units past cnt reload the wave's last
  //    unit (a wave without units: the range's first) and feed zero codes.
  const int tw = cnt > 0 ? t : t0;                               // the wave's tile
  const int sw0 = cnt > 0 ? v0 - slot * S : base;                // its first step
  const int jmax = cnt > 0 ? cnt - 1 : 0;
  uint4 w[kU];
  uint32_t wsd[kU];
  uint4 a[kU][kG];
  uint32_t as[kU][kG];
#pragma unroll
  for (int j = 0; j < kU; ++j) {
    const int s = sw0 + min(j, jmax);
    w[j] = *reinterpret_cast<const uint4*>(Wp + (static_cast<int64_t>(tw) * S + s) * 1024 + lane * 16);
    wsd[j] = reinterpret_cast<const uint32_t*>(Wps)[(static_cast<int64_t>(tw) * SG + (s >> 2)) * 64 + lane];
    const bool kin = s * kStepK + lk * 32 < K_aug;
#pragma unroll
    for (int g = 0; g < kG; ++g) {
      const int m = min(g * 16 + lr, M - 1);
      a[j][g] = *reinterpret_cast<const uint4*>(Aq + m * row_bytes + (kin ? s * 64 + lk * 16 : 0));
      as[j][g] = Asc[static_cast<int64_t>(m) * nb + (kin ? s * 4 + lk : 0)];
    }
    __builtin_amdgcn_sched_barrier(0);
  }

  // 2. The MFMAs, in load order.  acc[g][q] of this lane is
  //    Y[16 g + lr][16 tw + 4 lk + q] (partial over the wave's units).
  v4f acc[kG];
#pragma unroll
  for (int g = 0; g < kG; ++g) acc[g] = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int j = 0; j < kU; ++j) {
    const int s = sw0 + min(j, jmax);
    const bool kin = s * kStepK + lk * 32 < K_aug;
    const uint4 wj = j < cnt ? w[j] : make_uint4(0, 0, 0, 0);
    const uint32_t sw = (wsd[j] >> (8 * (s & 3))) & 0xFFu;
#pragma unroll
    for (int g = 0; g < kG; ++g) {
      const uint32_t sa = kin ? (as[j][g] & 0xFFu) : kNeutralScale;
      acc[g] = dev::mfma_fp4_16x16x128(wj, a[j][g], sw, sa, acc[g]);
    }
  }

  // 3. Sum the waves' accumulators through LDS (red[wave][g][lane][q]); a
  //    part's waves are added in wave order.
  float* const red = reinterpret_cast<float*>(smem);
#pragma unroll
  for (int g = 0; g < kG; ++g)
    *reinterpret_cast<v4f*>(red + ((wave * kG + g) * 64 + lane) * 4) = acc[g];
  __syncthreads();

  const int per = M * 16;                            // elements of one tile of Y
  constexpr int kThreads = kWaves * 64;
  constexpr int kPerThread = (kMaxRows * 16 + kThreads - 1) / kThreads;
  float own[2][kPerThread];
  bool partial[2] = {false, false};
#pragma unroll
  for (int f = 0; f < 2; ++f) {
    const int tf = t0 + f;
    if (tf > t_last) continue;
    const int tb = tf * S;
    partial[f] = u0 > tb || u1 < tb + S;
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
      const int idx = tid + i * kThreads;            // element (m, n) of the tile, n fastest
      if (idx < per) {
        const int m = idx >> 4, n = idx & 15;
        const int g = m >> 4, l = (n >> 2) * 16 + (m & 15), q = n & 3;
        float v = 0.0f;
        for (int wv = f == 0 ? 0 : nA; wv < (f == 0 ? nA : kWaves); ++wv)
          v += red[((wv * kG + g) * 64 + l) * 4 + q];
        own[f][i] = v;
        if (partial[f])
          __hip_atomic_store(part + (static_cast<int64_t>(wg) * 2 + f) * per + idx, v,
                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        else
          Y[static_cast<int64_t>(m) * N + tf * 16 + n] = v;
      }
    }
  }
  if (!partial[0] && !partial[1]) return;            // workgroup-uniform

  // 4. Arrival: the partial stores are complete before the counter moves.
  wait_all_vm();
  __syncthreads();
  if (tid < 2) {
    const int f = tid;
    int last = 0;
    if (f == 0 ? partial[0] : partial[1]) {
      const int t = t0 + f;
      const int tb = t * S;
      int wa = wg, wb = wg;
      while (wa > 0 && range_begin(U, wa, wgs) > tb) --wa;
      while (range_begin(U, wb + 1, wgs) < tb + S) ++wb;
      const uint32_t old =
          __hip_atomic_fetch_add(ctr + t, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      last = old == static_cast<uint32_t>(wb - wa) ? 1 : 0;
    }
    s_last[f] = last;
  }
  __syncthreads();

  // 5. The last arriver of a tile adds the covering workgroups' partials in
  //    workgroup order (all loads issued before the first add).
#pragma unroll
  for (int f = 0; f < 2; ++f) {
    if (!s_last[f]) continue;
    const int t = t0 + f;
    const int tb = t * S;
    int wa = wg, wb = wg;
    while (wa > 0 && range_begin(U, wa, wgs) > tb) --wa;
    while (range_begin(U, wb + 1, wgs) < tb + S) ++wb;   // wb - wa < kMaxFrags (host check)
    float pv[kMaxFrags][kPerThread];
#pragma unroll
    for (int x = 0; x < kMaxFrags; ++x) {
      const int w_x = wa + x;
      const bool load = w_x <= wb && w_x != wg;
      const int f_x = load && range_begin(U, w_x, wgs) / S != t ? 1 : 0;   // t: w_x's 1st or 2nd tile
#pragma unroll
      for (int i = 0; i < kPerThread; ++i) {
        const int idx = tid + i * kThreads;
        pv[x][i] = 0.0f;
        if (load && idx < per)
          pv[x][i] = __hip_atomic_load(part + (static_cast<int64_t>(w_x) * 2 + f_x) * per + idx,
                                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
      const int idx = tid + i * kThreads;
      if (idx < per) {
        float v = 0.0f;
#pragma unroll
        for (int x = 0; x < kMaxFrags; ++x)
          if (wa + x <= wb) v += wa + x == wg ? own[f][i] : pv[x][i];
        Y[static_cast<int64_t>(idx >> 4) * N + t * 16 + (idx & 15)] = v;
      }
    }
    if (tid == 0) __hip_atomic_store(ctr + t, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

template <int kWaves, int kU, int kG>
hipError_t launch_cfg(int wgs, const uint8_t* Aq, const uint8_t* Asc, int M, const uint8_t* Wp,
                      const uint8_t* Wps, int N, int K_aug, float* Y, float* part, uint32_t* ctr,
                      hipStream_t stream) {
  const size_t lds = static_cast<size_t>(kWaves) * kG * 256 * sizeof(float);
  static std::once_flag attr_once;   // dynamic LDS above the 64 KiB default
  std::call_once(attr_once, [lds] {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_streamk_kernel<kWaves, kU, kG>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
    (void)hipGetLastError();
  });
  gemm_streamk_kernel<kWaves, kU, kG><<<wgs, kWaves * 64, lds, stream>>>(Aq, Asc, M, Wp, Wps, N,
                                                                       K_aug, Y, part, ctr);
  return hipGetLastError();
}

template <int kU>
hipError_t launch_g(int G, int wgs, const uint8_t* Aq, const uint8_t* Asc, int M,
                    const uint8_t* Wp, const uint8_t* Wps, int N, int K_aug, float* Y, float* part,
                    uint32_t* ctr, hipStream_t stream) {
  switch (G) {
    case 1: return launch_cfg<8, kU, 1>(wgs, Aq, Asc, M, Wp, Wps, N, K_aug, Y, part, ctr, stream);
    case 2: return launch_cfg<8, kU, 2>(wgs, Aq, Asc, M, Wp, Wps, N, K_aug, Y, part, ctr, stream);
    case 3: return launch_cfg<8, kU, 3>(wgs, Aq, Asc, M, Wp, Wps, N, K_aug, Y, part, ctr, stream);
    default: return launch_cfg<8, kU, 4>(wgs, Aq, Asc, M, Wp, Wps, N, K_aug, Y, part, ctr, stream);
  }
}

constexpr int kStreamKWaves = 8;
const int kStreamKUnroll[] = {1, 2, 4, 7, 10};

}  // namespace

// The most units any wave of the launch gets: the kernel's split of each
// workgroup's range (one or two tile parts, waves dealt by wave_split),
// evaluated for every workgroup.
int streamk_max_wave_units(int64_t U, int S, int wgs, int waves) {
  int most = 0;
  for (int wg = 0; wg < wgs; ++wg) {
    const int64_t u0 = U * wg / wgs, u1 = U * (wg + 1) / wgs;
    const int base = static_cast<int>(u0 % S), nu = static_cast<int>(u1 - u0);
    const int a = std::min(nu, S - base);
    const int nA = wave_split(a, nu, waves);
    for (int w = 0; w < waves; ++w) {
      const bool first = w < nA;
      const int fw = first ? w : w - nA, fn = first ? nA : waves - nA, len = first ? a : nu - a;
      if (fn > 0) most = std::max(most, len * (fw + 1) / fn - len * fw / fn);
    }
  }
  return most;
}

namespace {

// The plan with exactly `wgs` workgroups (ok = false where it does not fit).
StreamKConfig streamk_plan(int M, int64_t T, int64_t S, int wgs) {
  StreamKConfig c;
  const int64_t U = T * S;
  c.groups = (std::max(M, 1) + 15) / 16;
  c.workgroups = static_cast<int>(std::min<int64_t>(wgs, U));
  // A range must touch at most two tiles: at most one tile of units per
  // workgroup; and every tile is shared by at most kMaxFrags workgroups (the
  // shortest range covers floor(U / workgroups) units).
  const int64_t per_wg = (U + c.workgroups - 1) / c.workgroups;
  const int64_t shortest = U / c.workgroups;
  if (per_wg > S || shortest < 1 || (S + shortest - 1) / shortest + 1 > kMaxFrags) return c;
  c.shared = U % c.workgroups != 0 || U / c.workgroups != S;   // else one tile per workgroup
  const int most = streamk_max_wave_units(U, static_cast<int>(S), c.workgroups, kStreamKWaves);
  c.unroll = 0;
  for (int x : kStreamKUnroll)
    if (x >= most) {
      c.unroll = x;
      break;
    }
  // ten units of four row groups would not fit a wave's registers
  c.ok = c.unroll > 0 && !(c.unroll > 7 && c.groups > 3);
  return c;
}

}  // namespace

StreamKConfig choose_streamk_config(int M, int N, int K_aug, int num_cus, int workgroups) {
  StreamKConfig c;
  const int64_t S = (K_aug + kStepK - 1) / kStepK;
  const int64_t T = N / 16;
  const int64_t U = T * S;
  const bool shape_ok = M >= 1 && M <= kMaxRows && N % 16 == 0 && T >= 1 &&
                        T <= kMaxStreamKTiles && K_aug > 0 && K_aug % 32 == 0 &&
                        U * std::max({num_cus, workgroups, 1}) < (int64_t{1} << 31);
  if (!shape_ok) return c;
  if (workgroups > 0) return streamk_plan(M, T, S, workgroups);
  // One workgroup per tile where the tiles fill at least half of the CUs (no
  // tile shared: no arrival protocol); else, or where that plan does not fit
  // the registers, one workgroup per CU.
  const int cus = std::max(num_cus, 1);
  if (T <= cus && 2 * T >= cus) {
    c = streamk_plan(M, T, S, static_cast<int>(T));
    if (c.ok) return c;
  }
  return streamk_plan(M, T, S, cus);
}

size_t streamk_workspace_bytes(int M, int N, int K_aug, int num_cus) {
  const StreamKConfig c = choose_streamk_config(M, N, K_aug, num_cus);
  if (!c.ok || !c.shared) return 0;
  return kWorkspaceStateBytes + static_cast<size_t>(c.workgroups) * 2 * M * 16 * sizeof(float);
}

hipError_t launch_gemm_streamk(const uint8_t* Aq, const uint8_t* Asc, int M, const uint8_t* Wp,
                               const uint8_t* Wps, int N, int K_aug, float* Y,
                               const StreamKConfig& c, void* workspace, hipStream_t stream) {
  uint32_t* ctr = static_cast<uint32_t*>(workspace);
  float* p = reinterpret_cast<float*>(static_cast<char*>(workspace) + kWorkspaceStateBytes);
  switch (c.unroll) {
    case 1: return launch_g<1>(c.groups, c.workgroups, Aq, Asc, M, Wp, Wps, N, K_aug, Y, p, ctr, stream);
    case 2: return launch_g<2>(c.groups, c.workgroups, Aq, Asc, M, Wp, Wps, N, K_aug, Y, p, ctr, stream);
    case 4: return launch_g<4>(c.groups, c.workgroups, Aq, Asc, M, Wp, Wps, N, K_aug, Y, p, ctr, stream);
    case 7: return launch_g<7>(c.groups, c.workgroups, Aq, Asc, M, Wp, Wps, N, K_aug, Y, p, ctr, stream);
    default: return launch_g<10>(c.groups, c.workgroups, Aq, Asc, M, Wp, Wps, N, K_aug, Y, p, ctr, stream);
  }
}

}  // namespace prq
