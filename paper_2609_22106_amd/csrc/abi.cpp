// C ABI of libprq.so: argument validation, device check, kernel selection and
// workspace sizing for the device calls declared in include/prq.h.
#include <array>
#include <cstdint>
#include <cstring>
#include <mutex>

#include <hip/hip_runtime_api.h>

#include "prq.h"
#include "prq_internal.h"

namespace {

constexpr int kMaxDevices = 64;
constexpr int kMaxK = 16384;        // activation row staged in LDS with its perm and scales
constexpr int kMaxKAug = 65536;
constexpr int kMaxGroups = 4096;

struct DeviceInfo {
  bool gfx950 = false;
  int num_cus = 0;
};

std::mutex g_dev_mu;
std::array<int, kMaxDevices> g_dev_state{};  // 0 unknown, 1 known
std::array<DeviceInfo, kMaxDevices> g_dev_info{};

// Properties of the current device, cached per device.
int current_device(DeviceInfo* out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return PRQ_EDEVICE;
  }
  std::lock_guard<std::mutex> lk(g_dev_mu);
  if (!g_dev_state[dev]) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) {
      (void)hipGetLastError();
      return PRQ_EDEVICE;
    }
    DeviceInfo info;
    info.gfx950 = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0;
    info.num_cus = prop.multiProcessorCount;
    g_dev_info[dev] = info;
    g_dev_state[dev] = 1;
  }
  *out = g_dev_info[dev];
  return out->gfx950 ? PRQ_OK : PRQ_EUNSUPPORTED;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int launch_status(hipError_t e) { return e == hipSuccess ? PRQ_OK : PRQ_EDEVICE; }

int check_gemm_common(const uint8_t* Aq, const uint8_t* Asc, int32_t M, const uint8_t* Wp,
                      const uint8_t* Wps, int32_t N, int32_t K_aug, const float* Y) {
  if (M < 0 || N <= 0 || K_aug <= 0) return PRQ_EINVAL;
  if (!Wp || !Wps) return PRQ_EINVAL;
  if (M > 0 && (!Aq || !Asc || !Y)) return PRQ_EINVAL;
  if (K_aug % PRQ_BLOCK) return PRQ_EALIGN;
  if (N % 16) return PRQ_EALIGN;
  if (K_aug > kMaxKAug) return PRQ_EUNSUPPORTED;
  if (!aligned16(Wp) || !aligned16(Wps) ||
      (M > 0 && (!aligned16(Aq) || (reinterpret_cast<uintptr_t>(Y) & 3u))))
    return PRQ_EALIGN;
  return PRQ_OK;
}

}  // namespace

extern "C" {

const char* prq_strerror(int status) {
  switch (status) {
    case PRQ_OK: return "success";
    case PRQ_EINVAL: return "invalid argument (null pointer, negative size, alpha, mode or variant)";
    case PRQ_EALIGN: return "alignment: K and k_tail must be multiples of 32 with k_tail <= K, "
                            "K_aug = K + k_tail, 16-byte aligned pointers and rows, N % 16 == 0";
    case PRQ_EDEVICE: return "HIP runtime error";
    case PRQ_EUNSUPPORTED: return "unsupported: device is not gfx950 or size beyond the limits";
    case PRQ_EWORKSPACE: return "workspace missing or too small";
    default: return "unknown status";
  }
}

int prq_abi_version(void) { return PRQ_ABI_VERSION; }

int prq_packed_weight_bytes(int32_t E, int32_t N, int32_t K_aug, size_t* code_bytes,
                            size_t* scale_bytes) {
  if (E < 1 || N <= 0 || K_aug <= 0 || !code_bytes || !scale_bytes) return PRQ_EINVAL;
  if (N % 16 || K_aug % PRQ_BLOCK) return PRQ_EALIGN;
  if (K_aug > kMaxKAug || E > kMaxGroups) return PRQ_EUNSUPPORTED;
  *code_bytes = prq::packed_code_bytes(N, K_aug, E);
  *scale_bytes = prq::packed_scale_bytes(N, K_aug, E);
  return PRQ_OK;
}

int prq_pack_weight(const uint8_t* Wq, const uint8_t* Wsc, int32_t E, int32_t N, int32_t K_aug,
                    uint8_t* Wp, uint8_t* Wps, hipStream_t stream) {
  size_t cb = 0, sb = 0;
  int st = prq_packed_weight_bytes(E, N, K_aug, &cb, &sb);
  if (st != PRQ_OK) return st;
  if (!Wq || !Wsc || !Wp || !Wps) return PRQ_EINVAL;
  if (!aligned16(Wq) || !aligned16(Wp) || !aligned16(Wps)) return PRQ_EALIGN;
  DeviceInfo dev;
  st = current_device(&dev);
  if (st != PRQ_OK) return st;
  return launch_status(prq::launch_pack_weight(Wq, Wsc, N, K_aug, E, Wp, Wps, stream));
}

int prq_quant_act(const void* X_bf16, int64_t ld_x, int32_t M, int32_t K, int32_t k_tail,
                  const float* inv_scale_pos, const int32_t* perm, const int32_t* group_offsets,
                  int32_t G, uint8_t* Aq, uint8_t* Asc, hipStream_t stream) {
  if (M < 0 || K <= 0 || G < 1 || ld_x < K) return PRQ_EINVAL;
  if (G > 1 && !group_offsets) return PRQ_EINVAL;
  if (K % PRQ_BLOCK || k_tail < 0 || k_tail % PRQ_BLOCK || k_tail > K) return PRQ_EALIGN;
  if (K > kMaxK || G > kMaxGroups) return PRQ_EUNSUPPORTED;
  if (M == 0) return PRQ_OK;
  if (!X_bf16 || !Aq || !Asc) return PRQ_EINVAL;
  if (!aligned16(X_bf16) || ld_x % 8 || !aligned16(Aq)) return PRQ_EALIGN;
  if ((inv_scale_pos && !aligned16(inv_scale_pos)) || (perm && !aligned16(perm)))
    return PRQ_EALIGN;
  DeviceInfo dev;
  int st = current_device(&dev);
  if (st != PRQ_OK) return st;
  return launch_status(prq::launch_act_quant(static_cast<const uint16_t*>(X_bf16), ld_x, M, K,
                                             k_tail, inv_scale_pos, perm, group_offsets, G, Aq, Asc,
                                             dev.num_cus, stream));
}

}  // extern "C"

namespace {

// Stream-kernel configuration for a dense call; splits_req > 0 forces the
// split count (the wave count and unroll are then re-derived for coverage).
prq::StreamConfig dense_stream_config(int M, int N, int K_aug, int splits_req, int num_cus) {
  prq::StreamConfig c = prq::choose_stream_config(M, N, K_aug, 0, num_cus);
  // split-K through the ABI always adds partial sums in a fixed order (the
  // workspace's scratch then never has to start at zero)
  c.reduce = 1;
  if (splits_req > 0 && splits_req != c.splits) {
    const int steps = (K_aug + 127) / 128;
    c.splits = splits_req;
    static const int kU[] = {1, 2, 3, 4, 6, 8};
    c.ok = false;
    const prq::StreamConfig base = c;
    for (int cand = 0; cand < 4 && !c.ok; ++cand) {  // keep the shape if it still covers K_aug
      c.tiles = (cand & 1) ? 1 : base.tiles;
      c.waves = (cand & 2) ? 16 : base.waves;
      const int chunks = c.waves / c.tiles;
      const int need = ((steps + c.splits - 1) / c.splits + chunks - 1) / chunks;
      c.unroll = 0;
      for (int x : kU)
        if (x >= need) {
          c.unroll = x;
          break;
        }
      c.ok = c.unroll > 0 && splits_req <= steps && prq::stream_config_covers(c, K_aug);
    }
  }
  return c;
}

// Workspace layout shared by every GEMM call: the state head (stream-K arrival
// counters, zero between calls), then the scratch of the kernel that runs.
size_t with_head(size_t scratch) { return scratch ? prq::kWorkspaceStateBytes + scratch : 0; }

void* scratch_of(void* workspace, size_t workspace_bytes) {
  return workspace && workspace_bytes > prq::kWorkspaceStateBytes
             ? static_cast<char*>(workspace) + prq::kWorkspaceStateBytes
             : nullptr;
}

size_t scratch_bytes(const void* workspace, size_t workspace_bytes) {
  return workspace && workspace_bytes > prq::kWorkspaceStateBytes
             ? workspace_bytes - prq::kWorkspaceStateBytes
             : 0;
}

int device_cus() {
  DeviceInfo dev;
  return current_device(&dev) == PRQ_OK ? dev.num_cus : 256;
}

// The variant an AUTO call runs: the whole-K decode kernel up to 64 rows, the
// LDS-tiled kernel above.  The stream-K kernel (PRQ_GEMM_STREAM_K) is not an
// AUTO choice: since the decode kernel stages each row group's activation in
// whole-row copies it is as fast or faster at every measured shape (weights
// rotated, back-to-back launches, decode / stream-K): 9728 -> 2560 M = 1 5.1 /
// 5.3 us, M = 8 5.5 / 6.3; 9728 -> 1792 (112 tiles, stream-K sharing tiles
// over all CUs) M = 1 5.1 / 8.2, M = 8 5.2 / 8.7; 2560 -> 4096 M = 8 3.9 /
// 4.0; 4096 -> 2560 M = 8 4.5 / 4.8.
int auto_variant(int M, int N, int K_aug) { return prq::choose_variant(M, N, K_aug); }

}  // namespace

extern "C" {

size_t prq_gemm_workspace_bytes_ex(int32_t M, int32_t N, int32_t K_aug, int32_t variant,
                                   int32_t splits) {
  if (M <= 0 || N <= 0 || K_aug <= 0 || N % 16 || K_aug % PRQ_BLOCK || splits < 0) return 0;
  if (variant == PRQ_GEMM_AUTO) variant = auto_variant(M, N, K_aug);
  if (variant == PRQ_GEMM_STREAM_K) return prq::streamk_workspace_bytes(M, N, K_aug, device_cus());
  if (variant == PRQ_GEMM_TILE)
    return with_head(prq::tile_workspace_bytes(M, N, K_aug, false, device_cus()));
  if (variant != PRQ_GEMM_STREAM) return 0;
  if (splits <= 1 && prq::choose_decode_config(M, N, K_aug, 0, 0, 0, device_cus()).ok) return 0;
  const prq::StreamConfig c = dense_stream_config(M, N, K_aug, splits, device_cus());
  return c.ok ? with_head(prq::stream_workspace_bytes(M, 1, N, c.splits, c.reduce)) : 0;
}

size_t prq_gemm_workspace_bytes(int32_t M, int32_t N, int32_t K_aug) {
  return prq_gemm_workspace_bytes_ex(M, N, K_aug, PRQ_GEMM_AUTO, 0);
}

int prq_gemm_ex(const uint8_t* Aq, const uint8_t* Asc, int32_t M, const uint8_t* Wp,
                const uint8_t* Wps, int32_t N, int32_t K_aug, float* Y, void* workspace,
                size_t workspace_bytes, int32_t variant, int32_t splits, hipStream_t stream) {
  int st = check_gemm_common(Aq, Asc, M, Wp, Wps, N, K_aug, Y);
  if (st != PRQ_OK) return st;
  if (variant < PRQ_GEMM_AUTO || variant > PRQ_GEMM_STREAM_K || splits < 0) return PRQ_EINVAL;
  if (M == 0) return PRQ_OK;
  DeviceInfo dev;
  st = current_device(&dev);
  if (st != PRQ_OK) return st;
  if (variant == PRQ_GEMM_AUTO) variant = auto_variant(M, N, K_aug);
  if (variant == PRQ_GEMM_STREAM_K) {
    const prq::StreamKConfig c = prq::choose_streamk_config(M, N, K_aug, dev.num_cus);
    if (!c.ok) return PRQ_EUNSUPPORTED;
    const size_t need = prq::streamk_workspace_bytes(M, N, K_aug, dev.num_cus);
    if (need && (!workspace || workspace_bytes < need || !aligned16(workspace)))
      return PRQ_EWORKSPACE;
    return launch_status(prq::launch_gemm_streamk(Aq, Asc, M, Wp, Wps, N, K_aug, Y, c, workspace,
                                                  stream));
  }
  if (variant == PRQ_GEMM_STREAM && splits <= 1) {
    // no split-K: the decode kernel, unless K_aug exceeds what it stages
    const prq::DecodeConfig d = prq::choose_decode_config(M, N, K_aug, 0, 0, 0, dev.num_cus);
    if (d.ok)
      return launch_status(prq::launch_gemm_decode(Aq, Asc, M, nullptr, 1, Wp, Wps, N, K_aug, Y, d,
                                                   stream));
  }
  if (variant == PRQ_GEMM_STREAM) {
    const prq::StreamConfig c = dense_stream_config(M, N, K_aug, splits, dev.num_cus);
    if (!c.ok) {
      if (splits > 0) return PRQ_EINVAL;   // the forced split count cannot cover K_aug
      variant = PRQ_GEMM_TILE;
    } else {
      const size_t need = with_head(prq::stream_workspace_bytes(M, 1, N, c.splits, c.reduce));
      if (need && (!workspace || workspace_bytes < need || !aligned16(workspace)))
        return PRQ_EWORKSPACE;
      return launch_status(prq::launch_gemm_stream(Aq, Asc, M, nullptr, 1, Wp, Wps, N, K_aug, Y, c,
                                                   scratch_of(workspace, workspace_bytes), stream));
    }
  }
  return launch_status(prq::launch_gemm_tile_planned(
      Aq, Asc, M, Wp, Wps, N, K_aug, Y, false, dev.num_cus, scratch_of(workspace, workspace_bytes),
      scratch_bytes(workspace, workspace_bytes), stream));
}

int prq_gemm(const uint8_t* Aq, const uint8_t* Asc, int32_t M, const uint8_t* Wp,
             const uint8_t* Wps, int32_t N, int32_t K_aug, float* Y, void* workspace,
             size_t workspace_bytes, hipStream_t stream) {
  return prq_gemm_ex(Aq, Asc, M, Wp, Wps, N, K_aug, Y, workspace, workspace_bytes, PRQ_GEMM_AUTO,
                     0, stream);
}

int prq_packed_act_bytes(int32_t M, int32_t K_aug, size_t* code_bytes, size_t* scale_bytes) {
  if (M < 0 || K_aug <= 0 || !code_bytes || !scale_bytes) return PRQ_EINVAL;
  if (K_aug % PRQ_BLOCK) return PRQ_EALIGN;
  if (K_aug > kMaxKAug) return PRQ_EUNSUPPORTED;
  const size_t blocks = (static_cast<size_t>(M) + 15) / 16;
  const size_t steps = (static_cast<size_t>(K_aug) + 127) / 128;
  *code_bytes = blocks * steps * 1024;
  *scale_bytes = blocks * ((steps + 3) / 4) * 256;
  return PRQ_OK;
}

int prq_quant_act_packed(const void* X_bf16, int64_t ld_x, int32_t M, int32_t K, int32_t k_tail,
                         const float* inv_scale_pos, const int32_t* perm,
                         const int32_t* group_offsets, int32_t G, uint8_t* Ap, uint8_t* Aps,
                         hipStream_t stream) {
  if (M < 0 || K <= 0 || G < 1 || ld_x < K) return PRQ_EINVAL;
  if (G > 1 && !group_offsets) return PRQ_EINVAL;
  if (K % PRQ_BLOCK || k_tail < 0 || k_tail % PRQ_BLOCK || k_tail > K) return PRQ_EALIGN;
  if (K > kMaxK || G > kMaxGroups) return PRQ_EUNSUPPORTED;
  if (M == 0) return PRQ_OK;
  if (!X_bf16 || !Ap || !Aps) return PRQ_EINVAL;
  if (!aligned16(X_bf16) || ld_x % 8 || !aligned16(Ap) || !aligned16(Aps)) return PRQ_EALIGN;
  if ((inv_scale_pos && !aligned16(inv_scale_pos)) || (perm && !aligned16(perm)))
    return PRQ_EALIGN;
  DeviceInfo dev;
  int st = current_device(&dev);
  if (st != PRQ_OK) return st;
  return launch_status(prq::launch_act_quant_packed(static_cast<const uint16_t*>(X_bf16), ld_x, M,
                                                    K, k_tail, inv_scale_pos, perm, group_offsets,
                                                    G, Ap, Aps, dev.num_cus, stream));
}

namespace {

int swiglu_quant_common(const void* gate, const void* up, int64_t ld, int32_t M, int32_t K_aug,
                        uint8_t* A, uint8_t* As, bool packed, hipStream_t stream) {
  if (M < 0 || K_aug <= 0 || ld < K_aug) return PRQ_EINVAL;
  if (K_aug % PRQ_BLOCK) return PRQ_EALIGN;
  if (K_aug > kMaxKAug) return PRQ_EUNSUPPORTED;
  if (M == 0) return PRQ_OK;
  if (!gate || !up || !A || !As) return PRQ_EINVAL;
  if (!aligned16(gate) || !aligned16(up) || ld % 8) return PRQ_EALIGN;
  if (packed && (!aligned16(A) || !aligned16(As))) return PRQ_EALIGN;
  DeviceInfo dev;
  const int st = current_device(&dev);
  if (st != PRQ_OK) return st;
  return launch_status(prq::launch_swiglu_quant(static_cast<const uint16_t*>(gate),
                                                static_cast<const uint16_t*>(up), ld, M, K_aug, A,
                                                As, packed, dev.num_cus, stream));
}

}  // namespace

int prq_swiglu_quant(const void* gate_bf16, const void* up_bf16, int64_t ld, int32_t M,
                     int32_t K_aug, uint8_t* Aq, uint8_t* Asc, hipStream_t stream) {
  return swiglu_quant_common(gate_bf16, up_bf16, ld, M, K_aug, Aq, Asc, false, stream);
}

int prq_swiglu_quant_packed(const void* gate_bf16, const void* up_bf16, int64_t ld, int32_t M,
                            int32_t K_aug, uint8_t* Ap, uint8_t* Aps, hipStream_t stream) {
  return swiglu_quant_common(gate_bf16, up_bf16, ld, M, K_aug, Ap, Aps, true, stream);
}

size_t prq_gemm_packed_workspace_bytes(int32_t M, int32_t N, int32_t K_aug) {
  if (M <= 0 || N <= 0 || K_aug <= 0 || N % 16 || K_aug % PRQ_BLOCK || K_aug > kMaxKAug) return 0;
  if (prq::choose_variant(M, N, K_aug) == PRQ_GEMM_STREAM &&
      prq::choose_decode_config(M, N, K_aug, 0, 0, 0, device_cus()).ok)
    return 0;   // the decode kernel: no workspace
  return with_head(prq::tile_workspace_bytes(M, N, K_aug, true, device_cus()));
}

int prq_gemm_packed(const uint8_t* Ap, const uint8_t* Aps, int32_t M, const uint8_t* Wp,
                    const uint8_t* Wps, int32_t N, int32_t K_aug, float* Y, void* workspace,
                    size_t workspace_bytes, hipStream_t stream) {
  int st = check_gemm_common(Ap, Aps, M, Wp, Wps, N, K_aug, Y);
  if (st != PRQ_OK) return st;
  if (M == 0) return PRQ_OK;
  if (!aligned16(Aps)) return PRQ_EALIGN;
  DeviceInfo dev;
  st = current_device(&dev);
  if (st != PRQ_OK) return st;
  // decode rows: the whole-K decode kernel on the packed operand (each row
  // group's operand one contiguous kilobyte per K step)
  if (prq::choose_variant(M, N, K_aug) == PRQ_GEMM_STREAM) {
    const prq::DecodeConfig d = prq::choose_decode_config(M, N, K_aug, 0, 0, 0, dev.num_cus, true);
    if (d.ok)
      return launch_status(prq::launch_gemm_decode(Ap, Aps, M, nullptr, 1, Wp, Wps, N, K_aug, Y, d,
                                                   stream, true));
  }
  return launch_status(prq::launch_gemm_tile_planned(
      Ap, Aps, M, Wp, Wps, N, K_aug, Y, true, dev.num_cus, scratch_of(workspace, workspace_bytes),
      scratch_bytes(workspace, workspace_bytes), stream));
}

int prq_grouped_gemm_packed(const uint8_t* Ap, const uint8_t* Aps, const int32_t* group_offsets,
                            int32_t E, int32_t M_total, const uint8_t* Wp, const uint8_t* Wps,
                            int32_t N, int32_t K_aug, float* Y, hipStream_t stream) {
  int st = check_gemm_common(Ap, Aps, M_total, Wp, Wps, N, K_aug, Y);
  if (st != PRQ_OK) return st;
  if (E < 1 || !group_offsets) return PRQ_EINVAL;
  if (E > kMaxGroups) return PRQ_EUNSUPPORTED;
  if (M_total == 0) return PRQ_OK;
  if (!aligned16(Aps)) return PRQ_EALIGN;
  DeviceInfo dev;
  st = current_device(&dev);
  if (st != PRQ_OK) return st;
  const int per_group = (M_total + E - 1) / E;
  return launch_status(prq::launch_grouped_gemm_tile_packed(
      Ap, Aps, M_total, group_offsets, E, Wp, Wps, N, K_aug, Y,
      prq::choose_grouped_packed_shape(per_group, N, K_aug, E), dev.num_cus, stream));
}

size_t prq_grouped_gemm_workspace_bytes(int32_t M_total, int32_t E, int32_t N, int32_t K_aug) {
  (void)M_total;
  (void)E;
  (void)N;
  (void)K_aug;
  return 0;  // the grouped kernels run without split-K
}

int prq_grouped_gemm_ex(const uint8_t* Aq, const uint8_t* Asc, const int32_t* group_offsets,
                        int32_t E, int32_t M_total, const uint8_t* Wp, const uint8_t* Wps,
                        int32_t N, int32_t K_aug, float* Y, void* workspace,
                        size_t workspace_bytes, int32_t variant, hipStream_t stream) {
  (void)workspace;
  (void)workspace_bytes;
  int st = check_gemm_common(Aq, Asc, M_total, Wp, Wps, N, K_aug, Y);
  if (st != PRQ_OK) return st;
  if (E < 1 || !group_offsets) return PRQ_EINVAL;
  if (E > kMaxGroups) return PRQ_EUNSUPPORTED;
  if (variant < PRQ_GEMM_AUTO || variant > PRQ_GEMM_STREAM) return PRQ_EINVAL;
  if (M_total == 0) return PRQ_OK;
  DeviceInfo dev;
  st = current_device(&dev);
  if (st != PRQ_OK) return st;
  const int per_group = (M_total + E - 1) / E;
  if (variant == PRQ_GEMM_AUTO) variant = prq::choose_variant(per_group, N, K_aug);
  if (variant == PRQ_GEMM_STREAM) {
    // (the decode kernel's grouped mode measured 2x slower on the expert
    // shapes, whose few K steps leave most of its 16 waves idle)
    const prq::StreamConfig c = prq::choose_stream_config(per_group, N, K_aug, 1, dev.num_cus);
    if (c.ok && prq::stream_config_covers(c, K_aug))
      return launch_status(prq::launch_gemm_stream(Aq, Asc, M_total, group_offsets, E, Wp, Wps, N,
                                                   K_aug, Y, c, nullptr, stream));
  }
  // Row tiles are per expert: pick the shape from the mean rows per expert
  // (~256 rows per expert at N = 2048, K + k = 832: 176 us with 256 x 256
  // tiles, 194 with 128 x 128, 248 with 256 x 128).
  const int shape = per_group >= 192 ? 0 : 2;
  return launch_status(prq::launch_gemm_tile(Aq, Asc, M_total, group_offsets, E, Wp, Wps, N, K_aug,
                                             Y, shape, stream));
}

int prq_grouped_gemm(const uint8_t* Aq, const uint8_t* Asc, const int32_t* group_offsets, int32_t E,
                     int32_t M_total, const uint8_t* Wp, const uint8_t* Wps, int32_t N,
                     int32_t K_aug, float* Y, void* workspace, size_t workspace_bytes,
                     hipStream_t stream) {
  return prq_grouped_gemm_ex(Aq, Asc, group_offsets, E, M_total, Wp, Wps, N, K_aug, Y, workspace,
                             workspace_bytes, PRQ_GEMM_AUTO, stream);
}

}  // extern "C"
