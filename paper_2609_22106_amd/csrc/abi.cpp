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

int check_gemm_common(const uint8_t* Aq, const uint8_t* Asc, int32_t M, const uint8_t* Wq,
                      const uint8_t* Wsc, int32_t N, int32_t K_aug, const float* Y) {
  if (M < 0 || N <= 0 || K_aug <= 0) return PRQ_EINVAL;
  if (!Wq || !Wsc) return PRQ_EINVAL;
  if (M > 0 && (!Aq || !Asc || !Y)) return PRQ_EINVAL;
  if (K_aug % PRQ_BLOCK) return PRQ_EALIGN;
  if (N % 16) return PRQ_EALIGN;
  if (K_aug > kMaxKAug) return PRQ_EUNSUPPORTED;
  if (!aligned16(Wq) || (M > 0 && (!aligned16(Aq) || (reinterpret_cast<uintptr_t>(Y) & 3u))))
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

int prq_quant_act(const void* X_bf16, int64_t ld_x, int32_t M, int32_t K, int32_t k_tail,
                  const float* inv_scale, const int32_t* perm, const int32_t* group_offsets,
                  int32_t G, uint8_t* Aq, uint8_t* Asc, hipStream_t stream) {
  if (M < 0 || K <= 0 || G < 1 || ld_x < K) return PRQ_EINVAL;
  if (G > 1 && !group_offsets) return PRQ_EINVAL;
  if (K % PRQ_BLOCK || k_tail < 0 || k_tail % PRQ_BLOCK || k_tail > K) return PRQ_EALIGN;
  if (K > kMaxK || G > kMaxGroups) return PRQ_EUNSUPPORTED;
  if (M == 0) return PRQ_OK;
  if (!X_bf16 || !Aq || !Asc) return PRQ_EINVAL;
  if (!aligned16(X_bf16) || ld_x % 8 || !aligned16(Aq)) return PRQ_EALIGN;
  if ((inv_scale && (reinterpret_cast<uintptr_t>(inv_scale) & 3u)) ||
      (perm && (reinterpret_cast<uintptr_t>(perm) & 3u)))
    return PRQ_EALIGN;
  DeviceInfo dev;
  int st = current_device(&dev);
  if (st != PRQ_OK) return st;
  return launch_status(prq::launch_act_quant(static_cast<const uint16_t*>(X_bf16), ld_x, M, K,
                                             k_tail, inv_scale, perm, group_offsets, G, Aq, Asc,
                                             dev.num_cus, stream));
}

size_t prq_gemm_workspace_bytes_ex(int32_t M, int32_t N, int32_t K_aug, int32_t variant,
                                   int32_t splits) {
  if (M <= 0 || N <= 0 || K_aug <= 0 || N % 16) return 0;
  if (variant == PRQ_GEMM_AUTO) variant = prq::choose_variant(M, N, K_aug);
  if (variant != PRQ_GEMM_STREAM) return 0;
  if (splits <= 0) {
    DeviceInfo dev;
    int cus = current_device(&dev) == PRQ_OK ? dev.num_cus : 256;
    splits = prq::choose_stream_splits(M, N, K_aug, cus);
  }
  return prq::stream_workspace_bytes(M, 1, N, splits);
}

size_t prq_gemm_workspace_bytes(int32_t M, int32_t N, int32_t K_aug) {
  return prq_gemm_workspace_bytes_ex(M, N, K_aug, PRQ_GEMM_AUTO, 0);
}

int prq_gemm_ex(const uint8_t* Aq, const uint8_t* Asc, int32_t M, const uint8_t* Wq,
                const uint8_t* Wsc, int32_t N, int32_t K_aug, float* Y, void* workspace,
                size_t workspace_bytes, int32_t variant, int32_t splits, hipStream_t stream) {
  int st = check_gemm_common(Aq, Asc, M, Wq, Wsc, N, K_aug, Y);
  if (st != PRQ_OK) return st;
  if (variant < PRQ_GEMM_AUTO || variant > PRQ_GEMM_STREAM || splits < 0) return PRQ_EINVAL;
  if (M == 0) return PRQ_OK;
  DeviceInfo dev;
  st = current_device(&dev);
  if (st != PRQ_OK) return st;
  if (variant == PRQ_GEMM_AUTO) variant = prq::choose_variant(M, N, K_aug);
  if (variant == PRQ_GEMM_TILE)
    return launch_status(prq::launch_gemm_tile(Aq, Asc, M, nullptr, 1, Wq, Wsc, N, K_aug, Y, stream));
  if (splits == 0) splits = prq::choose_stream_splits(M, N, K_aug, dev.num_cus);
  const int steps = (K_aug + 127) / 128;
  if (splits > steps) return PRQ_EINVAL;
  const size_t need = prq::stream_workspace_bytes(M, 1, N, splits);
  if (need && (!workspace || workspace_bytes < need || !aligned16(workspace))) return PRQ_EWORKSPACE;
  return launch_status(prq::launch_gemm_stream(Aq, Asc, M, nullptr, 1, Wq, Wsc, N, K_aug, Y, splits,
                                               workspace, stream));
}

int prq_gemm(const uint8_t* Aq, const uint8_t* Asc, int32_t M, const uint8_t* Wq,
             const uint8_t* Wsc, int32_t N, int32_t K_aug, float* Y, void* workspace,
             size_t workspace_bytes, hipStream_t stream) {
  return prq_gemm_ex(Aq, Asc, M, Wq, Wsc, N, K_aug, Y, workspace, workspace_bytes, PRQ_GEMM_AUTO,
                     0, stream);
}

size_t prq_grouped_gemm_workspace_bytes(int32_t M_total, int32_t E, int32_t N, int32_t K_aug) {
  (void)M_total;
  (void)E;
  (void)N;
  (void)K_aug;
  return 0;  // the grouped kernels run without split-K
}

int prq_grouped_gemm_ex(const uint8_t* Aq, const uint8_t* Asc, const int32_t* group_offsets,
                        int32_t E, int32_t M_total, const uint8_t* Wq, const uint8_t* Wsc,
                        int32_t N, int32_t K_aug, float* Y, void* workspace,
                        size_t workspace_bytes, int32_t variant, hipStream_t stream) {
  (void)workspace;
  (void)workspace_bytes;
  int st = check_gemm_common(Aq, Asc, M_total, Wq, Wsc, N, K_aug, Y);
  if (st != PRQ_OK) return st;
  if (E < 1 || !group_offsets) return PRQ_EINVAL;
  if (E > kMaxGroups) return PRQ_EUNSUPPORTED;
  if (variant < PRQ_GEMM_AUTO || variant > PRQ_GEMM_STREAM) return PRQ_EINVAL;
  if (M_total == 0) return PRQ_OK;
  DeviceInfo dev;
  st = current_device(&dev);
  if (st != PRQ_OK) return st;
  if (variant == PRQ_GEMM_AUTO) variant = prq::choose_variant((M_total + E - 1) / E, N, K_aug);
  if (variant == PRQ_GEMM_TILE)
    return launch_status(
        prq::launch_gemm_tile(Aq, Asc, M_total, group_offsets, E, Wq, Wsc, N, K_aug, Y, stream));
  return launch_status(prq::launch_gemm_stream(Aq, Asc, M_total, group_offsets, E, Wq, Wsc, N, K_aug,
                                               Y, 1, nullptr, stream));
}

int prq_grouped_gemm(const uint8_t* Aq, const uint8_t* Asc, const int32_t* group_offsets, int32_t E,
                     int32_t M_total, const uint8_t* Wq, const uint8_t* Wsc, int32_t N,
                     int32_t K_aug, float* Y, void* workspace, size_t workspace_bytes,
                     hipStream_t stream) {
  return prq_grouped_gemm_ex(Aq, Asc, group_offsets, E, M_total, Wq, Wsc, N, K_aug, Y, workspace,
                             workspace_bytes, PRQ_GEMM_AUTO, stream);
}

}  // extern "C"
