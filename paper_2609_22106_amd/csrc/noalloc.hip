// prq_gemm_noalloc: prq_gemm with its workspace in a file-scope device array
// instead of a caller buffer, for callers that cannot allocate device memory
// (code under HIP graph capture, serving loops that must not allocate,
// harnesses that forbid it).
//
// The array (kNoAllocScratchBytes, held by every GPU the library runs on until
// the process ends) has the layout of any GEMM workspace: a zero-state head
// (the stream-K arrival counters, zero at load and left zero by every call)
// and the scratch of the kernel that runs.  Host code never passes the
// array's name to a kernel (in host code it is a stand-in, not a device
// address): the device address comes from hipGetSymbolAddress, taken once per
// device with that device current and kept per device.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>

#include "prq.h"
#include "prq_internal.h"

namespace {

constexpr size_t kNoAllocScratchBytes = size_t{16} << 20;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};

// The current device's address of `scratch` (taken on the device's first call).
int scratch_address(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return PRQ_EDEVICE;
  }
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      (void)hipGetLastError();
      return PRQ_EDEVICE;
    }
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return PRQ_OK;
}

}  // namespace

extern "C" {

size_t prq_gemm_noalloc_max_workspace_bytes(void) { return kNoAllocScratchBytes; }

int prq_gemm_noalloc(const uint8_t* Aq, const uint8_t* Asc, int32_t M, const uint8_t* Wp,
                     const uint8_t* Wps, int32_t N, int32_t K_aug, float* Y, hipStream_t stream) {
  if (M < 0 || N <= 0 || K_aug <= 0) return PRQ_EINVAL;
  if (M == 0) return prq_gemm(Aq, Asc, M, Wp, Wps, N, K_aug, Y, nullptr, 0, stream);
  // the call's plan with a workspace of any size must fit the array
  if (prq_gemm_workspace_bytes(M, N, K_aug) > kNoAllocScratchBytes) return PRQ_EWORKSPACE;
  void* ws = nullptr;
  const int st = scratch_address(&ws);
  if (st != PRQ_OK) return st;
  return prq_gemm(Aq, Asc, M, Wp, Wps, N, K_aug, Y, ws, kNoAllocScratchBytes, stream);
}

}  // extern "C"
