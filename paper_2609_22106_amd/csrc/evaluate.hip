// Offline evaluation of the reconstruction error and the alpha search of
// Algorithm 1 (arXiv 2609.22106): for every candidate alpha, construct the
// scaling, selection, permutation and augmented weight (prq_prepare_ex), then
// evaluate Eq. 3 on the calibration activations with the device path
// (prq_pack_weight, prq_quant_act, prq_gemm) and keep the alpha whose
// normalized reconstruction error ||Y_hat - X W^T||_F / ||X W^T||_F is
// smallest (the first on equal errors).  The unquantized reference X W^T is
// computed once on the device from the bf16 inputs with float32 accumulation.
//
// These calls are offline: they take host arrays, allocate their own device
// buffers, run on the given stream and synchronize it before returning.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstring>
#include <vector>

#include "prq.h"
#include "prq_internal.h"

namespace prq {
namespace {

constexpr int kRefTile = 64;     // 64 x 64 outputs per 256-thread workgroup
constexpr int kRefK = 32;        // K chunk staged in LDS
constexpr int kErrThreads = 256;

__device__ __forceinline__ float bf16_value(uint16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

// Y[m, n] = sum_k X[m, k] W[n, k] (bf16 inputs, float32 accumulation in k order).
__global__ __launch_bounds__(256) void reference_product_kernel(const uint16_t* __restrict__ X,
                                                                const uint16_t* __restrict__ W,
                                                                int M, int N, int K,
                                                                float* __restrict__ Y) {
  __shared__ float xs[kRefTile][kRefK + 1];
  __shared__ float ws[kRefTile][kRefK + 1];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;   // 16 x 16 threads, 4 x 4 outputs each
  const int m0 = blockIdx.y * kRefTile, n0 = blockIdx.x * kRefTile;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += kRefK) {
    for (int i = threadIdx.x; i < kRefTile * kRefK; i += 256) {
      const int r = i / kRefK, c = i % kRefK;
      const int k = k0 + c;
      xs[r][c] = (m0 + r < M && k < K) ? bf16_value(X[static_cast<int64_t>(m0 + r) * K + k]) : 0.0f;
      ws[r][c] = (n0 + r < N && k < K) ? bf16_value(W[static_cast<int64_t>(n0 + r) * K + k]) : 0.0f;
    }
    __syncthreads();
    for (int c = 0; c < kRefK; ++c) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(xs[ty * 4 + i][c], ws[tx * 4 + j][c], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int m = m0 + ty * 4 + i, n = n0 + tx * 4 + j;
      if (m < M && n < N) Y[static_cast<int64_t>(m) * N + n] = acc[i][j];
    }
}

// Per-workgroup sums of (Y - R)^2 and R^2 in double: partial[2 b], partial[2 b + 1].
__global__ __launch_bounds__(kErrThreads) void squared_error_kernel(const float* __restrict__ Y,
                                                                    const float* __restrict__ R,
                                                                    int64_t n, int64_t per_block,
                                                                    double* __restrict__ partial) {
  __shared__ double s_e[kErrThreads], s_r[kErrThreads];
  const int64_t b0 = static_cast<int64_t>(blockIdx.x) * per_block;
  const int64_t b1 = b0 + per_block < n ? b0 + per_block : n;
  double e = 0.0, r = 0.0;
  for (int64_t i = b0 + threadIdx.x; i < b1; i += kErrThreads) {
    const double d = static_cast<double>(Y[i]) - static_cast<double>(R[i]);
    e += d * d;
    r += static_cast<double>(R[i]) * static_cast<double>(R[i]);
  }
  s_e[threadIdx.x] = e;
  s_r[threadIdx.x] = r;
  __syncthreads();
  for (int s = kErrThreads / 2; s > 0; s >>= 1) {
    if (static_cast<int>(threadIdx.x) < s) {
      s_e[threadIdx.x] += s_e[threadIdx.x + s];
      s_r[threadIdx.x] += s_r[threadIdx.x + s];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    partial[2 * blockIdx.x] = s_e[0];
    partial[2 * blockIdx.x + 1] = s_r[0];
  }
}

// Device buffers freed on scope exit.
struct DeviceBuffers {
  std::vector<void*> ptrs;
  ~DeviceBuffers() {
    for (void* p : ptrs) (void)hipFree(p);
  }
  template <class T>
  int alloc(T** out, size_t count) {
    void* p = nullptr;
    if (hipMalloc(&p, count * sizeof(T) > 0 ? count * sizeof(T) : 16) != hipSuccess) return PRQ_EDEVICE;
    ptrs.push_back(p);
    *out = static_cast<T*>(p);
    return PRQ_OK;
  }
};

#define PRQ_TRY(expr)              \
  do {                             \
    const int st_ = (expr);        \
    if (st_ != PRQ_OK) return st_; \
  } while (0)

int hip_status(hipError_t e) { return e == hipSuccess ? PRQ_OK : PRQ_EDEVICE; }

// Evaluation of one or more alphas on M rows X (host bf16), against the
// reference on the same rows; writes nrmse[a] for each alpha.
int evaluate_alphas(const uint16_t* W_bf16, int32_t N, int32_t K, const uint16_t* Xcal_bf16,
                    int32_t T, const uint16_t* X_bf16, int32_t M, const double* alphas,
                    int32_t n_alpha, int32_t k_tail, int32_t scale_mode, int32_t flags,
                    double* nrmse, hipStream_t stream) {
  const int64_t K_aug = static_cast<int64_t>(K) + k_tail;
  DeviceBuffers buf;
  uint16_t *dW = nullptr, *dX = nullptr;
  float *dYref = nullptr, *dY = nullptr, *dInv = nullptr;
  int32_t* dPerm = nullptr;
  uint8_t *dWq = nullptr, *dWsc = nullptr, *dAq = nullptr, *dAsc = nullptr, *dWp = nullptr,
          *dWps = nullptr, *dWs = nullptr;
  double* dPartial = nullptr;
  size_t code_bytes = 0, scale_bytes = 0;
  PRQ_TRY(prq_packed_weight_bytes(1, N, static_cast<int32_t>(K_aug), &code_bytes, &scale_bytes));
  const size_t ws_bytes = prq_gemm_workspace_bytes(M, N, static_cast<int32_t>(K_aug));
  const int64_t outs = static_cast<int64_t>(M) * N;
  const int err_blocks = static_cast<int>(std::min<int64_t>(1024, (outs + 4095) / 4096));
  const int64_t per_block = (outs + err_blocks - 1) / err_blocks;
  PRQ_TRY(buf.alloc(&dW, static_cast<size_t>(N) * K));
  PRQ_TRY(buf.alloc(&dX, static_cast<size_t>(M) * K));
  PRQ_TRY(buf.alloc(&dYref, static_cast<size_t>(outs)));
  PRQ_TRY(buf.alloc(&dY, static_cast<size_t>(outs)));
  PRQ_TRY(buf.alloc(&dInv, static_cast<size_t>(K)));
  PRQ_TRY(buf.alloc(&dPerm, static_cast<size_t>(K)));
  PRQ_TRY(buf.alloc(&dWq, static_cast<size_t>(N) * K_aug / 2));
  PRQ_TRY(buf.alloc(&dWsc, static_cast<size_t>(N) * K_aug / 32));
  PRQ_TRY(buf.alloc(&dAq, static_cast<size_t>(M) * K_aug / 2));
  PRQ_TRY(buf.alloc(&dAsc, static_cast<size_t>(M) * K_aug / 32));
  PRQ_TRY(buf.alloc(&dWp, code_bytes));
  PRQ_TRY(buf.alloc(&dWps, scale_bytes));
  PRQ_TRY(buf.alloc(&dWs, ws_bytes));
  PRQ_TRY(buf.alloc(&dPartial, static_cast<size_t>(2) * err_blocks));
  if (ws_bytes) PRQ_TRY(hip_status(hipMemsetAsync(dWs, 0, ws_bytes, stream)));
  PRQ_TRY(hip_status(hipMemcpyAsync(dW, W_bf16, static_cast<size_t>(N) * K * 2, hipMemcpyHostToDevice, stream)));
  PRQ_TRY(hip_status(hipMemcpyAsync(dX, X_bf16, static_cast<size_t>(M) * K * 2, hipMemcpyHostToDevice, stream)));
  reference_product_kernel<<<dim3((N + kRefTile - 1) / kRefTile, (M + kRefTile - 1) / kRefTile), 256, 0,
                             stream>>>(dX, dW, M, N, K, dYref);
  PRQ_TRY(hip_status(hipGetLastError()));

  std::vector<float> scale(K), inv(K), inv_pos(K);
  std::vector<int32_t> perm(K);
  std::vector<uint8_t> Wq(static_cast<size_t>(N) * K_aug / 2), Wsc(static_cast<size_t>(N) * K_aug / 32);
  std::vector<double> partial(static_cast<size_t>(2) * err_blocks);
  for (int a = 0; a < n_alpha; ++a) {
    PRQ_TRY(prq_prepare_ex(W_bf16, N, K, Xcal_bf16, T, alphas[a], k_tail, scale_mode, flags,
                           scale.data(), inv.data(), perm.data(), inv_pos.data(), Wq.data(), Wsc.data(),
                           nullptr));
    // The host buffers are reused by the next alpha: finish this one's copies first.
    PRQ_TRY(hip_status(hipMemcpyAsync(dWq, Wq.data(), Wq.size(), hipMemcpyHostToDevice, stream)));
    PRQ_TRY(hip_status(hipMemcpyAsync(dWsc, Wsc.data(), Wsc.size(), hipMemcpyHostToDevice, stream)));
    PRQ_TRY(hip_status(hipMemcpyAsync(dInv, inv_pos.data(), K * sizeof(float), hipMemcpyHostToDevice, stream)));
    PRQ_TRY(hip_status(hipMemcpyAsync(dPerm, perm.data(), K * sizeof(int32_t), hipMemcpyHostToDevice, stream)));
    PRQ_TRY(prq_pack_weight(dWq, dWsc, 1, N, static_cast<int32_t>(K_aug), dWp, dWps, stream));
    PRQ_TRY(prq_quant_act(dX, K, M, K, k_tail, dInv, dPerm, nullptr, 1, dAq, dAsc, stream));
    PRQ_TRY(prq_gemm(dAq, dAsc, M, dWp, dWps, N, static_cast<int32_t>(K_aug), dY, dWs, ws_bytes, stream));
    squared_error_kernel<<<err_blocks, kErrThreads, 0, stream>>>(dY, dYref, outs, per_block, dPartial);
    PRQ_TRY(hip_status(hipGetLastError()));
    PRQ_TRY(hip_status(hipMemcpyAsync(partial.data(), dPartial, partial.size() * sizeof(double),
                                      hipMemcpyDeviceToHost, stream)));
    PRQ_TRY(hip_status(hipStreamSynchronize(stream)));
    double e = 0.0, r = 0.0;
    for (int b = 0; b < err_blocks; ++b) {   // fixed order
      e += partial[2 * b];
      r += partial[2 * b + 1];
    }
    nrmse[a] = r > 0.0 ? std::sqrt(e / r) : (e > 0.0 ? INFINITY : 0.0);
  }
  return PRQ_OK;
}

}  // namespace
}  // namespace prq

extern "C" {

int prq_evaluate_nrmse(const uint16_t* W_bf16, int32_t N, int32_t K, const uint16_t* Xcal_bf16,
                       int32_t T, const uint16_t* X_bf16, int32_t M, double alpha, int32_t k_tail,
                       int32_t scale_mode, int32_t flags, double* nrmse, hipStream_t stream) {
  if (!W_bf16 || !Xcal_bf16 || !X_bf16 || !nrmse || N <= 0 || K <= 0 || T <= 0 || M <= 0)
    return PRQ_EINVAL;
  if (N % 16) return PRQ_EALIGN;
  if (K > 16384) return PRQ_EUNSUPPORTED;
  return prq::evaluate_alphas(W_bf16, N, K, Xcal_bf16, T, X_bf16, M, &alpha, 1, k_tail, scale_mode,
                              flags, nrmse, stream);
}

int prq_search_alpha(const uint16_t* W_bf16, int32_t N, int32_t K, const uint16_t* Xcal_bf16,
                     int32_t T, const double* alphas, int32_t n_alpha, int32_t k_tail,
                     int32_t scale_mode, int32_t flags, double* nrmse, int32_t* best,
                     hipStream_t stream) {
  if (!W_bf16 || !Xcal_bf16 || !alphas || !nrmse || !best || N <= 0 || K <= 0 || T <= 0 ||
      n_alpha <= 0)
    return PRQ_EINVAL;
  for (int a = 0; a < n_alpha; ++a)
    if (!(alphas[a] >= 0.0 && alphas[a] <= 1.0)) return PRQ_EINVAL;
  if (N % 16) return PRQ_EALIGN;
  if (K > 16384) return PRQ_EUNSUPPORTED;
  const int st = prq::evaluate_alphas(W_bf16, N, K, Xcal_bf16, T, Xcal_bf16, T, alphas, n_alpha,
                                      k_tail, scale_mode, flags, nrmse, stream);
  if (st != PRQ_OK) return st;
  int b = 0;
  for (int a = 1; a < n_alpha; ++a)
    if (nrmse[a] < nrmse[b]) b = a;
  *best = b;
  return PRQ_OK;
}

}  // extern "C"
