// Internal declarations shared by the host ABI layer and the kernel launchers
// of libprq.so.  Not part of the public C ABI (include/prq.h).
#pragma once

#include <cstddef>
#include <cstdint>

#include <hip/hip_runtime_api.h>

namespace prq {

// Launch parameters decided on the host from the shape.
struct StreamPlan {
  int splits;        // workgroups along K_aug per 16-row output tile
  int ksteps;        // 128-element K steps in K_aug (last one may be partial)
};

// act_quant.hip
hipError_t launch_act_quant(const uint16_t* X, int64_t ld_x, int M, int K, int k_tail,
                            const float* inv_scale, const int32_t* perm,
                            const int32_t* group_offsets, int G, uint8_t* Aq, uint8_t* Asc,
                            int num_cus, hipStream_t stream);

// gemm.hip.  group_offsets == nullptr means one group of M rows.
hipError_t launch_gemm_tile(const uint8_t* Aq, const uint8_t* Asc, int M,
                            const int32_t* group_offsets, int E, const uint8_t* Wq,
                            const uint8_t* Wsc, int N, int K_aug, float* Y, hipStream_t stream);
hipError_t launch_gemm_stream(const uint8_t* Aq, const uint8_t* Asc, int M,
                              const int32_t* group_offsets, int E, const uint8_t* Wq,
                              const uint8_t* Wsc, int N, int K_aug, float* Y, int splits,
                              void* workspace, hipStream_t stream);

// Workspace of the split-K stream kernel: float partials [splits][M][N] plus
// one uint32 arrival counter per 16-row output tile (and per expert).
size_t stream_workspace_bytes(int M, int E, int N, int splits);
int choose_stream_splits(int M, int N, int K_aug, int num_cus);
int choose_variant(int M_per_group, int N, int K_aug);

}  // namespace prq
