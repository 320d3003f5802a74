// Internal declarations shared by the host ABI layer and the kernel launchers
// of libprq.so.  Not part of the public C ABI (include/prq.h).
#pragma once

#include <cstddef>
#include <cstdint>

#include <hip/hip_runtime_api.h>

namespace prq {

// Launch parameters of the weight-streaming GEMM, decided on the host from
// the shape.  Coverage invariant: (waves / tiles) * unroll * splits >= K steps,
// so every 128-element K step of every tile belongs to exactly one wave.
struct StreamConfig {
  int splits = 1;   // workgroups along K_aug per 16-feature output tile
  int waves = 16;   // waves per workgroup (4, 8 or 16)
  int unroll = 8;   // K steps per wave (1, 2, 3, 4, 6 or 8)
  int groups = 1;   // 16-row activation column groups per pass (1, 2 or 4)
  int tiles = 1;    // 16-feature tile groups per workgroup (1 or 4)
  int wave_tiles = 1;  // 16-feature tiles per wave (1, or 4 with one tile group)
  bool stage_lds = true;  // activation staged in LDS per workgroup (else per-wave loads)
  int reduce = 0;   // split-K: 0 atomic accumulator + last arriver, 1 partial sums +
                    // reduce kernel (deterministic), 2 atomics into Y zeroed first
  bool ok = true;   // false: no configuration covers K_aug (use the tile kernel)
};

// Launch parameters of the decode GEMM (gemm_decode.hip): a workgroup per
// 16-row group and `tiles` 16-feature tiles over the whole K range.
struct DecodeConfig {
  int tiles = 1;    // feature tiles per workgroup (1, 2 or 4)
  int row_splits = 1;  // workgroup rows the 16-row groups are dealt to (dense)
  int unroll = 5;   // K steps per wave (2, 5 or 10), >= ceil(steps / (16 / tiles))
  bool ok = true;   // false: K_aug needs more LDS or steps than the kernel takes
  bool direct = false;  // packed dense only: the register-direct variant
                        // (tiles = tiles per wave, 1 or 2; unroll 2 or 5)
};

// Launch parameters of the stream-K decode GEMM (gemm_streamk.hip): one
// workgroup per CU, each an equal contiguous range of the weight's
// (16-feature tile, 128-element K step) units.
struct StreamKConfig {
  int workgroups = 0;  // one per tile, or min(CUs, units)
  bool shared = false; // some tile is covered by several workgroups (needs the workspace)
  int groups = 1;      // 16-row activation groups (1..4)
  int unroll = 0;      // units per wave (1, 2, 4, 7 or 10), >= ceil(units per workgroup / 8)
  bool ok = false;     // false: M > 64, or a workgroup's range would exceed one tile
};

// act_quant.hip
hipError_t launch_act_quant(const uint16_t* X, int64_t ld_x, int M, int K, int k_tail,
                            const float* inv_scale, const int32_t* perm,
                            const int32_t* group_offsets, int G, uint8_t* Aq, uint8_t* Asc,
                            int num_cus, hipStream_t stream);
// kernel: 0 = by row count, 1 = the few-rows kernel, 2 = the many-rows kernel with
// register-staged rows, 3 = the many-rows kernel with rows copied into LDS stages.
hipError_t launch_act_quant_kernel(const uint16_t* X, int64_t ld_x, int M, int K, int k_tail,
                                   const float* inv_scale, const int32_t* perm,
                                   const int32_t* group_offsets, int G, uint8_t* Aq, uint8_t* Asc,
                                   int num_cus, int kernel, hipStream_t stream);

// The same with the output in the packed (weight) layout: Ap [ceil(M/16)][S][64][16],
// Aps [ceil(M/16)][ceil(S/4)][64] uint32, rows past M and K parts past K_aug padded
// (zero codes, scale byte 127).  Groups as in launch_act_quant (nullptr: one).
hipError_t launch_act_quant_packed(const uint16_t* X, int64_t ld_x, int M, int K, int k_tail,
                                   const float* inv_scale_pos, const int32_t* perm,
                                   const int32_t* group_offsets, int G, uint8_t* Ap, uint8_t* Aps,
                                   int num_cus, hipStream_t stream);
// kernel: 0 = automatic, 2 = register-staged rows, 3 = rows copied into LDS stages
// with the output through an 8-row LDS window wherever it fits (automatic: only
// where it pays), 4 = as 3 with the output stored directly.
// Q(SiLU(G) * U) of bf16 gate/up outputs [M, K_aug] (row stride ld elements,
// 16-byte aligned rows) into row-major Aq / Asc or, with `packed`, the packed
// activation layout (offline copy, producer side).
hipError_t launch_swiglu_quant(const uint16_t* G, const uint16_t* U, int64_t ld, int M, int K_aug,
                               uint8_t* Aq, uint8_t* Asc, bool packed, int num_cus,
                               hipStream_t stream);
hipError_t launch_act_quant_packed_kernel(const uint16_t* X, int64_t ld_x, int M, int K,
                                          int k_tail, const float* inv_scale_pos,
                                          const int32_t* perm, const int32_t* group_offsets,
                                          int G, uint8_t* Ap, uint8_t* Aps, int num_cus,
                                          int kernel, hipStream_t stream);

// pack.hip: the packed weight layout the GEMM kernels read.
size_t packed_code_bytes(int N, int K_aug, int E);
size_t packed_scale_bytes(int N, int K_aug, int E);
hipError_t launch_pack_weight(const uint8_t* Wq, const uint8_t* Wsc, int N, int K_aug, int E,
                              uint8_t* Wp, uint8_t* Wps, hipStream_t stream);

// gemm_tile.hip / gemm_stream.hip (packed weights Wp/Wps).  group_offsets ==
// nullptr means one group of M rows.
// Tile shapes: 0 = 256x256 (8 waves, two per SIMD), 1 = 256x128, 2 = 128x128 (4 waves),
// 3 = 256x320 (8 waves).
int choose_tile_shape(int M_rows, int N, int num_cus, bool packed);
hipError_t launch_gemm_tile(const uint8_t* Aq, const uint8_t* Asc, int M,
                            const int32_t* group_offsets, int E, const uint8_t* Wp,
                            const uint8_t* Wps, int N, int K_aug, float* Y, int shape,
                            hipStream_t stream);
// Dense tile GEMM over all columns with the planned shapes (one launch, or a
// main column region and the rest in another shape, each filling the CUs in
// whole rounds, or one shape split along K with a deterministic reduction when
// the workspace holds tile_workspace_bytes).
size_t tile_workspace_bytes(int M, int N, int K_aug, bool packed, int num_cus);
hipError_t launch_gemm_tile_planned(const uint8_t* Aq, const uint8_t* Asc, int M,
                                    const uint8_t* Wp, const uint8_t* Wps, int N, int K_aug,
                                    float* Y, bool packed, int num_cus, void* workspace,
                                    size_t workspace_bytes, hipStream_t stream);
// One shape, `splits` K ranges (ws: (splits - 1) * M * N floats, 16-byte
// aligned like Y); the tuning entry.
hipError_t launch_gemm_tile_split(const uint8_t* Aq, const uint8_t* Asc, int M, const uint8_t* Wp,
                                  const uint8_t* Wps, int N, int K_aug, float* Y, bool packed,
                                  int shape, int splits, float* ws, hipStream_t stream);
// The grouped (MoE) tile GEMM on a packed activation: an expert's row tiles
// start on 16-row block boundaries (rows of neighbouring experts are masked).
// shape 0-3: a workgroup per tile; kShapePersist: the persistent kernel
// (128 x 128 tiles, each XCD working through its own experts, pipelined across
// tiles; up to 512 experts) over num_cus CUs.
constexpr int kShapePersist = 4;
hipError_t launch_grouped_gemm_tile_packed(const uint8_t* Ap, const uint8_t* Aps, int M_total,
                                           const int32_t* group_offsets, int E, const uint8_t* Wp,
                                           const uint8_t* Wps, int N, int K_aug, float* Y,
                                           int shape, int num_cus, hipStream_t stream);
int choose_grouped_packed_shape(int rows_per_expert, int N, int K_aug, int E);
// The tile GEMM with the activation in the packed layout (dense).
hipError_t launch_gemm_tile_packed(const uint8_t* Ap, const uint8_t* Aps, int M,
                                   const uint8_t* Wp, const uint8_t* Wps, int N, int K_aug,
                                   float* Y, int shape, hipStream_t stream);
hipError_t launch_gemm_stream(const uint8_t* Aq, const uint8_t* Asc, int M,
                              const int32_t* group_offsets, int E, const uint8_t* Wp,
                              const uint8_t* Wps, int N, int K_aug, float* Y,
                              const StreamConfig& cfg, void* workspace, hipStream_t stream);

// Workspace of the split-K stream kernel: a float accumulator [M][N] plus one
// uint32 arrival counter per 16-feature output tile (per expert); zero between calls.
size_t stream_workspace_bytes(int M, int E, int N, int splits, int reduce);
StreamConfig choose_stream_config(int M_per_group, int N, int K_aug, int grouped, int num_cus);
bool stream_config_covers(const StreamConfig& c, int K_aug);
int choose_variant(int M_per_group, int N, int K_aug);
// Every GEMM workspace starts with a state head of kWorkspaceStateBytes: the
// stream-K kernel's uint32 arrival counters, one per 16-feature tile (up to
// kMaxStreamKTiles), zero before a workspace's first use and left zero by
// every call.  Nothing else is written there; the scratch of every kernel
// (partial tiles or sums, rewritten before they are read) follows it.
constexpr size_t kWorkspaceStateBytes = 16384;
constexpr int kMaxStreamKTiles = static_cast<int>(kWorkspaceStateBytes / 4);

// gemm_streamk.hip.  Workspace: the state head, then partial tiles
// [workgroups][2][M][16] floats.
// workgroups 0: one per CU, or one per tile where the tiles fill at least
// half of the CUs (no tile is then shared: no arrival protocol at all).
StreamKConfig choose_streamk_config(int M, int N, int K_aug, int num_cus, int workgroups = 0);
size_t streamk_workspace_bytes(int M, int N, int K_aug, int num_cus);
hipError_t launch_gemm_streamk(const uint8_t* Aq, const uint8_t* Asc, int M, const uint8_t* Wp,
                               const uint8_t* Wps, int N, int K_aug, float* Y,
                               const StreamKConfig& c, void* workspace, hipStream_t stream);
// gemm_decode.hip.  tiles / row_splits = 0 pick them from the rows.
size_t decode_lds_bytes(int K_aug, int tiles);
// packed: the activation is in the packed layout (may pick the direct variant).
DecodeConfig choose_decode_config(int M_per_group, int N, int K_aug, int grouped, int tiles,
                                  int row_splits, int num_cus, bool packed = false);
size_t decode_direct_lds_bytes(int M, int tiles, int row_splits);
// packed_a: Aq / Asc in the packed activation layout (dense calls only).
hipError_t launch_gemm_decode(const uint8_t* Aq, const uint8_t* Asc, int M,
                              const int32_t* group_offsets, int E, const uint8_t* Wp,
                              const uint8_t* Wps, int N, int K_aug, float* Y,
                              const DecodeConfig& cfg, hipStream_t stream, bool packed_a = false);

}  // namespace prq
