/*
 * prq.h -- PRQuant (Permutation Residual Quantization, arXiv 2609.22106)
 * MXFP4 + tail-residual hot path for AMD Instinct MI355X (gfx950).
 *
 * Plain C ABI of libprq.so.  Every array is row-major and contiguous unless a
 * leading dimension is given; sizes are in elements unless stated.  Notation
 * follows the paper: K (the paper's C) is the reduction dimension of the
 * down-projection, k = k_tail is the number of "hardest" input channels moved
 * to the contiguous tail, K_aug = K + k.  MXFP4 (the format the paper cites in
 * Sec. 1): blocks of 32 elements along K share one E8M0 scale byte
 * (value 2^(code-127)); elements are E2M1 nibbles (s<<3 | e<<1 | m,
 * magnitudes 0, .5, 1, 1.5, 2, 3, 4, 6), two per byte, element 2i in bits 0-3
 * and element 2i+1 in bits 4-7 of byte i.  Quantization rule: scale code =
 * clamp(floor(log2(amax)) - 2 + 127, 0, 254) (0 for an all-zero block);
 * elements divided by the scale, rounded to nearest E2M1 with ties to even
 * code, saturating at 6; sign from the input's sign bit.
 *
 * Requirements common to every call: K and k_tail are multiples of 32 and
 * 0 <= k_tail <= K.  Device pointers must be 16-byte aligned and every row
 * start (ld_x * 2 bytes, K_aug/2 bytes) a multiple of 16 bytes, i.e.
 * ld_x % 8 == 0 and K_aug % 32 == 0.  Device calls are asynchronous: they
 * validate their arguments on the host, enqueue kernels on `stream` and return;
 * they never allocate, never synchronize, and keep no mutable global state
 * (apart from a per-device cache of the device's properties filled on first
 * use).  They are safe to call from several host threads.  The caller owns
 * every buffer.
 */
#ifndef PRQ_H
#define PRQ_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PRQ_BLOCK 32
#define PRQ_ABI_VERSION 1

/* Status codes.  Negative values are errors; no kernel is enqueued when a call
 * returns an error detected on the host. */
enum {
  PRQ_OK = 0,
  PRQ_EINVAL = -1,       /* null pointer where data is needed, negative size,
                            alpha outside [0, 1], unknown mode or variant      */
  PRQ_EALIGN = -2,       /* K or k_tail not a multiple of 32, k_tail > K,
                            K_aug != K + k_tail, misaligned pointer or stride  */
  PRQ_EDEVICE = -3,      /* HIP reported an error (device query or launch)    */
  PRQ_EUNSUPPORTED = -4, /* current device is not gfx950, or a size is beyond
                            the limits stated below                             */
  PRQ_EWORKSPACE = -5    /* workspace missing or smaller than required         */
};

/* Scaling rule of prq_prepare (Sec. Method, "Offline scaling"; the scaling
 * step of Algorithm 1).  a_j = max_t |Xcal[t, j]|, b_j = max_n |W[n, j]|, both
 * clamped below at 1e-5; s_j computed in double with the C library pow and
 * rounded to float; inv_s_j = 1.0f / s_j in float. */
enum {
  PRQ_SCALE_SMOOTH = 0,   /* s_j = a_j^alpha / b_j^(1 - alpha) (default)      */
  PRQ_SCALE_ACT_ONLY = 1, /* s_j = a_j^alpha (the form printed in the paper)  */
  PRQ_SCALE_NONE = 2      /* s_j = 1 (no scaling: the "w/o AWQ" ablation)     */
};

/* GEMM kernel selection for the _ex calls. */
enum {
  PRQ_GEMM_AUTO = 0,   /* chosen from the shape                               */
  PRQ_GEMM_TILE = 1,   /* LDS-tiled block-scaled MFMA kernel (prefill shapes) */
  PRQ_GEMM_STREAM = 2, /* weight-streaming decode kernels: whole-K workgroups
                          (splits 0 or 1), split-K for a forced split count > 1 */
  PRQ_GEMM_STREAM_K = 3 /* stream-K decode kernel (up to 64 rows; never AUTO's
                          choice): equal contiguous ranges of the weight's
                          (16-feature tile, 128-element K step) units, one
                          workgroup per tile where the tiles fill at least half
                          of the CUs, else one per CU; a tile shared by several
                          workgroups is finished by the last to arrive, which
                          adds the partial tiles in a fixed order (bitwise
                          reproducible) and needs the workspace. */
};

/* Human-readable text of a status code (static storage). */
const char* prq_strerror(int status);

/* PRQ_ABI_VERSION of the library. */
int prq_abi_version(void);

/*
 * prq_prepare -- offline calibration and export for one alpha (Algorithm 1:
 * per-channel maxima, scaling D_alpha, top-k columns of W D_alpha by MXFP4
 * quantization error, permutation P_alpha to a contiguous tail, tail residual
 * R_W of Eq. 2, augmented weight Q([W~, R_W]) of Eq. 3).  Host memory only,
 * synchronous, deterministic; touches no GPU.
 *
 *   W_bf16     [N, K]  bf16 bit patterns of the down-projection weight
 *   Xcal_bf16  [T, K]  bf16 calibration activations (T >= 1)
 *   alpha      scaling strength in [0, 1]
 *   k_tail     number of tail channels (multiple of 32, <= K)
 *   scale_mode PRQ_SCALE_*
 * Outputs (caller-allocated host buffers):
 *   scale      [K] float   s_j
 *   inv_scale  [K] float   1/s_j (the activation side multiplies by it)
 *   perm       [K] int32   perm[p] = source channel of position p: channels
 *                          not selected in increasing order, then the k
 *                          selected ones in increasing order
 *   inv_scale_pos [K] float or NULL   inv_scale[perm[p]]: D^-1 at the
 *                          permuted positions, the form prq_quant_act takes
 *   Wq         [N, K_aug/2] uint8   packed E2M1 codes of [W~ | R_W]
 *   Wsc        [N, K_aug/32] uint8  E8M0 scale codes
 *   col_err    [K] double or NULL   per-channel squared MXFP4 error of
 *                          W D_alpha (original channel order), summed in
 *                          double over n in increasing order
 * Selection: the k largest col_err, ties to the smaller channel index.
 * Returns PRQ_OK, PRQ_EINVAL, PRQ_EALIGN; PRQ_EUNSUPPORTED if K > 65536.
 */
int prq_prepare(const uint16_t* W_bf16, int32_t N, int32_t K,
                const uint16_t* Xcal_bf16, int32_t T,
                double alpha, int32_t k_tail, int32_t scale_mode,
                float* scale, float* inv_scale, int32_t* perm, float* inv_scale_pos,
                uint8_t* Wq, uint8_t* Wsc, double* col_err);

/* Options of prq_prepare_ex. */
enum {
  PRQ_PREPARE_E8M0_SEARCH = 1  /* weight-side E8M0 block-scale search (below)  */
};

/*
 * prq_prepare_ex -- prq_prepare with options; flags = 0 is prq_prepare.
 *   PRQ_PREPARE_E8M0_SEARCH: the "E8M0-W" variant of Sec. Ablation Studies, a
 *   local search of the weight block scales.  The paper gives no rule; the one
 *   used here: every 32-element block of Q(W~) and of Q(R_W) takes the first of
 *   the E8M0 codes c0, c0 - 1, c0 + 1 (c0 the OCP code of the block, each
 *   clamped to [0, 254]) whose sum of squared errors sum_i (w_i - deq_i)^2 --
 *   accumulated in double, one element at a time in index order -- is smallest,
 *   so no block is worse than under plain Q(.).  R_W is taken against the
 *   searched Q(W~); col_err and the tail selection use plain Q(.) (Algorithm 1
 *   unchanged).  The activation side is not affected.
 * Returns as prq_prepare, and PRQ_EINVAL for unknown flag bits.
 */
int prq_prepare_ex(const uint16_t* W_bf16, int32_t N, int32_t K,
                   const uint16_t* Xcal_bf16, int32_t T,
                   double alpha, int32_t k_tail, int32_t scale_mode, int32_t flags,
                   float* scale, float* inv_scale, int32_t* perm, float* inv_scale_pos,
                   uint8_t* Wq, uint8_t* Wsc, double* col_err);

/*
 * prq_quant_act -- activation side of Eq. 3 with the online copy (Sec.
 * "Activation tail construction" and "Kernel design"; Algorithm 1, step 11):
 *   Z~[m, p] = X[m, perm[p]] * inv_scale_pos[p]     (float32 product,
 *              inv_scale_pos[p] = 1/s_{perm[p]} from prq_prepare)
 * quantized to MXFP4 once; the k/32 tail blocks are then written a second time,
 * codes and scale bytes, after the K/32 main blocks, which equals quantizing
 * [Z~, Z~[:, K-k:]].
 *
 *   X_bf16        device [M, ld_x] bf16 (K used columns), ld_x >= K, ld_x % 8 == 0
 *   inv_scale_pos device [G, K] float in position order, or NULL (no scaling)
 *   perm          device [G, K] int32, or NULL (identity: X is already permuted);
 *                 perm and inv_scale_pos must be 16-byte aligned
 *                 values must lie in [0, K) (an entry outside it reads channel 0)
 *   group_offsets device [G + 1] int32, or NULL when G == 1.  Rows
 *                 [off[g], off[g+1]) use expert g's perm and inv_scale
 *                 (MoE experts, each calibrated separately).  Offsets must be
 *                 non-decreasing with off[0] = 0 and off[G] = M.
 *   Aq            device [M, K_aug/2] uint8 output
 *   Asc           device [M, K_aug/32] uint8 output
 * Limits: K <= 16384, G <= 4096.  M == 0 is a no-op.
 */
int prq_quant_act(const void* X_bf16, int64_t ld_x, int32_t M, int32_t K, int32_t k_tail,
                  const float* inv_scale_pos, const int32_t* perm,
                  const int32_t* group_offsets, int32_t G,
                  uint8_t* Aq, uint8_t* Asc, hipStream_t stream);

/*
 * prq_packed_weight_bytes / prq_pack_weight -- the weight layout the GEMM
 * kernels read: an invertible byte permutation of prq_prepare's canonical
 * Wq [E][N][K_aug/2] / Wsc [E][N][K_aug/32], applied once per weight (offline).
 * With S = ceil(K_aug / 128) K steps of 128 elements and T = N / 16 tiles:
 *   Wp  [E][T][S][64][16] bytes: entry (e, t, s, l) holds the 16 code bytes of
 *       row 16 t + l % 16, K elements [128 s + 32 (l / 16), +32) -- exactly
 *       what lane l of the 16x16x128 block-scaled FP4 MFMA consumes -- and
 *       zero bytes past K_aug;
 *   Wps [E][T][ceil(S/4)][64] uint32: byte j of entry (e, t, q, l) is the
 *       E8M0 scale of row 16 t + l % 16, 32-block 4 (4 q + j) + l / 16 (127
 *       past K_aug).
 * One wave thus reads one contiguous kilobyte per MFMA operand.  Both calls
 * require N % 16 == 0 and K_aug % 32 == 0; prq_pack_weight runs on `stream`
 * (device pointers; Wq, Wp and Wps 16-byte aligned).
 */
int prq_packed_weight_bytes(int32_t E, int32_t N, int32_t K_aug, size_t* code_bytes,
                            size_t* scale_bytes);
int prq_pack_weight(const uint8_t* Wq, const uint8_t* Wsc, int32_t E, int32_t N, int32_t K_aug,
                    uint8_t* Wp, uint8_t* Wps, hipStream_t stream);

/*
 * prq_gemm -- the augmented MXFP4 GEMM of Eq. 3, one GEMM over K_aug = K + k:
 *   Y[m, n] = sum_b 2^(Asc[m,b]-127) 2^(Wsc[n,b]-127) sum_i e2m1(A[m,32b+i]) e2m1(W[n,32b+i])
 * accumulated in float32 (block-scaled MFMA), Y float32 [M, N] (ld = N).
 *
 *   Aq [M, K_aug/2], Asc [M, K_aug/32]: from prq_quant_act (row-major)
 *   Wp, Wps: the weight in the packed layout above (E = 1), from
 *            prq_pack_weight of prq_prepare's Wq / Wsc
 *   workspace: device buffer of at least prq_gemm_workspace_bytes(M, N, K_aug)
 *   bytes (may be NULL when that is 0), 16-byte aligned.  Every GEMM
 *   workspace (this call, prq_gemm_ex, prq_gemm_packed) starts with a 16 KiB
 *   state head: the stream-K kernel's uint32 arrival counters, one per
 *   16-feature tile, which must be zero before the buffer's first use
 *   (zero-fill it once) and which every call leaves zero; no kernel writes
 *   anything else there.  The scratch of the kernel that runs follows it and
 *   is rewritten before it is read: the stream-K kernel's partial tiles
 *   [workgroups][2][M][16] floats (only where its plan shares tiles between
 *   workgroups; none for the 9728 -> 2560 down_proj); for a forced split count of the
 *   split-K kernel partial sums [splits][M][N] added in a fixed order; for the
 *   LDS-tiled kernel's split along K, splits - 1 partial sums [M][N] (Y
 *   16-byte aligned).  One buffer may therefore serve calls of any shape in
 *   turn, as long as it is large enough for each; calls that share it must be
 *   ordered (same stream).  AUTO runs the whole-K decode kernel up to 64
 *   rows (no workspace) and the LDS-tiled kernel above; the stream-K kernel
 *   runs only when asked for (PRQ_GEMM_STREAM_K).  A call whose plan would
 *   use more workspace than it is given (or NULL) runs without it (the
 *   LDS-tiled kernel unsplit; same result up to float rounding).
 * Limits: N % 16 == 0, K_aug <= 65536.  M == 0 is a no-op.
 */
size_t prq_gemm_workspace_bytes(int32_t M, int32_t N, int32_t K_aug);
int prq_gemm(const uint8_t* Aq, const uint8_t* Asc, int32_t M,
             const uint8_t* Wp, const uint8_t* Wps, int32_t N, int32_t K_aug,
             float* Y, void* workspace, size_t workspace_bytes, hipStream_t stream);
/* As prq_gemm with an explicit kernel (PRQ_GEMM_*) and, for PRQ_GEMM_STREAM,
 * an explicit split count along K_aug (0 = chosen from the shape). */
size_t prq_gemm_workspace_bytes_ex(int32_t M, int32_t N, int32_t K_aug, int32_t variant,
                                   int32_t splits);
int prq_gemm_ex(const uint8_t* Aq, const uint8_t* Asc, int32_t M,
                const uint8_t* Wp, const uint8_t* Wps, int32_t N, int32_t K_aug,
                float* Y, void* workspace, size_t workspace_bytes,
                int32_t variant, int32_t splits, hipStream_t stream);

/*
 * prq_gemm_noalloc -- prq_gemm (AUTO) with no workspace argument and no
 * allocation, for callers that cannot allocate device memory: code under HIP
 * graph capture, serving loops that must not allocate, harnesses that forbid
 * it.  The workspace is a device array inside the library of
 * prq_gemm_noalloc_max_workspace_bytes() bytes (16 MiB), one per GPU the
 * library runs on, held until the process ends, in prq_gemm's workspace layout
 * (its zero-state head is zero when the library loads and every call leaves
 * it zero).  Every call on a GPU shares that GPU's array: calls that overlap
 * on one GPU (concurrent streams, or host threads without ordering) race and
 * give wrong results; calls ordered on one stream are safe.  Arguments,
 * errors and results as prq_gemm; additionally PRQ_EWORKSPACE when the call's
 * plan would need more than the array (prq_gemm_workspace_bytes(M, N, K_aug)
 * above the maximum; nothing is launched), PRQ_EDEVICE when the array's device
 * address cannot be taken (on the first call on a device).
 */
size_t prq_gemm_noalloc_max_workspace_bytes(void);
int prq_gemm_noalloc(const uint8_t* Aq, const uint8_t* Asc, int32_t M,
                     const uint8_t* Wp, const uint8_t* Wps, int32_t N, int32_t K_aug,
                     float* Y, hipStream_t stream);

/*
 * Packed activations (prefill): the activation side of Eq. 3 written by the
 * quantizer directly in the packed layout of the weights (prq_pack_weight's
 * layout with the M rows in the place of the N output features), so that the
 * LDS-tiled GEMM copies both operands in whole contiguous kilobytes.  With
 * S = ceil(K_aug / 128) and B = ceil(M / 16) row blocks:
 *   Ap  [B][S][64][16] bytes: entry (b, s, l) the 16 code bytes of row
 *       16 b + l % 16, K elements [128 s + 32 (l / 16), +32);
 *   Aps [B][ceil(S/4)][64] uint32: byte j of entry (b, q, l) the E8M0 scale of
 *       row 16 b + l % 16, 32-block 4 (4 q + j) + l / 16.
 * Rows past M and K positions past K_aug hold zero codes and scale byte 127.
 * The codes and scales are those of prq_quant_act, byte for byte.
 *
 * prq_packed_act_bytes -- sizes of Ap and Aps for M rows.  Returns PRQ_OK,
 *   PRQ_EINVAL, PRQ_EALIGN (K_aug % 32), PRQ_EUNSUPPORTED (K_aug > 65536).
 * prq_quant_act_packed -- prq_quant_act into Ap / Aps (device, 16-byte
 *   aligned, of the sizes above), with the same arguments: one perm and
 *   inv_scale_pos (G = 1), or G groups of sorted rows (group_offsets, and G
 *   rows of K in perm / inv_scale_pos).  Rows of different groups may share a
 *   16-row block.  Limits and errors as prq_quant_act.  M == 0 is a no-op.
 * prq_gemm_packed -- prq_gemm on a packed activation (the whole-K decode
 *   kernel up to 64 rows, which needs no workspace: from two to four 16-row
 *   blocks the operands loaded straight into registers, one or two tiles per
 *   wave; at one block the block's operand copied into LDS in whole
 *   kilobytes; the LDS-tiled kernel above):
 *   Y [M, N] float32 = Eq. 3 over K_aug; Ap / Aps from prq_quant_act_packed,
 *   Wp / Wps from prq_pack_weight (E = 1).  workspace: at least
 *   prq_gemm_packed_workspace_bytes(M, N, K_aug) bytes, 16-byte aligned, in
 *   prq_gemm's layout (the 16 KiB state head, which this call never writes,
 *   then the scratch), for the split along K that the planner picks when few
 *   output tiles would leave CUs idle (splits - 1 partial sums [M][N],
 *   rewritten before being read, added to Y in a fixed order by a second
 *   kernel); with less (or NULL) the call runs unsplit.  Calls sharing a
 *   workspace must be ordered.  Limits as prq_gemm.
 * prq_grouped_gemm_packed -- prq_grouped_gemm on a packed activation (rows
 *   sorted by expert, from prq_quant_act_packed with G = E and the same
 *   offsets).  An expert's row tiles start on its first 16-row block; rows of
 *   a neighbouring expert in a shared block are computed but not stored.
 *   Arguments, limits and errors as prq_grouped_gemm, no workspace; Aps must
 *   be 16-byte aligned (else PRQ_EALIGN).
 */
int prq_packed_act_bytes(int32_t M, int32_t K_aug, size_t* code_bytes, size_t* scale_bytes);
int prq_quant_act_packed(const void* X_bf16, int64_t ld_x, int32_t M, int32_t K, int32_t k_tail,
                         const float* inv_scale_pos, const int32_t* perm,
                         const int32_t* group_offsets, int32_t G,
                         uint8_t* Ap, uint8_t* Aps, hipStream_t stream);
size_t prq_gemm_packed_workspace_bytes(int32_t M, int32_t N, int32_t K_aug);
int prq_gemm_packed(const uint8_t* Ap, const uint8_t* Aps, int32_t M,
                    const uint8_t* Wp, const uint8_t* Wps, int32_t N, int32_t K_aug,
                    float* Y, void* workspace, size_t workspace_bytes, hipStream_t stream);
int prq_grouped_gemm_packed(const uint8_t* Ap, const uint8_t* Aps,
                            const int32_t* group_offsets, int32_t E, int32_t M_total,
                            const uint8_t* Wp, const uint8_t* Wps, int32_t N, int32_t K_aug,
                            float* Y, hipStream_t stream);

/*
 * prq_grouped_gemm -- Eq. 3 for E MoE experts in one launch (the paper applies
 * PRQuant to every expert down-projection).  Rows are sorted by expert; rows
 * [off[e], off[e+1]) multiply expert e's augmented weight.
 *
 *   Aq [M_total, K_aug/2], Asc [M_total, K_aug/32]
 *   group_offsets device [E + 1] int32 (non-decreasing, off[0] = 0,
 *                 off[E] = M_total), read on the device only; offsets outside
 *                 [0, M_total] are clamped into it
 *   Wp, Wps  the E experts' weights in the packed layout (prq_pack_weight with E)
 *   Y  [M_total, N] float32
 *   workspace: as for prq_gemm, sized by prq_grouped_gemm_workspace_bytes
 *   (currently 0: the grouped kernels do not split K).
 * Limits: N % 16 == 0, K_aug <= 65536, E <= 4096.
 */
size_t prq_grouped_gemm_workspace_bytes(int32_t M_total, int32_t E, int32_t N, int32_t K_aug);
int prq_grouped_gemm(const uint8_t* Aq, const uint8_t* Asc,
                     const int32_t* group_offsets, int32_t E, int32_t M_total,
                     const uint8_t* Wp, const uint8_t* Wps, int32_t N, int32_t K_aug,
                     float* Y, void* workspace, size_t workspace_bytes, hipStream_t stream);
int prq_grouped_gemm_ex(const uint8_t* Aq, const uint8_t* Asc,
                        const int32_t* group_offsets, int32_t E, int32_t M_total,
                        const uint8_t* Wp, const uint8_t* Wps, int32_t N, int32_t K_aug,
                        float* Y, void* workspace, size_t workspace_bytes,
                        int32_t variant, hipStream_t stream);

/*
 * prq_expand_producer -- offline copy (Sec. Method, "Activation tail
 * construction", and Eq. 1): fold D^-1 into the up-projection and P into the
 * up- and gate-projections, and duplicate their last k output channels, so
 * that the gated FFN emits [Z~, Z~_tail] (C + k channels) directly and the
 * down-projection's activation needs a plain MXFP4 quantizer only
 * (prq_quant_act with K = C + k, k_tail = 0, no perm, no scales).
 *   W_up_bf16, W_gate_bf16 [C, H]  bf16 bit patterns; row = output channel
 *                                  (the down-projection's input channel);
 *                                  W_gate_bf16 may be NULL (no gate)
 *   inv_scale [C], perm [C]        from prq_prepare (channel order / position)
 * Outputs (caller-allocated host buffers) [C + k, H]:
 *   W_up_aug[r]   = bf16_rne(W_up[perm[p]] * inv_scale[perm[p]]), p = r for
 *                   r < C, p = r - k for r >= C (the tail copies)
 *   W_gate_aug[r] = W_gate[perm[p]] (same p)
 * The scaled up-projection is rounded once to bf16 (nearest, ties to even).
 * Host memory only, synchronous.  Returns PRQ_OK or PRQ_EINVAL.
 */
int prq_expand_producer(const uint16_t* W_up_bf16, const uint16_t* W_gate_bf16,
                        int32_t C, int32_t H, const float* inv_scale, const int32_t* perm,
                        int32_t k_tail, uint16_t* W_up_aug, uint16_t* W_gate_aug);

/*
 * prq_swiglu_quant / prq_swiglu_quant_packed -- offline copy, producer side
 * (Sec. Method, "Activation tail construction"; Eq. 1 with sigma = SiLU): the
 * gated activation of the expanded producers quantized as it is formed.
 *   gate_bf16, up_bf16 [M, ld] device, bf16 bit patterns: the outputs of the
 *       up/gate projections expanded by prq_expand_producer (first K_aug =
 *       C + k columns used; row stride ld elements, ld % 8 == 0, 16-byte
 *       aligned), so that SiLU(gate) * up is [Z~, Z~_tail]
 *   Aq [M, K_aug/2], Asc [M, K_aug/32] (row-major, as prq_quant_act), or
 *   Ap / Aps in the packed activation layout below (16-byte aligned, sizes
 *   from prq_packed_act_bytes; rows past M and K positions past K_aug written
 *   as zero codes and scale byte 127)
 * Output: Q(SiLU(gate) * up), the product in float32 (never rounded to bf16),
 * SiLU(g) = g / (1 + e^-g) with e^x by a fixed float32 sequence -- x clamped
 * to [-104, 89], n = rint(x log2 e), r = (x - n ln2_hi) - n ln2_lo with ln 2
 * split into a 15-bit head and a tail, e^r by its degree-6 Taylor polynomial
 * in Horner form, scaled by 2^n -- one IEEE float32 operation per step, so
 * the codes do not depend on the device's exp.  Finite inputs whose product
 * is finite; the quantized value of a non-finite product is unspecified.
 * Device, asynchronous on `stream`, allocates nothing.  Returns PRQ_OK,
 * PRQ_EINVAL (null pointer, M < 0, ld < K_aug), PRQ_EALIGN (K_aug % 32,
 * alignment), PRQ_EUNSUPPORTED (K_aug > 65536), PRQ_EDEVICE.  M == 0 is a
 * no-op.
 */
int prq_swiglu_quant(const void* gate_bf16, const void* up_bf16, int64_t ld, int32_t M,
                     int32_t K_aug, uint8_t* Aq, uint8_t* Asc, hipStream_t stream);
int prq_swiglu_quant_packed(const void* gate_bf16, const void* up_bf16, int64_t ld, int32_t M,
                            int32_t K_aug, uint8_t* Ap, uint8_t* Aps, hipStream_t stream);

/*
 * prq_evaluate_nrmse -- offline: the normalized reconstruction error of one
 * configuration, ||Y_hat - X W^T||_F / ||X W^T||_F, where Y_hat is Eq. 3
 * evaluated on the rows X with the device path (prq_prepare_ex on the
 * calibration rows Xcal with alpha, k_tail, scale_mode and flags, then
 * prq_pack_weight, prq_quant_act, prq_gemm) and X W^T is computed on the device
 * from the bf16 inputs with float32 accumulation.
 *   W_bf16 [N, K], Xcal_bf16 [T, K], X_bf16 [M, K]: host arrays (bf16 bits)
 *   nrmse: host double
 * Allocates and frees its own device buffers, runs on `stream` and
 * synchronizes it before returning.  N % 16 == 0 and K <= 16384 (the device
 * kernels' limits) besides prq_prepare's conditions.
 */
int prq_evaluate_nrmse(const uint16_t* W_bf16, int32_t N, int32_t K,
                       const uint16_t* Xcal_bf16, int32_t T,
                       const uint16_t* X_bf16, int32_t M,
                       double alpha, int32_t k_tail, int32_t scale_mode, int32_t flags,
                       double* nrmse, hipStream_t stream);

/*
 * prq_search_alpha -- offline: the alpha search of Algorithm 1.  For every
 * candidate alphas[a] (in [0, 1]) the export is built as by prq_prepare_ex and
 * Eq. 3 is evaluated on the calibration rows themselves; nrmse[a] receives the
 * normalized reconstruction error (as in prq_evaluate_nrmse with X = Xcal) and
 * *best the index of the smallest (the first on equal errors).  Export the
 * chosen configuration with prq_prepare_ex(alphas[*best], ...).
 *   alphas [n_alpha] host doubles; nrmse [n_alpha] host doubles; best host int32.
 * Device buffers, stream and limits as for prq_evaluate_nrmse.
 */
int prq_search_alpha(const uint16_t* W_bf16, int32_t N, int32_t K,
                     const uint16_t* Xcal_bf16, int32_t T,
                     const double* alphas, int32_t n_alpha, int32_t k_tail,
                     int32_t scale_mode, int32_t flags,
                     double* nrmse, int32_t* best, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* PRQ_H */
