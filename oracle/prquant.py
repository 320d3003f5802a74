"""PRQuant calibration/export and the augmented MXFP4 GEMM -- oracle.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).  Plain NumPy, float64
unless a step's precision is fixed below.  Each function cites the passage of
arXiv 2609.22106 it follows.  Readings of points the paper leaves open:

* scale formula (Sec. Method, "Offline scaling and channel reordering"): the
  paper prints s_j = (max_t |Z_tj|)^alpha ("act_only"); the SmoothQuant form
  s_j = max_t|Z_tj|^alpha / max_n|W_nj|^(1-alpha) ("smooth", the default here)
  and s = 1 ("none", the "w/o AWQ" ablation of Sec. 4.3) are also provided.
  Both maxima are clamped below at 1e-5.  s_j is computed in float64 with the
  scalar C-library pow and rounded once to float32; the inverse is the float32
  quotient 1/s_j.  The scaled weight is the float32 product W_nj * s_j and the
  transformed activation the float32 product X_mj * (1/s_j).
* column-wise MXFP4 error (Algorithm 1, selection step): Q is applied to the
  scaled weight in its ORIGINAL column order (selection precedes the
  permutation), the error of column j is sum_n (W_s - Q(W_s))_nj^2, each term
  exact in float64 and summed in float64 in increasing n.  The k columns with
  the largest error are selected, ties to the smaller index.
* permutation (Algorithm 1, permutation step): unselected channels in
  increasing order, then the selected channels in increasing order (the
  "contiguous tail"); perm[p] is the source channel of position p.
* residual (Eq. 2): R = W~_tail - Q(W~)_tail where Q(W~) quantizes the whole
  permuted weight; because the tail starts on a block boundary this equals
  Q(W~_tail).  The difference is exact in float32 (checked here).
* activation side of Eq. 3: quantize the concatenation [Z~, Z~_tail]; the
  kernel's quantize-once-then-copy (Sec. "Kernel design") must equal it.
* GEMM output: float64 here (exact up to the cross-block float64 sums).
"""
from __future__ import annotations

import math

import numpy as np

from .mxfp4 import BLOCK, mx_dequantize, mx_quantize, mx_quantize_searched, pack_codes, qdq

SCALE_MODES = ("smooth", "act_only", "none")
CLAMP_MIN = 1e-5


def bf16_bits_to_f32(u16):
    """bfloat16 bit patterns (uint16) -> float32 (exact: append 16 zero bits)."""
    u16 = np.asarray(u16, dtype=np.uint16)
    return (u16.astype(np.uint32) << 16).view(np.float32)


def _check_sizes(K, k_tail):
    if K <= 0 or K % BLOCK:
        raise ValueError("K must be a positive multiple of 32")
    if k_tail < 0 or k_tail % BLOCK or k_tail > K:
        raise ValueError("k_tail must be a multiple of 32 in [0, K]")


# --------------------------------------------------------------------------- #
# Algorithm 1, steps 1 and 3: per-channel maxima and the scaling D_alpha
# --------------------------------------------------------------------------- #
def channel_scales(W_bf16, Xcal_bf16, alpha, scale_mode="smooth"):
    """(s, inv_s) float32[K] for D_alpha = diag(s) (Sec. Method, Algorithm 1)."""
    if scale_mode not in SCALE_MODES:
        raise ValueError(f"scale_mode must be one of {SCALE_MODES}")
    if not (0.0 <= alpha <= 1.0):
        raise ValueError("alpha must lie in [0, 1]")
    W = bf16_bits_to_f32(W_bf16)
    X = bf16_bits_to_f32(Xcal_bf16)
    K = W.shape[1]
    a = np.maximum(np.abs(X).max(axis=0).astype(np.float64), CLAMP_MIN)
    b = np.maximum(np.abs(W).max(axis=0).astype(np.float64), CLAMP_MIN)
    s64 = np.empty(K, dtype=np.float64)
    for j in range(K):                      # scalar libm pow, one channel at a time
        if scale_mode == "smooth":
            s64[j] = math.pow(a[j], alpha) / math.pow(b[j], 1.0 - alpha)
        elif scale_mode == "act_only":
            s64[j] = math.pow(a[j], alpha)
        else:
            s64[j] = 1.0
    s = s64.astype(np.float32)
    inv = np.float32(1.0) / s               # float32 quotient, correctly rounded
    return s, inv.astype(np.float32)


# --------------------------------------------------------------------------- #
# Algorithm 1, steps 4-5: top-k columns by MXFP4 error, contiguous-tail perm
# --------------------------------------------------------------------------- #
def column_errors(W_s):
    """e_j = sum_n (W_s - Q(W_s))_nj^2 over the ORIGINAL column order."""
    E = W_s.astype(np.float64) - qdq(W_s)          # exact (see module notes)
    E2 = E * E                                      # exact: <= 48 significant bits
    acc = np.zeros(W_s.shape[1], dtype=np.float64)
    for n in range(E2.shape[0]):                    # sequential in n
        acc += E2[n]
    return acc


def select_topk(col_err, k_tail):
    """The k largest errors, ties to the smaller channel index; returned sorted."""
    K = col_err.shape[0]
    order = np.lexsort((np.arange(K), -col_err))   # primary -e, secondary j
    return np.sort(order[:k_tail]).astype(np.int32)


def tail_permutation(K, selected):
    """perm = [unselected ascending, selected ascending]; perm[p] = source channel."""
    mask = np.zeros(K, dtype=bool)
    mask[selected] = True
    head = np.flatnonzero(~mask)
    tail = np.flatnonzero(mask)
    return np.concatenate([head, tail]).astype(np.int32)


# --------------------------------------------------------------------------- #
# Algorithm 1 for one alpha: scaling, selection, permutation, Eq. 2, Eq. 3
# --------------------------------------------------------------------------- #
def prepare(W_bf16, Xcal_bf16, alpha, k_tail, scale_mode="smooth", scale_search=False):
    """Offline calibration/export for one alpha (Algorithm 1, steps 1, 3-7, 10).

    W_bf16: uint16 [N, K] (bf16 bits of W_down); Xcal_bf16: uint16 [T, K].
    Returns a dict with the exported artefacts (scale, inv_scale, perm, packed
    Wq [N, (K+k)/2], Wsc [N, (K+k)/32]) and the intermediates the tests check.
    scale_search: the E8M0-W variant of Sec. Ablation Studies -- Q(W~) and
    Q(R_W) with the local block-scale search (mx_quantize_searched); the
    residual is taken against the searched Q(W~); the column errors that pick
    the tail keep the plain Q(.) (Algorithm 1, step 4, unchanged).
    """
    W_bf16 = np.asarray(W_bf16, dtype=np.uint16)
    Xcal_bf16 = np.asarray(Xcal_bf16, dtype=np.uint16)
    N, K = W_bf16.shape
    _check_sizes(K, k_tail)
    if Xcal_bf16.ndim != 2 or Xcal_bf16.shape[1] != K or Xcal_bf16.shape[0] < 1:
        raise ValueError("calibration activations must be [T >= 1, K]")
    s, inv = channel_scales(W_bf16, Xcal_bf16, alpha, scale_mode)
    W = bf16_bits_to_f32(W_bf16)
    W_s = (W * s[None, :]).astype(np.float32)               # W D_alpha, float32 product
    err = column_errors(W_s)
    selected = select_topk(err, k_tail)
    perm = tail_permutation(K, selected)
    W_t = np.ascontiguousarray(W_s[:, perm])                # W D P (Eq. 1)
    quantize = mx_quantize_searched if scale_search else mx_quantize
    codes_t, scales_t = quantize(W_t)                       # Q(W~)
    deq_t = mx_dequantize(codes_t, scales_t)
    R64 = W_t[:, K - k_tail:].astype(np.float64) - deq_t[:, K - k_tail:]   # Eq. 2
    R = R64.astype(np.float32)
    if not np.array_equal(R.astype(np.float64), R64):
        raise AssertionError("tail residual is not exact in float32")
    codes_r, scales_r = quantize(R)                         # Q(R_W)
    codes_aug = np.concatenate([codes_t, codes_r], axis=1)  # Q([W~, R_W]) (Eq. 3)
    scales_aug = np.concatenate([scales_t, scales_r], axis=1)
    return {
        "scale": s, "inv_scale": inv, "perm": perm, "selected": selected,
        "col_err": err, "W_s": W_s, "W_tilde": W_t, "R": R,
        "codes": codes_aug, "Wq": pack_codes(codes_aug), "Wsc": scales_aug,
        "K": K, "k_tail": k_tail, "K_aug": K + k_tail,
    }


# --------------------------------------------------------------------------- #
# Activation side of Eq. 3 (online copy) -- Algorithm 1, step 11
# --------------------------------------------------------------------------- #
def transformed_activation(X_bf16, inv_scale=None, perm=None):
    """Z~ = X D^-1 P as float32: Z~[m, p] = X[m, perm[p]] * inv_s[perm[p]]."""
    X = bf16_bits_to_f32(X_bf16)
    K = X.shape[1]
    if perm is None:
        perm = np.arange(K)
    perm = np.asarray(perm)
    Z = X[:, perm]
    if inv_scale is not None:
        Z = (Z * np.asarray(inv_scale, dtype=np.float32)[perm][None, :]).astype(np.float32)
    return np.ascontiguousarray(Z, dtype=np.float32)


def quant_act(X_bf16, inv_scale, perm, k_tail):
    """Q([Z~, Z~_tail]) packed: (Aq uint8 [M, (K+k)/2], Asc uint8 [M, (K+k)/32])."""
    X_bf16 = np.asarray(X_bf16, dtype=np.uint16)
    K = X_bf16.shape[1]
    _check_sizes(K, k_tail)
    Z = transformed_activation(X_bf16, inv_scale, perm)
    Z_aug = np.concatenate([Z, Z[:, K - k_tail:]], axis=1)  # [Z~, Z~_tail]
    codes, scales = mx_quantize(Z_aug)
    return pack_codes(codes), scales


def quant_act_grouped(X_bf16, inv_scale, perm, group_offsets, k_tail):
    """Rows [off[g], off[g+1]) use expert g's perm_g and inv_s_g (MoE experts)."""
    X_bf16 = np.asarray(X_bf16, dtype=np.uint16)
    M, K = X_bf16.shape
    off = np.asarray(group_offsets, dtype=np.int64)
    K_aug = K + k_tail
    Aq = np.zeros((M, K_aug // 2), dtype=np.uint8)
    Asc = np.zeros((M, K_aug // BLOCK), dtype=np.uint8)
    for g in range(off.shape[0] - 1):
        r0, r1 = int(off[g]), int(off[g + 1])
        if r1 > r0:
            inv_g = None if inv_scale is None else np.asarray(inv_scale)[g]
            perm_g = None if perm is None else np.asarray(perm)[g]
            Aq[r0:r1], Asc[r0:r1] = quant_act(X_bf16[r0:r1], inv_g, perm_g, k_tail)
    return Aq, Asc


# --------------------------------------------------------------------------- #
# Eq. 3: the augmented GEMM over K + k, and its grouped (MoE) form
# --------------------------------------------------------------------------- #
def _deq_packed(q, sc):
    from .mxfp4 import unpack_codes
    return mx_dequantize(unpack_codes(q), sc)


def gemm(Aq, Asc, Wq, Wsc):
    """Y = deq(A_aug) deq(W_aug)^T in float64 ([M, N])."""
    A = _deq_packed(Aq, Asc)
    W = _deq_packed(Wq, Wsc)
    if A.shape[1] != W.shape[1]:
        raise ValueError("reduction lengths differ")
    return A @ W.T


def grouped_gemm(Aq, Asc, group_offsets, Wq, Wsc):
    """Rows of expert e multiply W_aug,e; rows are sorted by expert."""
    off = np.asarray(group_offsets, dtype=np.int64)
    M = Aq.shape[0]
    N = Wq.shape[1]
    Y = np.zeros((M, N), dtype=np.float64)
    for e in range(off.shape[0] - 1):
        r0, r1 = int(off[e]), int(off[e + 1])
        if r1 > r0:
            Y[r0:r1] = gemm(Aq[r0:r1], Asc[r0:r1], Wq[e], Wsc[e])
    return Y


# --------------------------------------------------------------------------- #
# Reference product, Eq. 1 without quantization, reconstruction error
# --------------------------------------------------------------------------- #
def reference_product(X_bf16, W_bf16):
    """X W^T in float64 from the bf16 inputs (the unquantized target)."""
    X = bf16_bits_to_f32(X_bf16).astype(np.float64)
    W = bf16_bits_to_f32(W_bf16).astype(np.float64)
    return X @ W.T


def unquantized_transform_product(X_bf16, W_bf16, s, perm):
    """(X D^-1 P)(W D P)^T in float64 with no quantization (Eq. 1)."""
    X = bf16_bits_to_f32(X_bf16).astype(np.float64)
    W = bf16_bits_to_f32(W_bf16).astype(np.float64)
    s = np.asarray(s, dtype=np.float64)
    Zt = (X / s[None, :])[:, perm]
    Wt = (W * s[None, :])[:, perm]
    return Zt @ Wt.T


def nrmse(Y_hat, Y_ref):
    """Normalized reconstruction error ||Y_hat - Y_ref||_F / ||Y_ref||_F."""
    Y_hat = np.asarray(Y_hat, dtype=np.float64)
    Y_ref = np.asarray(Y_ref, dtype=np.float64)
    return float(np.linalg.norm(Y_hat - Y_ref) / np.linalg.norm(Y_ref))


def prquant_forward(X_bf16, W_bf16, Xcal_bf16, alpha, k_tail, scale_mode="smooth",
                    scale_search=False):
    """Y_hat of Eq. 3 end to end: prepare, quantize the activation, GEMM."""
    art = prepare(W_bf16, Xcal_bf16, alpha, k_tail, scale_mode, scale_search)
    Aq, Asc = quant_act(X_bf16, art["inv_scale"], art["perm"], k_tail)
    return gemm(Aq, Asc, art["Wq"], art["Wsc"]), art


# --------------------------------------------------------------------------- #
# Algorithm 1, steps 2-9: the alpha search
# --------------------------------------------------------------------------- #
def search_alpha(W_bf16, Xcal_bf16, alphas, k_tail, scale_mode="smooth", scale_search=False):
    """For each candidate alpha build the export and evaluate Eq. 3 on the
    calibration rows; return (index of the smallest reconstruction error --
    the first on equal errors --, the errors).  The error is nrmse against the
    unquantized product of the bf16 inputs."""
    ref = reference_product(Xcal_bf16, W_bf16)
    errs = []
    for a in alphas:
        y, _ = prquant_forward(Xcal_bf16, W_bf16, Xcal_bf16, a, k_tail, scale_mode, scale_search)
        errs.append(nrmse(y, ref))
    best = min(range(len(errs)), key=lambda i: (errs[i], i))
    return best, np.array(errs)


# --------------------------------------------------------------------------- #
# Sec. Ablation Studies: the "w/o Perm" variant (numerics only)
# --------------------------------------------------------------------------- #
def prepare_no_perm(W_bf16, Xcal_bf16, alpha, k_tail, scale_mode="smooth"):
    """The selected channels stay in place: W_aug = [Q(W D) | Q(R_S)] with
    R_S = (W D)[:, S] - deq Q(W D)[:, S] (S ascending; Q(W D) in the original
    channel order), so the residual columns are gathered from scattered
    blocks.  Returns scale, inv_scale, selected and the unpacked codes / scales."""
    W_bf16 = np.asarray(W_bf16, dtype=np.uint16)
    N, K = W_bf16.shape
    _check_sizes(K, k_tail)
    s, inv = channel_scales(W_bf16, np.asarray(Xcal_bf16, dtype=np.uint16), alpha, scale_mode)
    W_s = (bf16_bits_to_f32(W_bf16) * s[None, :]).astype(np.float32)
    selected = select_topk(column_errors(W_s), k_tail)
    codes, scales = mx_quantize(W_s)
    deq = mx_dequantize(codes, scales)
    R = (W_s[:, selected].astype(np.float64) - deq[:, selected]).astype(np.float32)
    codes_r, scales_r = mx_quantize(R)
    return {"scale": s, "inv_scale": inv, "selected": selected,
            "codes": np.concatenate([codes, codes_r], axis=1),
            "Wsc": np.concatenate([scales, scales_r], axis=1)}


def no_perm_forward(X_bf16, W_bf16, Xcal_bf16, alpha, k_tail, scale_mode="smooth"):
    """Y_hat of the w/o Perm variant: A_aug = Q([Z, Z[:, S]]) with Z = X D^-1 in
    the original channel order, times the augmented weight."""
    art = prepare_no_perm(W_bf16, Xcal_bf16, alpha, k_tail, scale_mode)
    Z = transformed_activation(X_bf16, art["inv_scale"], None)
    Z_aug = np.concatenate([Z, Z[:, art["selected"]]], axis=1)
    a_codes, a_scales = mx_quantize(np.ascontiguousarray(Z_aug))
    A = mx_dequantize(a_codes, a_scales)
    Wd = mx_dequantize(art["codes"], art["Wsc"])
    return A @ Wd.T, art


ABLATION_VARIANTS = {   # name -> (scale_mode, uses k_tail, E8M0 search)
    "plain MXFP4": ("none", False, False),
    "PRQuant": ("smooth", True, False),
    "w/o AWQ": ("none", True, False),
    "w/o Res": ("smooth", False, False),
    "E8M0-W": ("smooth", True, True),
}


def ablation_grid(X_bf16, W_bf16, Xcal_bf16, alpha, k_tail):
    """y-NRMSE of every variant of Sec. Ablation Studies on the rows X."""
    ref = reference_product(X_bf16, W_bf16)
    out = {}
    for name, (mode, use_k, search) in ABLATION_VARIANTS.items():
        y, _ = prquant_forward(X_bf16, W_bf16, Xcal_bf16, alpha, k_tail if use_k else 0, mode, search)
        out[name] = nrmse(y, ref)
    y, _ = no_perm_forward(X_bf16, W_bf16, Xcal_bf16, alpha, k_tail)
    out["w/o Perm"] = nrmse(y, ref)
    return out


# --------------------------------------------------------------------------- #
# Offline copy (Sec. Method, "Activation tail construction"; Eq. 1)
# --------------------------------------------------------------------------- #
def bf16_round_bits(x):
    """float32 -> bf16 bit patterns, nearest with ties to even (finite input)."""
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = u + 0x7FFF + ((u >> 16) & 1)
    return (u >> 16).astype(np.uint16)


def expand_producer(W_up_bf16, W_gate_bf16, inv_scale, perm, k_tail):
    """D^-1 folded into the up-projection rows, P into the up- and
    gate-projection rows, the last k output channels duplicated: row r of the
    result is channel perm[p] with p = r (r < C) or r - k (r >= C); the scaled
    up-projection is rounded once to bf16.  Returns bf16 bit patterns."""
    C = len(perm)
    p = np.concatenate([np.arange(C), np.arange(C - k_tail, C)])
    src = np.asarray(perm)[p]
    up = bf16_bits_to_f32(np.asarray(W_up_bf16, dtype=np.uint16))[src]
    d = np.asarray(inv_scale, dtype=np.float32)[src][:, None]
    up_aug = bf16_round_bits((up * d).astype(np.float32))
    gate_aug = None if W_gate_bf16 is None else np.asarray(W_gate_bf16, dtype=np.uint16)[src]
    return up_aug, gate_aug


def gated_ffn(X_hidden_bf16, W_up_bf16, W_gate_bf16):
    """(X W_up^T) * silu(X W_gate^T) in float64 (the producer of the
    down-projection's input; Eq. 1 with sigma = SiLU)."""
    X = bf16_bits_to_f32(np.asarray(X_hidden_bf16, dtype=np.uint16)).astype(np.float64)
    up = X @ bf16_bits_to_f32(np.asarray(W_up_bf16, dtype=np.uint16)).astype(np.float64).T
    g = X @ bf16_bits_to_f32(np.asarray(W_gate_bf16, dtype=np.uint16)).astype(np.float64).T
    return up * (g / (1.0 + np.exp(-g)))


# --------------------------------------------------------------------------- #
# Offline copy, producer side: the gated activation quantized as it is formed
# (Sec. Method, "Activation tail construction", offline copy; Eq. 1 with
# sigma = SiLU).  The expanded up/gate projections (expand_producer) emit
# gate and up outputs C + k wide whose product is already [Z~, Z~_tail]; the
# down-projection's MXFP4 input is Q(SiLU(gate) * up) over those C + k
# columns.  Reading: gate and up are the producer GEMMs' bf16 outputs; the
# product is formed in float32 and quantized without rounding it to bf16; the
# paper fixes no precision for SiLU, so it is computed by the fixed float32
# sequence below, one IEEE float32 operation per step (no fused multiply-add),
# which a kernel can repeat bit for bit.
# --------------------------------------------------------------------------- #
# e^x = 2^n e^r with n = rint(x log2 e) and r = x - n ln 2 (|r| <= ln 2 / 2);
# ln 2 is split into a head with 15 significant bits (n * head exact for
# |n| <= 256) and a tail; e^r by its degree-6 Taylor polynomial (truncation
# below 2^-23 relative on |r| <= 0.35) in Horner form; x is first clamped to
# [-104, 89], where e^x is 0 or inf in float32 anyway.
EXP_LOG2E = np.float32(1.4426950408889634)
EXP_LN2_HI = np.float32(0.693145751953125)
EXP_LN2_LO = np.float32(1.4286067653301870e-06)
EXP_TAYLOR = tuple(np.float32(1.0 / math.factorial(i)) for i in range(6, -1, -1))   # c6 .. c0
EXP_X_MIN, EXP_X_MAX = np.float32(-104.0), np.float32(89.0)


def exp_f32(x):
    """e^x in float32 by the fixed sequence above (elementwise)."""
    x = np.minimum(np.maximum(np.asarray(x, dtype=np.float32), EXP_X_MIN), EXP_X_MAX)
    n = np.rint(x * EXP_LOG2E).astype(np.float32)
    r = ((x - n * EXP_LN2_HI).astype(np.float32) - n * EXP_LN2_LO).astype(np.float32)
    p = np.full_like(r, EXP_TAYLOR[0])
    for c in EXP_TAYLOR[1:]:
        p = ((p * r).astype(np.float32) + c).astype(np.float32)
    with np.errstate(over="ignore"):   # e^x past float32's range is inf, as intended
        return np.ldexp(p, n.astype(np.int32)).astype(np.float32)


def silu_f32(g):
    """SiLU(g) = g / (1 + e^-g) in float32 (one rounding per operation)."""
    g = np.asarray(g, dtype=np.float32)
    d = (np.float32(1.0) + exp_f32(-g)).astype(np.float32)
    return (g / d).astype(np.float32)


def swiglu_f32(gate_bf16, up_bf16):
    """SiLU(gate) * up in float32 from the producers' bf16 outputs."""
    g = bf16_bits_to_f32(np.asarray(gate_bf16, dtype=np.uint16))
    u = bf16_bits_to_f32(np.asarray(up_bf16, dtype=np.uint16))
    return (silu_f32(g) * u).astype(np.float32)


def swiglu_quant(gate_bf16, up_bf16):
    """Q(SiLU(gate) * up) packed: (Aq uint8 [M, K_aug/2], Asc uint8 [M, K_aug/32])
    for gate/up [M, K_aug] (K_aug = C + k from the expanded producers)."""
    codes, scales = mx_quantize(swiglu_f32(gate_bf16, up_bf16))
    return pack_codes(codes), scales
