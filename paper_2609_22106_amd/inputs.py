"""Seeded synthetic workloads shaped like the paper's down-projections.

Random draws only: this module holds none of the method's arithmetic, and is
the one module that both the CPU oracle's tests and the HIP path's tests and
benchmark use.  The paper evaluates Qwen3-4B (dense down_proj, C = 9728 ->
2560) and Qwen3-30B-A3B (128 experts, top-8 routing, expert down_proj
C = 768 -> 2048) on a calibration set and five benchmarks (Sec. Experimental
Setup); none of those checkpoints or datasets is used.  Instead:

* weights W ~ 0.02 * N(0, 1);
* activations ~ N(0, 1) except a small set of outlier channels (shared by the
  calibration rows and the evaluation rows of one "model", as the paper's
  motivation describes) whose entries are scale * Student-t(3) (heavy tails)
  or scale * N(0, 1);
* bf16 by round-to-nearest-even from the float32 draws.

Draw order from ``numpy.random.default_rng(seed)``: outlier set, W,
calibration X, evaluation X (and for the MoE case, per expert: outlier set, W,
calibration X; then the routing; then the routed rows).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


def f32_to_bf16_bits(x):
    """float32 -> bfloat16 bits, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    return ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)


def bf16_bits_to_f32(u16):
    return (np.asarray(u16, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _activations(rng, rows, K, out_idx, out_scale, heavy_tail):
    x = rng.standard_normal((rows, K), dtype=np.float64)
    if len(out_idx):
        if heavy_tail:
            o = rng.standard_t(3, size=(rows, len(out_idx)))
        else:
            o = rng.standard_normal((rows, len(out_idx)))
        x[:, out_idx] = out_scale * o
    return f32_to_bf16_bits(x.astype(np.float32))


def _weights(rng, N, K):
    return f32_to_bf16_bits((0.02 * rng.standard_normal((N, K))).astype(np.float32))


@dataclass
class DenseCase:
    """One linear layer: W [N, K], calibration X [T, K], evaluation X [M, K]."""
    name: str
    N: int
    K: int
    k_tail: int
    alpha: float
    W: np.ndarray
    Xcal: np.ndarray
    X: np.ndarray
    outliers: np.ndarray
    M_list: tuple = ()


@dataclass
class MoECase:
    """E experts of W_e [N, K] with rows routed top-k and sorted by expert."""
    name: str
    E: int
    N: int
    K: int
    k_tail: int
    alpha: float
    W: np.ndarray            # [E, N, K] bf16 bits
    Xcal: np.ndarray         # [E, T, K] bf16 bits
    X: np.ndarray            # [M_total, K] bf16 bits, rows sorted by (expert, token)
    group_offsets: np.ndarray  # int32 [E + 1]
    token_of_row: np.ndarray   # int32 [M_total]
    outliers: list = field(default_factory=list)


def make_dense(name, N, K, M, T, k_tail, alpha=0.5, n_out=None, out_scale=30.0,
               heavy_tail=True, seed=0, M_list=()):
    """Dense down_proj-like layer; n_out defaults to round(0.5 % of K)."""
    rng = np.random.default_rng(seed)
    if n_out is None:
        n_out = int(round(0.005 * K))
    out_idx = np.sort(rng.choice(K, n_out, replace=False)) if n_out else np.zeros(0, np.int64)
    W = _weights(rng, N, K)
    Xcal = _activations(rng, T, K, out_idx, out_scale, heavy_tail)
    X = _activations(rng, M, K, out_idx, out_scale, heavy_tail)
    return DenseCase(name, N, K, k_tail, alpha, W, Xcal, X, out_idx, tuple(M_list) or (M,))


def tiny_case(seed=0):
    """16 x 1024 -> 512, k = 64, 8 outlier channels x40 (normal), 64 calibration rows."""
    return make_dense("tiny_16x1024x512_k64", N=512, K=1024, M=16, T=64, k_tail=64,
                      n_out=8, out_scale=40.0, heavy_tail=False, seed=seed)


def down_proj_decode(seed=0, M_max=64):
    """Qwen3-4B-shaped down_proj 9728 -> 2560, k = 256, decode rows."""
    return make_dense("qwen3_4b_down_decode", N=2560, K=9728, M=M_max, T=256, k_tail=256,
                      seed=seed, M_list=(1, 8, 32, 64))


def down_proj_prefill(seed=0, M_max=8192):
    """Qwen3-4B-shaped down_proj 9728 -> 2560, k = 256, prefill rows."""
    return make_dense("qwen3_4b_down_prefill", N=2560, K=9728, M=M_max, T=256, k_tail=256,
                      seed=seed, M_list=(512, 2048, 8192))


def tail_width(K):
    """k = K/40 rounded down to a multiple of 32 (the layer-set workload)."""
    return (K // 40) // 32 * 32


LAYER_SET = (  # name, N (out features), K (in features), hidden 2560
    ("q_proj", 4096, 2560), ("k_proj", 1024, 2560), ("v_proj", 1024, 2560),
    ("o_proj", 2560, 4096), ("gate_proj", 9728, 2560), ("up_proj", 9728, 2560),
    ("down_proj", 2560, 9728),
)


def layer_case(layer, M=4096, seed=0):
    """One linear of the Qwen3-4B-shaped decoder-layer set at prefill M."""
    for name, N, K in LAYER_SET:
        if name == layer:
            return make_dense(f"qwen3_4b_{name}", N=N, K=K, M=M, T=256, k_tail=tail_width(K),
                              seed=seed)
    raise KeyError(layer)


def make_moe(name, E, N, K, tokens, topk, T, k_tail, alpha=0.5, out_frac=0.005,
             out_scale=30.0, seed=0):
    """Grouped experts: per-expert W, calibration rows and outlier set; each
    token routed to ``topk`` distinct uniformly random experts, one independent
    K-wide row per (token, slot) drawn with that expert's outlier set."""
    rng = np.random.default_rng(seed)
    n_out = int(round(out_frac * K))
    W = np.empty((E, N, K), dtype=np.uint16)
    Xcal = np.empty((E, T, K), dtype=np.uint16)
    outs = []
    for e in range(E):
        o = np.sort(rng.choice(K, n_out, replace=False))
        outs.append(o)
        W[e] = _weights(rng, N, K)
        Xcal[e] = _activations(rng, T, K, o, out_scale, True)
    experts = np.stack([rng.choice(E, topk, replace=False) for _ in range(tokens)]) \
        if tokens else np.zeros((0, topk), np.int64)
    pairs = sorted((int(experts[t, j]), t) for t in range(tokens) for j in range(topk))
    M_total = len(pairs)
    token_of_row = np.array([t for _, t in pairs], dtype=np.int32)
    expert_of_row = np.array([e for e, _ in pairs], dtype=np.int64)
    counts = np.bincount(expert_of_row, minlength=E)
    offsets = routed_offsets(counts)
    x = rng.standard_normal((M_total, K))
    for e in range(E):
        r0, r1 = int(offsets[e]), int(offsets[e + 1])
        if r1 > r0 and n_out:
            x[r0:r1, outs[e]] = out_scale * rng.standard_t(3, size=(r1 - r0, n_out))
    X = f32_to_bf16_bits(x.astype(np.float32))
    return MoECase(name, E, N, K, k_tail, alpha, W, Xcal, X, offsets, token_of_row, outs)


def moe_experts(tokens, seed=0, E=128):
    """Qwen3-30B-A3B-shaped expert down_proj 768 -> 2048, k = 64, top-8 routing."""
    return make_moe(f"qwen3_30b_a3b_experts_{tokens}tok", E=E, N=2048, K=768, tokens=tokens,
                    topk=8, T=256, k_tail=64, seed=seed)


def routed_offsets(counts):
    """group_offsets int32 [E + 1] from per-expert row counts."""
    off = np.zeros(len(counts) + 1, dtype=np.int32)
    off[1:] = np.cumsum(counts)
    return off


def random_mxfp4(rng, shape_rows, K_aug, scale_lo=118, scale_hi=136):
    """Random packed MXFP4 operand: uniform code bytes and E8M0 scale bytes in
    [scale_lo, scale_hi] (any such pair is a valid GEMM input)."""
    rows = tuple(np.atleast_1d(shape_rows).tolist())
    q = rng.integers(0, 256, rows + (K_aug // 2,), dtype=np.uint8)
    s = rng.integers(scale_lo, scale_hi + 1, rows + (K_aug // 32,), dtype=np.uint8)
    return q, s


@dataclass
class FFNCase:
    """A gated FFN (the down-projection's producer) with random weights."""
    name: str
    H: int            # hidden size
    C: int            # intermediate size = the down-projection's K
    W_up: np.ndarray  # bf16 [C, H]
    W_gate: np.ndarray
    W_down: np.ndarray   # bf16 [H, C]
    X_hidden: np.ndarray  # bf16 [M, H]
    X_cal: np.ndarray     # bf16 [T, H]
    out_idx: np.ndarray   # intermediate channels with 30x up-projection rows


def make_ffn(name, H, C, M, T, n_out=8, out_scale=30.0, seed=0):
    """W_up, W_gate, W_down ~ 0.02 N(0,1); n_out up-projection rows scaled by
    out_scale (outlier intermediate channels); hidden states ~ N(0,1)."""
    rng = np.random.default_rng(seed)
    out_idx = np.sort(rng.choice(C, n_out, replace=False))
    W_up = 0.02 * rng.standard_normal((C, H))
    W_up[out_idx] *= out_scale
    W_gate = 0.02 * rng.standard_normal((C, H))
    W_down = 0.02 * rng.standard_normal((H, C))
    Xc = rng.standard_normal((T, H))
    X = rng.standard_normal((M, H))
    b = lambda a: f32_to_bf16_bits(a.astype(np.float32))
    return FFNCase(name, H, C, b(W_up), b(W_gate), b(W_down), b(X), b(Xc), out_idx)
