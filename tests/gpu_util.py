"""Helpers shared by the GPU tests: host<->device copies and the tolerance
of the GEMM parity checks."""
import sys

import numpy as np
import torch

# GEMM bar: float32 accumulation on the GPU against the float64 oracle,
# max |dY| <= 1e-3 * max |Y_oracle|.
GEMM_RTOL_OF_MAX = 1e-3


def dev(a):
    """numpy -> device tensor with the same bytes (uint16 travels as int16)."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    elif a.dtype == np.uint32:
        a = a.view(np.int32)
    return torch.from_numpy(a).cuda()


def host(t, dtype=None):
    a = t.detach().cpu().numpy()
    return a.view(dtype) if dtype is not None else a


def say(*msg):
    print(*msg, file=sys.stderr, flush=True)


def assert_gemm_close(Y_gpu, Y_ref, what=""):
    Y_gpu = np.asarray(Y_gpu, dtype=np.float64)
    Y_ref = np.asarray(Y_ref, dtype=np.float64)
    assert Y_gpu.shape == Y_ref.shape, (Y_gpu.shape, Y_ref.shape)
    assert np.all(np.isfinite(Y_gpu)), what
    scale = np.max(np.abs(Y_ref)) if Y_ref.size else 0.0
    err = np.max(np.abs(Y_gpu - Y_ref)) if Y_ref.size else 0.0
    assert err <= GEMM_RTOL_OF_MAX * scale, f"{what}: max|dY| = {err:.3e}, max|Y| = {scale:.3e}"
    return err / scale if scale else 0.0


def nan_output(M, N):
    """A float32 [M, N] device output filled with NaN, so that an element the
    kernel never writes fails the finiteness check."""
    return torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")


def rows_per_block(M, rng, block=16):
    """One random row of every `block`-row block of [0, M) plus the first and
    the last row: every row tile of every tile shape (whose heights are
    multiples of 16) holds at least one checked row."""
    starts = np.arange(0, M, block)
    picks = starts + rng.integers(0, block, starts.size)
    return np.unique(np.concatenate([np.minimum(picks, M - 1), [0, M - 1]]))


def tail_permutation(rng, K, k, swaps=0):
    """A permutation of the form Algorithm 1 exports: K - k channels in
    increasing order, then k randomly chosen channels in increasing order
    (the head then reads runs of consecutive channels at every alignment);
    `swaps` random transpositions inside the head break some runs."""
    sel = np.sort(rng.choice(K, k, replace=False))
    head = np.setdiff1d(np.arange(K), sel)
    perm = np.concatenate([head, sel]).astype(np.int32)
    for _ in range(swaps):
        i, j = rng.integers(0, K - k, 2)
        perm[i], perm[j] = perm[j], perm[i]
    return perm
