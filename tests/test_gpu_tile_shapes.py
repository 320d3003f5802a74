"""Every tile shape of the LDS-tiled GEMM (Eq. 3 over K + k), forced one at a
time through the library's tuning entry point, against the oracle's float64
GEMM: max |dY| <= 1e-3 max |Y|.  Covers both ways the kernel stages the
activation scales (one aligned dword per row and step when K + k is a multiple
of 128, single bytes otherwise), ragged M, N and K + k, row and feature tiles
cut by the operand edges, steps fewer than the pipeline's stages, and grouped
calls with empty experts."""
import ctypes

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import prquant as pq                               # noqa: E402
from paper_2609_22106_amd import inputs                        # noqa: E402
from tests.gpu_util import assert_gemm_close, dev, host, say   # noqa: E402

pytestmark = pytest.mark.gpu

SHAPE_IDS = (0, 1, 2, 3)   # 256x256, 256x128, 128x128, 256x320


def _lib():
    from paper_2609_22106_amd import build, prq  # noqa: F401  (prq loads torch first)
    lib = ctypes.CDLL(build.PROBE_LIB)
    P, I = ctypes.c_void_p, ctypes.c_int
    lib.prq_tune_gemm_tile.argtypes = [P, P, I, P, I, P, P, I, I, P, I, P]
    lib.prq_tune_gemm_tile.restype = I
    return lib


def _run(shape, Aq, Asc, Wq, Wsc, off=None, E=1):
    from paper_2609_22106_amd import prq
    M, N, K_aug = Aq.shape[0], Wq.shape[-2], Aq.shape[1] * 2
    A, As = dev(Aq), dev(Asc)
    W = prq.prq_pack_weight(dev(Wq), dev(Wsc))
    Y = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    offd = dev(off) if off is not None else None
    rc = _lib().prq_tune_gemm_tile(A.data_ptr(), As.data_ptr(), M,
                                   offd.data_ptr() if offd is not None else None, E,
                                   W.Wp.data_ptr(), W.Wps.data_ptr(), N, K_aug, Y.data_ptr(),
                                   shape, torch.cuda.current_stream().cuda_stream)
    assert rc == 0, rc
    torch.cuda.synchronize()
    return host(Y)


DENSE = [(300, 384, 1024),    # dword scales, ragged rows
         (513, 272, 1152),    # dword, ragged rows and features (272 = 17 tiles of 16)
         (40, 512, 9984),     # dword, the down_proj reduction length, one row tile
         (257, 272, 1088),    # byte scales (1088 = 8.5 steps of 128)
         (130, 144, 4192),    # byte, 32.75 steps
         (17, 48, 96),        # byte, one partial step (fewer steps than stages)
         (64, 256, 256)]      # dword, two steps


@pytest.mark.parametrize("M,N,K_aug", DENSE)
@pytest.mark.parametrize("shape", SHAPE_IDS)
def test_tile_shape_dense(shape, M, N, K_aug):
    rng = np.random.default_rng(M * 131 + N * 7 + K_aug + shape)
    Aq, Asc = inputs.random_mxfp4(rng, M, K_aug)
    Wq, Wsc = inputs.random_mxfp4(rng, N, K_aug)
    say("tile shape case:", shape, M, N, K_aug)
    assert_gemm_close(_run(shape, Aq, Asc, Wq, Wsc), pq.gemm(Aq, Asc, Wq, Wsc),
                      f"shape {shape} {M}x{N}x{K_aug}")


GROUPED = [([0, 300, 0, 5, 260], 272, 1024),   # dword
           ([3, 0, 17, 1, 0], 48, 1088),       # byte
           ([0, 0, 200], 128, 832)]            # byte, the expert reduction length


@pytest.mark.parametrize("counts,N,K_aug", GROUPED)
@pytest.mark.parametrize("shape", SHAPE_IDS)
def test_tile_shape_grouped(shape, counts, N, K_aug):
    rng = np.random.default_rng(sum(counts) * 17 + N + K_aug + shape)
    E, M = len(counts), sum(counts)
    off = inputs.routed_offsets(counts)
    Aq, Asc = inputs.random_mxfp4(rng, M, K_aug)
    Wq, Wsc = inputs.random_mxfp4(rng, (E, N), K_aug)
    say("tile shape grouped case:", shape, counts, N, K_aug)
    Y = _run(shape, Aq, Asc, Wq, Wsc, off=off, E=E)
    assert_gemm_close(Y, pq.grouped_gemm(Aq, Asc, off, Wq, Wsc),
                      f"grouped shape {shape} {counts} {N}x{K_aug}")


def _split_lib():
    from paper_2609_22106_amd import build, prq  # noqa: F401
    lib = ctypes.CDLL(build.PROBE_LIB)
    P, I = ctypes.c_void_p, ctypes.c_int
    lib.prq_tune_gemm_tile_split.argtypes = [P, P, I, P, P, I, I, P, I, I, I, P, ctypes.c_size_t,
                                             P]
    lib.prq_tune_gemm_tile_split.restype = I
    return lib


# (M, N, K_aug, splits): split ranges of unequal length, more splits than
# whole 4-step groups, a last range of one step, ragged rows and features.
SPLIT = [(300, 272, 1024, 3),      # 8 steps -> 3 + 3 + 2
         (513, 144, 9984, 8),      # 78 steps -> 10 x 7 + 8
         (40, 512, 4192, 4),       # 33 steps -> 9 + 9 + 9 + 6 (byte scales when row-major)
         (129, 64, 1152, 9),       # 9 steps -> one step each
         (64, 256, 640, 2)]        # 5 steps -> 3 + 2


@pytest.mark.parametrize("M,N,K_aug,splits", SPLIT)
@pytest.mark.parametrize("packed", [True, False])
@pytest.mark.parametrize("shape", SHAPE_IDS)
def test_tile_split_k(shape, packed, M, N, K_aug, splits):
    """The tile GEMM split along K (partial sums in the workspace, added to Y in
    a fixed order by the reduction): within the tolerance of the oracle, and
    bit-identical over two calls (deterministic)."""
    from paper_2609_22106_amd import prq
    from tests.packing import pack_rows
    rng = np.random.default_rng(M * 3 + N + K_aug + splits)
    Aq, Asc = inputs.random_mxfp4(rng, M, K_aug)
    Wq, Wsc = inputs.random_mxfp4(rng, N, K_aug)
    W = prq.prq_pack_weight(dev(Wq), dev(Wsc))
    A, As = (map(dev, pack_rows(Aq, Asc)) if packed else (dev(Aq), dev(Asc)))
    ws = torch.full((max(splits - 1, 1) * M * N,), float("nan"), dtype=torch.float32, device="cuda")
    outs = []
    for _ in range(2):
        Y = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
        say("tile split case:", shape, packed, M, N, K_aug, splits)
        rc = _split_lib().prq_tune_gemm_tile_split(
            A.data_ptr(), As.data_ptr(), M, W.Wp.data_ptr(), W.Wps.data_ptr(), N, K_aug,
            Y.data_ptr(), shape, splits, int(packed), ws.data_ptr(), ws.numel() * 4,
            torch.cuda.current_stream().cuda_stream)
        assert rc == 0, rc
        torch.cuda.synchronize()
        outs.append(host(Y))
    np.testing.assert_array_equal(outs[0], outs[1])
    assert_gemm_close(outs[0], pq.gemm(Aq, Asc, Wq, Wsc),
                      f"split shape {shape} packed {packed} {M}x{N}x{K_aug} / {splits}")
