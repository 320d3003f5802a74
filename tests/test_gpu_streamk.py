"""The stream-K decode GEMM (PRQ_GEMM_STREAM_K: Eq. 3 over K + k for up to 64
activation rows, one workgroup per CU, each an equal contiguous share of the
weight's (tile, K step) units, shared tiles finished by the last workgroup to
arrive) against the oracle's float64 GEMM, max |dY| <= 1e-3 max |Y|, every
element of Y written (it starts as NaN); bitwise reproducibility; the arrival
counters left at zero; grids planned for other CU counts."""
import ctypes

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import prquant as pq                                           # noqa: E402
from paper_2609_22106_amd import inputs                                    # noqa: E402
from tests.gpu_util import assert_gemm_close, dev, host, nan_output, say   # noqa: E402

pytestmark = pytest.mark.gpu


def _prq():
    from paper_2609_22106_amd import prq
    return prq


def _counters(ws, N):
    """The uint32 arrival counters in the workspace's state head."""
    return host(ws[:(N // 16) * 4]).view(np.uint32)


# (M, N, K_aug), the planner's grid: the down_proj shape at every decode M
# (and plain MXFP4's K_aug = 9728, the layer down_proj's 9952: one workgroup
# per tile), ragged rows, tiles fewer than (shared) and exactly as many as the
# CUs, short K, tiny shapes whose whole range fits one workgroup.
SHAPES = [(1, 2560, 9984), (8, 2560, 9984), (32, 2560, 9984), (64, 2560, 9984),
          (5, 2560, 9728), (17, 2560, 9952), (48, 2560, 9984), (33, 3072, 9984),
          (16, 4096, 2624), (64, 4096, 4192), (3, 2048, 832), (64, 2048, 832),
          (1, 16, 32), (64, 48, 96), (5, 1792, 9984), (64, 1760, 9952)]


@pytest.mark.parametrize("M,N,K_aug", SHAPES)
def test_streamk_random_operands(M, N, K_aug):
    prq = _prq()
    rng = np.random.default_rng(M * 7 + N + K_aug)
    Aq, Asc = inputs.random_mxfp4(rng, M, K_aug)
    Wq, Wsc = inputs.random_mxfp4(rng, N, K_aug)
    W = prq.prq_pack_weight(dev(Wq), dev(Wsc))
    need = prq.prq_gemm_workspace_bytes(M, N, K_aug, prq.GEMM_STREAM_K)
    ws = torch.zeros(max(need, 16), dtype=torch.uint8, device="cuda")
    Y = nan_output(M, N)
    say("stream-K case:", M, N, K_aug)
    prq.prq_gemm(dev(Aq), dev(Asc), W, Y=Y, workspace=ws, variant=prq.GEMM_STREAM_K)
    torch.cuda.synchronize()
    assert_gemm_close(host(Y), pq.gemm(Aq, Asc, Wq, Wsc), f"stream-K {M}x{N}x{K_aug}")
    assert not np.any(_counters(ws, N)), "arrival counters not reset"


def test_streamk_is_reproducible_and_reuses_its_workspace():
    """A plan whose tiles are shared (N = 1792: 112 tiles over one workgroup
    per CU): two calls give the same bits (the partial tiles are added in a fixed
    order whichever workgroup arrives last); the workspace left by them serves
    a call on fresh operands of another M, and, after a prefill call that
    splits along K on the same buffer, a decode call still finds zero arrival
    counters."""
    prq = _prq()
    rng = np.random.default_rng(11)
    N, K_aug = 1792, 9984
    Wq, Wsc = inputs.random_mxfp4(rng, N, K_aug)
    W = prq.prq_pack_weight(dev(Wq), dev(Wsc))
    need = prq.prq_gemm_workspace_bytes(64, N, K_aug, prq.GEMM_STREAM_K)
    assert need > 16384
    ws = torch.zeros(need, dtype=torch.uint8, device="cuda")
    Aq, Asc = inputs.random_mxfp4(rng, 64, K_aug)
    A, As = dev(Aq), dev(Asc)
    say("stream-K case: reproducibility")
    Y1 = host(prq.prq_gemm(A, As, W, workspace=ws, variant=prq.GEMM_STREAM_K))
    Y2 = host(prq.prq_gemm(A, As, W, workspace=ws, variant=prq.GEMM_STREAM_K))
    np.testing.assert_array_equal(Y1.view(np.uint32), Y2.view(np.uint32))
    assert_gemm_close(Y1, pq.gemm(Aq, Asc, Wq, Wsc), "stream-K M=64")
    Bq, Bsc = inputs.random_mxfp4(rng, 8, K_aug)
    Y3 = nan_output(8, N)
    prq.prq_gemm(dev(Bq), dev(Bsc), W, Y=Y3, workspace=ws, variant=prq.GEMM_STREAM_K)
    torch.cuda.synchronize()
    assert_gemm_close(host(Y3), pq.gemm(Bq, Bsc, Wq, Wsc), "stream-K M=8 after M=64")
    assert not np.any(_counters(ws, N))
    Cq, Csc = inputs.random_mxfp4(rng, 1024, K_aug)
    big_n = prq.prq_gemm_workspace_bytes(1024, N, K_aug)
    assert big_n > need, "the prefill call should split along K"
    big = torch.zeros(big_n, dtype=torch.uint8, device="cuda")
    big[:need] = ws
    prq.prq_gemm(dev(Cq), dev(Csc), W, workspace=big)
    Y4 = nan_output(8, N)
    prq.prq_gemm(dev(Bq), dev(Bsc), W, Y=Y4, workspace=big, variant=prq.GEMM_STREAM_K)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(Y4).view(np.uint32), host(Y3).view(np.uint32))
    assert not np.any(_counters(big, N))


def test_auto_runs_the_whole_k_decode_kernel():
    """prq_gemm (AUTO) runs the whole-K decode kernel at every M up to 64, with
    many output tiles (N = 2560: 160) or few (N = 1792: 112), and needs no
    workspace: the same bits as forcing it; the stream-K kernel runs only when
    asked for (it gives the same result within the GEMM bar)."""
    prq = _prq()
    rng = np.random.default_rng(12)
    K_aug = 9984
    for N, cases in ((2560, (1, 8, 9, 64)), (1792, (1, 8, 9))):
        Wq, Wsc = inputs.random_mxfp4(rng, N, K_aug)
        W = prq.prq_pack_weight(dev(Wq), dev(Wsc))
        for M in cases:
            Aq, Asc = inputs.random_mxfp4(rng, M, K_aug)
            A, As = dev(Aq), dev(Asc)
            assert prq.prq_gemm_workspace_bytes(M, N, K_aug) == 0
            say("decode case: auto, N =", N, "M =", M)
            Ya = host(prq.prq_gemm(A, As, W))
            Yf = host(prq.prq_gemm(A, As, W, variant=prq.GEMM_STREAM, splits=1))
            np.testing.assert_array_equal(Ya.view(np.uint32), Yf.view(np.uint32))
            assert_gemm_close(Ya, pq.gemm(Aq, Asc, Wq, Wsc), f"auto N={N} M={M}")
            if M <= 8:
                Ys = host(prq.prq_gemm(A, As, W, variant=prq.GEMM_STREAM_K))
                assert_gemm_close(Ys, pq.gemm(Aq, Asc, Wq, Wsc), f"stream-K N={N} M={M}")


def _tune(lib, A, As, M, W, N, K_aug, Y, cus, wgs, ws):
    return lib.prq_tune_gemm_streamk(A.data_ptr(), As.data_ptr(), M, W.Wp.data_ptr(),
                                     W.Wps.data_ptr(), N, K_aug, Y.data_ptr(), cus, wgs, ws.data_ptr(),
                                     ws.numel(), torch.cuda.current_stream().cuda_stream)


# (M, N, K_aug, CUs), one workgroup per CU forced: the down_proj shape with
# its tiles shared (one per CU instead of the planner's one per tile), one
# tile per workgroup exactly, odd workgroup counts, tiles shared by two to four
# workgroups, ten units per wave.
CU_CASES = [(1, 2560, 9984, 256), (8, 2560, 9984, 256), (64, 2560, 9984, 256),
            (17, 2560, 9984, 160), (17, 2560, 9984, 255), (64, 2560, 9728, 255),
            (2, 512, 4096, 80), (5, 512, 4096, 32), (40, 1024, 2624, 100),
            (64, 1024, 2624, 64), (33, 512, 4096, 48), (9, 2560, 9984, 200),
            (1, 2560, 9984, 241), (48, 256, 2624, 30)]


@pytest.mark.parametrize("M,N,K_aug,cus", CU_CASES)
def test_streamk_other_cu_counts(M, N, K_aug, cus):
    """The launch planned for other CU counts: ranges of exactly one tile,
    longer and shorter ranges, tiles shared by two to four workgroups."""
    prq = _prq()
    from paper_2609_22106_amd import build
    lib = ctypes.CDLL(build.PROBE_LIB)
    P, I, Z = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
    lib.prq_tune_gemm_streamk.argtypes = [P, P, I, P, P, I, I, P, I, I, P, Z, P]
    lib.prq_tune_gemm_streamk.restype = I
    lib.prq_tune_streamk_workspace_bytes.argtypes = [I, I, I, I, I]
    lib.prq_tune_streamk_workspace_bytes.restype = Z
    need = lib.prq_tune_streamk_workspace_bytes(M, N, K_aug, cus, cus)
    rng = np.random.default_rng(cus + M)
    Aq, Asc = inputs.random_mxfp4(rng, M, K_aug)
    Wq, Wsc = inputs.random_mxfp4(rng, N, K_aug)
    W = prq.prq_pack_weight(dev(Wq), dev(Wsc))
    ws = torch.zeros(max(need, 16), dtype=torch.uint8, device="cuda")
    Y = nan_output(M, N)
    say("stream-K case: cus", cus, M, N, K_aug)
    assert _tune(lib, dev(Aq), dev(Asc), M, W, N, K_aug, Y, cus, cus, ws) == 0
    torch.cuda.synchronize()
    assert_gemm_close(host(Y), pq.gemm(Aq, Asc, Wq, Wsc), f"stream-K cus={cus}")
    assert not np.any(_counters(ws, N)), "arrival counters not reset"
