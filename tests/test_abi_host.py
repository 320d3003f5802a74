"""The C ABI on the host (no GPU): symbols, status strings, argument checks, and
the native prq_prepare bit-exact against the oracle (Algorithm 1, Eqs. 1-3)."""
import ctypes

import numpy as np
import pytest

from oracle import prquant as pq
from paper_2609_22106_amd import inputs, prq


def test_library_exports_every_declared_symbol():
    names = prq.exported_symbols()
    assert {"prq_prepare", "prq_quant_act", "prq_gemm", "prq_grouped_gemm"} <= set(names)
    lib = ctypes.CDLL(prq._build.LIB)
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing
    assert prq.prq_abi_version() == 1


def test_strerror():
    for st in (0, -1, -2, -3, -4, -5):
        assert prq.prq_strerror(st)
    assert prq.prq_strerror(-99) == "unknown status"


def _assert_prepare_equal(ours, ref):
    np.testing.assert_array_equal(ours["scale"], ref["scale"])
    np.testing.assert_array_equal(ours["inv_scale"], ref["inv_scale"])
    np.testing.assert_array_equal(ours["perm"], ref["perm"])
    np.testing.assert_array_equal(ours["inv_scale_pos"], ref["inv_scale"][ref["perm"]])
    np.testing.assert_array_equal(ours["Wsc"], ref["Wsc"])
    np.testing.assert_array_equal(ours["Wq"], ref["Wq"])
    if "col_err" in ours:
        np.testing.assert_array_equal(ours["col_err"], ref["col_err"])


@pytest.mark.parametrize("mode", ["smooth", "act_only", "none"])
@pytest.mark.parametrize("k", [0, 64, 256])
def test_prepare_matches_oracle_small(mode, k):
    c = inputs.make_dense("s", N=96, K=256, M=4, T=48, k_tail=k, n_out=5, seed=11)
    ours = prq.prq_prepare(c.W, c.Xcal, 0.5, k, mode, with_col_err=True)
    ref = pq.prepare(c.W, c.Xcal, 0.5, k, mode)
    _assert_prepare_equal(ours, ref)


@pytest.mark.parametrize("alpha", [0.0, 0.3, 0.85, 1.0])
def test_prepare_matches_oracle_alphas(alpha):
    c = inputs.tiny_case()
    ours = prq.prq_prepare(c.W, c.Xcal, alpha, 64, with_col_err=True)
    _assert_prepare_equal(ours, pq.prepare(c.W, c.Xcal, alpha, 64))


def test_prepare_matches_oracle_tiny_workload():
    c = inputs.tiny_case()
    _assert_prepare_equal(prq.prq_prepare(c.W, c.Xcal, 0.5, 64, with_col_err=True),
                          pq.prepare(c.W, c.Xcal, 0.5, 64))


def test_prepare_ties_and_degenerate_columns():
    """Zero columns, identical columns (tied errors) and a zero calibration channel."""
    rng = np.random.default_rng(5)
    W = (0.02 * rng.standard_normal((32, 128))).astype(np.float32)
    W[:, 7] = 0
    W[:, 20] = W[:, 90]
    W[:, 21] = W[:, 90]
    W[:, 5] *= 50
    X = rng.standard_normal((8, 128)).astype(np.float32)
    X[:, 9] = 0
    Wb, Xb = inputs.f32_to_bf16_bits(W), inputs.f32_to_bf16_bits(X)
    _assert_prepare_equal(prq.prq_prepare(Wb, Xb, 0.5, 32, with_col_err=True),
                          pq.prepare(Wb, Xb, 0.5, 32))


def test_prepare_matches_oracle_moe_expert_shape():
    """Three experts of the 768 -> 2048 expert down_proj shape, k = 64."""
    c = inputs.make_moe("m", E=3, N=2048, K=768, tokens=4, topk=2, T=256, k_tail=64, seed=2)
    for e in range(3):
        _assert_prepare_equal(prq.prq_prepare(c.W[e], c.Xcal[e], 0.5, 64, with_col_err=True),
                              pq.prepare(c.W[e], c.Xcal[e], 0.5, 64))


@pytest.mark.slow
def test_prepare_matches_oracle_down_proj_full():
    """Full 9728 -> 2560 down_proj, k = 256 (about 20 s in the oracle)."""
    c = inputs.down_proj_decode(M_max=1)
    _assert_prepare_equal(prq.prq_prepare(c.W, c.Xcal, 0.5, 256, with_col_err=True),
                          pq.prepare(c.W, c.Xcal, 0.5, 256))


@pytest.mark.parametrize("mode", ["smooth", "none"])
@pytest.mark.parametrize("k", [0, 64])
def test_prepare_e8m0_search_matches_oracle(mode, k):
    """prq_prepare_ex with the weight-side E8M0 search, bit for bit."""
    c = inputs.make_dense("s", N=96, K=256, M=4, T=48, k_tail=k, n_out=5, seed=12)
    ours = prq.prq_prepare(c.W, c.Xcal, 0.5, k, mode, with_col_err=True, scale_search=True)
    _assert_prepare_equal(ours, pq.prepare(c.W, c.Xcal, 0.5, k, mode, scale_search=True))


def test_prepare_e8m0_search_matches_oracle_workloads():
    c = inputs.tiny_case()
    _assert_prepare_equal(prq.prq_prepare(c.W, c.Xcal, 0.5, 64, scale_search=True),
                          pq.prepare(c.W, c.Xcal, 0.5, 64, scale_search=True))
    m = inputs.make_moe("m", E=1, N=2048, K=768, tokens=4, topk=1, T=256, k_tail=64, seed=3)
    _assert_prepare_equal(prq.prq_prepare(m.W[0], m.Xcal[0], 0.5, 64, scale_search=True),
                          pq.prepare(m.W[0], m.Xcal[0], 0.5, 64, scale_search=True))


def test_prepare_ex_rejects_unknown_flags():
    c = inputs.make_dense("s", N=16, K=64, M=1, T=4, k_tail=32, n_out=1)
    K = 64
    bufs = [np.empty(K, np.float32), np.empty(K, np.float32), np.empty(K, np.int32),
            np.empty(K, np.float32), np.empty((16, 48), np.uint8), np.empty((16, 3), np.uint8)]
    st = prq._prepare_ex(c.W.ctypes.data, 16, K, c.Xcal.ctypes.data, 4, 0.5, 32, 0, 2,
                         *[b.ctypes.data for b in bufs], None)
    assert st == prq.PRQ_EINVAL


def test_prepare_rejects_bad_arguments():
    c = inputs.make_dense("s", N=16, K=64, M=1, T=4, k_tail=32, n_out=1)
    with pytest.raises(prq.PRQError) as ei:
        prq.prq_prepare(c.W, c.Xcal, 0.5, 48)
    assert ei.value.status == prq.PRQ_EALIGN
    with pytest.raises(prq.PRQError) as ei:
        prq.prq_prepare(c.W, c.Xcal, 0.5, 96)              # k > K
    assert ei.value.status == prq.PRQ_EALIGN
    with pytest.raises(prq.PRQError) as ei:
        prq.prq_prepare(c.W, c.Xcal, 1.5, 32)
    assert ei.value.status == prq.PRQ_EINVAL
    with pytest.raises(prq.PRQError) as ei:
        prq.prq_prepare(c.W[:, :48], c.Xcal[:, :48], 0.5, 32)  # K % 32
    assert ei.value.status == prq.PRQ_EALIGN
    st = prq._prepare(None, 16, 64, None, 4, 0.5, 32, 0, None, None, None, None, None, None, None)
    assert st == prq.PRQ_EINVAL


def test_device_calls_validate_before_touching_the_gpu():
    """Errors the host detects are returned before any HIP call, so they are
    checkable without a GPU; M == 0 is a no-op."""
    fake = ctypes.c_void_p(4096)   # never dereferenced: every call below fails validation
    s = ctypes.c_void_p(0)
    assert prq._quant_act(fake, 1024, 4, 1000, 64, None, None, None, 1, fake, fake, s) == prq.PRQ_EALIGN
    assert prq._quant_act(fake, 1024, 4, 1024, 48, None, None, None, 1, fake, fake, s) == prq.PRQ_EALIGN
    assert prq._quant_act(fake, 1024, 4, 1024, 2048, None, None, None, 1, fake, fake, s) == prq.PRQ_EALIGN
    assert prq._quant_act(fake, 1000, 4, 1024, 64, None, None, None, 1, fake, fake, s) == prq.PRQ_EINVAL
    assert prq._quant_act(fake, 1024, 4, 1024, 64, None, None, None, 2, fake, fake, s) == prq.PRQ_EINVAL
    assert prq._quant_act(fake, 1024, -1, 1024, 64, None, None, None, 1, fake, fake, s) == prq.PRQ_EINVAL
    assert prq._quant_act(fake, 1024 * 32, 4, 32768, 64, None, None, None, 1, fake, fake, s) == prq.PRQ_EUNSUPPORTED
    assert prq._quant_act(None, 1024, 0, 1024, 64, None, None, None, 1, None, None, s) == prq.PRQ_OK
    assert prq._gemm(fake, fake, 4, fake, fake, 24, 1088, fake, None, 0, s) == prq.PRQ_EALIGN   # N % 16
    assert prq._gemm(fake, fake, 4, fake, fake, 32, 1080, fake, None, 0, s) == prq.PRQ_EALIGN   # K_aug % 32
    assert prq._gemm(fake, fake, 4, None, fake, 32, 1088, fake, None, 0, s) == prq.PRQ_EINVAL
    assert prq._gemm(None, None, 0, fake, fake, 32, 1088, None, None, 0, s) == prq.PRQ_OK
    assert prq._gemm_ex(fake, fake, 4, fake, fake, 32, 1088, fake, None, 0, 7, 0, s) == prq.PRQ_EINVAL
    assert prq._ggemm(fake, fake, None, 4, 8, fake, fake, 32, 1088, fake, None, 0, s) == prq.PRQ_EINVAL
    assert prq._ggemm(None, None, fake, 4, 0, fake, fake, 32, 1088, None, None, 0, s) == prq.PRQ_OK


def test_packed_activation_calls_validate_before_touching_the_gpu():
    fake = ctypes.c_void_p(4096)   # 16-byte aligned, never dereferenced
    odd = ctypes.c_void_p(4100)    # 4-byte aligned only
    s = ctypes.c_void_p(0)
    assert prq._quant_act_packed(fake, 1024, 4, 1000, 64, None, None, None, 1, fake, fake, s) == prq.PRQ_EALIGN
    assert prq._quant_act_packed(fake, 1024, 4, 1024, 2048, None, None, None, 1, fake, fake, s) == prq.PRQ_EALIGN
    assert prq._quant_act_packed(fake, 1024, 4, 1024, 64, None, None, None, 1, fake, odd, s) == prq.PRQ_EALIGN
    assert prq._quant_act_packed(fake, 1024, 4, 1024, 64, None, None, None, 1, None, fake, s) == prq.PRQ_EINVAL
    assert prq._quant_act_packed(fake, 1000, 4, 1024, 64, None, None, None, 1, fake, fake, s) == prq.PRQ_EINVAL
    assert prq._quant_act_packed(None, 1024, 0, 1024, 64, None, None, None, 1, None, None, s) == prq.PRQ_OK
    assert prq._gemm_packed(fake, fake, 4, fake, fake, 24, 1088, fake, None, 0, s) == prq.PRQ_EALIGN   # N % 16
    assert prq._gemm_packed(fake, odd, 4, fake, fake, 32, 1088, fake, None, 0, s) == prq.PRQ_EALIGN    # Aps
    assert prq._gemm_packed(fake, fake, 4, fake, odd, 32, 1088, fake, None, 0, s) == prq.PRQ_EALIGN    # Wps
    assert prq._gemm_packed(None, None, 0, fake, fake, 32, 1088, None, None, 0, s) == prq.PRQ_OK
    # grouped: G > 1 needs offsets; E >= 1 with offsets; Aps alignment
    assert prq._quant_act_packed(fake, 1024, 4, 1024, 64, None, None, None, 3, fake, fake, s) == prq.PRQ_EINVAL
    assert prq._quant_act_packed(fake, 1024, 4, 1024, 64, None, None, fake, 0, fake, fake, s) == prq.PRQ_EINVAL
    assert prq._ggemm_packed(fake, fake, None, 4, 8, fake, fake, 32, 1088, fake, s) == prq.PRQ_EINVAL
    assert prq._ggemm_packed(fake, fake, fake, 0, 8, fake, fake, 32, 1088, fake, s) == prq.PRQ_EINVAL
    assert prq._ggemm_packed(fake, odd, fake, 4, 8, fake, fake, 32, 1088, fake, s) == prq.PRQ_EALIGN
    assert prq._ggemm_packed(fake, fake, fake, 4, 8, fake, fake, 24, 1088, fake, s) == prq.PRQ_EALIGN
    assert prq._ggemm_packed(None, None, fake, 4, 0, fake, fake, 32, 1088, None, s) == prq.PRQ_OK


def test_packed_activation_sizes():
    """Row blocks of 16 rows, K steps of 128, scale groups of four steps."""
    assert prq.prq_packed_act_bytes(1, 32) == (1024, 256)
    assert prq.prq_packed_act_bytes(16, 128) == (1024, 256)
    assert prq.prq_packed_act_bytes(17, 129 * 32) == (2 * 33 * 1024, 2 * 9 * 256)
    assert prq.prq_packed_act_bytes(8192, 9984) == (512 * 78 * 1024, 512 * 20 * 256)
    assert prq.prq_packed_act_bytes(0, 9984) == (0, 0)
    with pytest.raises(prq.PRQError):
        prq.prq_packed_act_bytes(4, 1000)


def test_reference_packer_is_a_padded_permutation():
    """The tests' layout reference moves every code and scale byte exactly
    once and fills the rest with zero codes and scale byte 127."""
    from tests.packing import pack_rows
    rng = np.random.default_rng(3)
    for R, K_aug in ((1, 32), (17, 96), (33, 1088), (16, 512)):
        q = rng.integers(1, 256, (R, K_aug // 2), dtype=np.uint8)
        sc = rng.integers(0, 127, (R, K_aug // 32), dtype=np.uint8)
        P, Ps = pack_rows(q, sc)
        cb, sb = prq.prq_packed_act_bytes(R, K_aug)
        assert (P.size, Ps.size) == (cb, sb)
        assert np.sort(P[P != 0]).tolist() == np.sort(q.ravel()).tolist()
        assert np.sort(Ps[Ps != 127]).tolist() == np.sort(sc.ravel()).tolist()
        assert np.count_nonzero(Ps == 127) == sb - sc.size


HEAD = 16384   # every GEMM workspace: stream-K arrival counters first, scratch after


def test_workspace_sizes():
    # the LDS-tiled kernel splits along K when its tiles would leave CUs idle:
    # splits - 1 partial sums of M x N floats after the state head; a full
    # round of tiles is unsplit
    ws = prq.prq_gemm_workspace_bytes(64, 2560, 9984, prq.GEMM_TILE)
    assert ws > HEAD and (ws - HEAD) % (64 * 2560 * 4) == 0
    assert prq.prq_gemm_workspace_bytes(8192, 2560, 9984, prq.GEMM_TILE) == 0
    ws = prq.prq_gemm_packed_workspace_bytes(512, 2560, 9984)
    assert ws > HEAD and (ws - HEAD) % (512 * 2560 * 4) == 0
    assert prq.prq_gemm_packed_workspace_bytes(8192, 2560, 9984) == 0
    assert prq.prq_gemm_packed_workspace_bytes(512, 2560, 9980) == 0     # invalid K_aug
    assert prq.prq_gemm_workspace_bytes(64, 2560, 9984, prq.GEMM_STREAM, 1) == 0
    # a forced split count: partial sums [splits][M][N] added in a fixed order
    assert prq.prq_gemm_workspace_bytes(64, 2560, 9984, prq.GEMM_STREAM, 4) == HEAD + 4 * 64 * 2560 * 4
    assert prq.prq_gemm_workspace_bytes(16, 2560, 9984, prq.GEMM_STREAM, 2) == HEAD + 2 * 16 * 2560 * 4
    assert prq.prq_packed_weight_bytes(1, 2560, 9984) == (160 * 78 * 1024, 160 * 20 * 256)
    assert prq.prq_packed_weight_bytes(128, 2048, 832) == (128 * 128 * 7 * 1024, 128 * 128 * 2 * 256)
    assert prq.prq_grouped_gemm_workspace_bytes(512, 128, 2048, 832) == 0


def test_binding_rejects_operands_that_do_not_match_the_weight():
    """The binding checks tensor extents the C ABI cannot see (it gets bare
    pointers) before anything is launched: activations quantized for one
    K_aug against a weight packed for another, wrong dtypes, wrong Y, host
    tensors.  CPU tensors suffice: every check runs before the library call."""
    import torch
    M, N = 8, 64
    cb, sb = prq.prq_packed_weight_bytes(1, N, 9952)
    W = prq.PackedWeight(torch.zeros(cb, dtype=torch.uint8), torch.zeros(sb, dtype=torch.uint8),
                         1, N, 9952)
    Aq_small = torch.zeros((M, 2624 // 2), dtype=torch.uint8)
    Asc_small = torch.zeros((M, 2624 // 32), dtype=torch.uint8)
    with pytest.raises(ValueError, match="Aq has shape"):
        prq.prq_gemm(Aq_small, Asc_small, W, Y=torch.zeros((M, N)))
    Aq = torch.zeros((M, 9952 // 2), dtype=torch.uint8)
    Asc = torch.zeros((M, 9952 // 32), dtype=torch.uint8)
    with pytest.raises(ValueError, match="Asc has shape"):
        prq.prq_gemm(Aq, Asc_small, W, Y=torch.zeros((M, N)))
    with pytest.raises(ValueError, match="Y has shape"):
        prq.prq_gemm(Aq, Asc, W, Y=torch.zeros((M, N + 16)))
    with pytest.raises(ValueError, match="Y has dtype"):
        prq.prq_gemm(Aq, Asc, W, Y=torch.zeros((M, N), dtype=torch.float64))
    short = prq.PackedWeight(W.Wp[:-1], W.Wps, 1, N, 9952)
    with pytest.raises(ValueError, match="W.Wp has"):
        prq.prq_gemm(Aq, Asc, short, Y=torch.zeros((M, N)))
    with pytest.raises(ValueError, match="GPU tensor"):
        prq.prq_gemm(Aq, Asc, W, Y=torch.zeros((M, N)))
    off = torch.tensor([0, 3, M], dtype=torch.int32)
    W2 = prq.PackedWeight(torch.zeros(2 * cb, dtype=torch.uint8), torch.zeros(2 * sb, dtype=torch.uint8),
                          2, N, 9952)
    with pytest.raises(ValueError, match="group_offsets has shape"):
        prq.prq_grouped_gemm(Aq, Asc, off[:2], W2, Y=torch.zeros((M, N)))
    with pytest.raises(ValueError, match="group_offsets has dtype"):
        prq.prq_grouped_gemm(Aq, Asc, off.long(), W2, Y=torch.zeros((M, N)))
    with pytest.raises(ValueError, match="single weight"):
        prq.prq_gemm(Aq, Asc, W2, Y=torch.zeros((M, N)))

    K, k = 2560, 64
    X = torch.zeros((M, K), dtype=torch.int16)
    inv = torch.ones(K, dtype=torch.float32)
    perm = torch.arange(K, dtype=torch.int32)
    with pytest.raises(ValueError, match="X rows"):
        prq.prq_quant_act(X[:, :K - 32], K, k, inv, perm)
    with pytest.raises(ValueError, match="perm has dtype"):
        prq.prq_quant_act(X, K, k, inv, perm.long())
    with pytest.raises(ValueError, match="inv_scale_pos has"):
        prq.prq_quant_act(X, K, k, inv[: K // 2], perm)
    with pytest.raises(ValueError, match="perm has"):
        prq.prq_quant_act(X, K, k, torch.ones(2 * K), torch.arange(K, dtype=torch.int32),
                          group_offsets=torch.tensor([0, 4, M], dtype=torch.int32), G=2)
    with pytest.raises(ValueError, match="Aq has shape"):
        prq.prq_quant_act(X, K, k, inv, perm, Aq=torch.zeros((M, 9952 // 2), dtype=torch.uint8))
    with pytest.raises(ValueError, match="GPU tensor"):
        prq.prq_quant_act(X, K, k, inv, perm)
    with pytest.raises(ValueError, match="Wsc has shape"):
        prq.prq_pack_weight(torch.zeros((N, 1312), dtype=torch.uint8),
                            torch.zeros((N, 80), dtype=torch.uint8))


def test_evaluation_calls_reject_bad_arguments_before_the_gpu():
    """Argument errors of the offline evaluation calls are reported before any
    device work (these run on hosts without a GPU)."""
    import ctypes
    c = inputs.make_dense("s", N=32, K=64, M=4, T=4, k_tail=32, n_out=1)
    a = np.array([0.5, 1.5], np.float64)
    err = np.empty(2, np.float64)
    best = ctypes.c_int32()
    st = prq._search(c.W.ctypes.data, 32, 64, c.Xcal.ctypes.data, 4, a.ctypes.data, 2, 32, 0, 0,
                     err.ctypes.data, ctypes.byref(best), None)
    assert st == prq.PRQ_EINVAL                      # alpha outside [0, 1]
    st = prq._search(c.W.ctypes.data, 32, 64, c.Xcal.ctypes.data, 4, a.ctypes.data, 0, 32, 0, 0,
                     err.ctypes.data, ctypes.byref(best), None)
    assert st == prq.PRQ_EINVAL                      # no candidates
    st = prq._evaluate(c.W.ctypes.data, 30, 64, c.Xcal.ctypes.data, 4, c.X.ctypes.data, 4, 0.5, 32,
                       0, 0, err.ctypes.data, None)
    assert st == prq.PRQ_EALIGN                      # N not a multiple of 16
    st = prq._evaluate(None, 32, 64, c.Xcal.ctypes.data, 4, c.X.ctypes.data, 4, 0.5, 32, 0, 0,
                       err.ctypes.data, None)
    assert st == prq.PRQ_EINVAL


@pytest.mark.parametrize("gate", [True, False])
def test_expand_producer_matches_oracle(gate):
    rng = np.random.default_rng(4)
    f = inputs.make_ffn("f", H=96, C=320, M=2, T=2, seed=4)
    perm = rng.permutation(f.C).astype(np.int32)
    inv = rng.uniform(0.01, 30.0, f.C).astype(np.float32)
    up, gt = prq.prq_expand_producer(f.W_up, f.W_gate if gate else None, inv, perm, 96)
    rup, rgt = pq.expand_producer(f.W_up, f.W_gate if gate else None, inv, perm, 96)
    np.testing.assert_array_equal(up, rup)
    if gate:
        np.testing.assert_array_equal(gt, rgt)
    else:
        assert gt is None
    with pytest.raises(prq.PRQError):
        bad = perm.copy()
        bad[0] = f.C
        prq.prq_expand_producer(f.W_up, None, inv, bad, 96)


def test_streamk_workspace_sizes():
    """Stream-K workspace (256 CUs assumed without a GPU): none where the plan
    gives every tile its own workgroup (the down_proj's 160 tiles up to three
    row groups), else the
    state head and partial tiles [256][2][M][16] floats; 0 where the kernel does
    not apply (more than 64 rows, a tile over more than four workgroups).
    AUTO (the whole-K decode kernel at decode rows) asks for none."""
    for M in (1, 8, 32, 48):
        assert prq.prq_gemm_workspace_bytes(M, 2560, 9984, prq.GEMM_STREAM_K) == 0
    # four row groups of ten units a wave do not fit: one workgroup per CU
    assert prq.prq_gemm_workspace_bytes(64, 2560, 9984, prq.GEMM_STREAM_K) == HEAD + 256 * 2 * 64 * 16 * 4
    for M in (1, 8, 32, 64):
        assert prq.prq_gemm_workspace_bytes(M, 2560, 9984) == 0
        assert prq.prq_gemm_workspace_bytes(M, 1792, 9984) == 0
        assert prq.prq_gemm_workspace_bytes(M, 1792, 9984, prq.GEMM_STREAM_K) == HEAD + 256 * 2 * M * 16 * 4
    assert prq.prq_gemm_workspace_bytes(65, 2560, 9984, prq.GEMM_STREAM_K) == 0
    assert prq.prq_gemm_workspace_bytes(31, 1024, 9984, prq.GEMM_STREAM_K) == 0


def test_swiglu_quant_rejects_bad_arguments_before_the_gpu():
    """prq_swiglu_quant(_packed): argument errors are reported before any
    device work (null, negative M, ld below K_aug, K_aug not a multiple of 32,
    unaligned rows or outputs, K_aug past the limit); M == 0 is a no-op."""
    for fn in (prq._swiglu_quant, prq._swiglu_quant_packed):
        a = 256                                          # a 16-byte aligned stand-in address
        assert fn(a, a, 64, 0, 64, a, a, None) == prq.PRQ_OK
        assert fn(a, a, 64, -1, 64, a, a, None) == prq.PRQ_EINVAL
        assert fn(a, a, 32, 4, 64, a, a, None) == prq.PRQ_EINVAL
        assert fn(None, a, 64, 4, 64, a, a, None) == prq.PRQ_EINVAL
        assert fn(a, a, 64, 4, 64, None, a, None) == prq.PRQ_EINVAL
        assert fn(a, a, 96, 4, 80, a, a, None) == prq.PRQ_EALIGN
        assert fn(a + 2, a, 64, 4, 64, a, a, None) == prq.PRQ_EALIGN
        assert fn(a, a, 68, 4, 64, a, a, None) == prq.PRQ_EALIGN
        assert fn(a, a, 70000, 4, 65568, a, a, None) == prq.PRQ_EUNSUPPORTED
    assert prq._swiglu_quant_packed(256, 256, 64, 4, 64, 256, 260, None) == prq.PRQ_EALIGN
