"""The packed prefill pair: prq_quant_act_packed against the oracle's
quantizer (Algorithm 1, step 11; online copy) laid out by the reference packer
-- every code and scale byte, padding included -- and prq_gemm_packed (Eq. 3
over K + k) against the oracle's float64 GEMM, max |dY| <= 1e-3 max |Y|, for
every tile shape; then the two end to end on the down_proj shape."""
import ctypes

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import prquant as pq                               # noqa: E402
from paper_2609_22106_amd import inputs                        # noqa: E402
from tests.gpu_util import (assert_gemm_close, dev, host, nan_output, rows_per_block,  # noqa: E402
                            say)
from tests.packing import pack_rows                            # noqa: E402

pytestmark = pytest.mark.gpu


def _prq():
    from paper_2609_22106_amd import prq
    return prq


def _pos(inv, perm):
    return inv if perm is None else np.asarray(inv)[np.asarray(perm)]


QUANT = [(1, 1024, 64), (15, 1024, 64), (16, 1024, 0), (17, 96, 32), (300, 2560, 64),
         (33, 9728, 256), (257, 1088, 0)]


@pytest.mark.parametrize("M,K,k", QUANT)
@pytest.mark.parametrize("scaled", [True, False])
def test_quant_act_packed_bytes(M, K, k, scaled):
    prq = _prq()
    rng = np.random.default_rng(M * 13 + K + k + scaled)
    X = inputs.f32_to_bf16_bits((rng.standard_normal((M, K)) *
                                 rng.uniform(0.01, 30.0, K)).astype(np.float32))
    inv = rng.uniform(0.25, 4.0, K).astype(np.float32) if scaled else None
    perm = rng.permutation(K).astype(np.int32) if scaled else None
    say("packed quant case:", M, K, k, scaled)
    A = prq.prq_quant_act_packed(dev(X), K, k, None if inv is None else dev(_pos(inv, perm)),
                                 None if perm is None else dev(perm))
    torch.cuda.synchronize()
    rq, rs = pq.quant_act(X, inv, perm, k)
    ep, es = pack_rows(rq, rs)
    np.testing.assert_array_equal(host(A.Aps), es, err_msg="packed scales")
    np.testing.assert_array_equal(host(A.Ap), ep, err_msg="packed codes")


def test_quant_act_packed_overwrites_stale_padding():
    """Padding bytes are written, not left from a previous use of the buffers."""
    prq = _prq()
    rng = np.random.default_rng(5)
    M, K, k = 21, 1088, 32
    X = inputs.f32_to_bf16_bits(rng.standard_normal((M, K)).astype(np.float32))
    cb, sb = prq.prq_packed_act_bytes(M, K + k)
    out = prq.PackedAct(torch.full((cb,), 0xAB, dtype=torch.uint8, device="cuda"),
                        torch.full((sb,), 0xCD, dtype=torch.uint8, device="cuda"), M, K + k)
    prq.prq_quant_act_packed(dev(X), K, k, out=out)
    torch.cuda.synchronize()
    ep, es = pack_rows(*pq.quant_act(X, None, None, k))
    np.testing.assert_array_equal(host(out.Aps), es)
    np.testing.assert_array_equal(host(out.Ap), ep)


def _tune_quant_packed(X, K, k, inv_pos, perm, off, G, kernel, num_cus):
    """The packed quantizer through the tuning entry (kernel 3: output through
    the 8-row LDS window where it fits; 4: stored directly), its row ranges
    sized for num_cus CUs, into buffers pre-filled with other bytes."""
    from paper_2609_22106_amd import build
    prq = _prq()
    lib = ctypes.CDLL(build.PROBE_LIB)
    P, I = ctypes.c_void_p, ctypes.c_int
    lib.prq_tune_act_quant_packed.argtypes = [P, ctypes.c_int64, I, I, I, P, P, P, I, P, P, I, I,
                                              P]
    lib.prq_tune_act_quant_packed.restype = I
    M = X.shape[0]
    cb, sb = prq.prq_packed_act_bytes(M, K + k)
    Ap = torch.full((cb,), 0xAB, dtype=torch.uint8, device="cuda")
    Aps = torch.full((sb,), 0xCD, dtype=torch.uint8, device="cuda")
    Xd = dev(X)
    args = [dev(a) if a is not None else None for a in (inv_pos, perm, off)]
    rc = lib.prq_tune_act_quant_packed(
        Xd.data_ptr(), K, M, K, k, *[a.data_ptr() if a is not None else None for a in args], G,
        Ap.data_ptr(), Aps.data_ptr(), kernel, num_cus, torch.cuda.current_stream().cuda_stream)
    assert rc == 0, rc
    torch.cuda.synchronize()
    return host(Ap), host(Aps)


# (M, K, k, num_cus): row ranges of several rows that start and end inside
# 8-row windows (a CU count that makes them so), ragged M, K + k not a whole
# number of 128-element steps, the largest K + k each stage class takes through
# the window (2K in the first three classes, 14336 = 60928 window bytes in the
# 20480-byte class, 15360 = 65280 bytes in the 24576-byte class) and sizes past
# it (stored directly), the largest class (always direct).
WINDOW_QUANT = [(1000, 2560, 64, 13),     # 39 rows per workgroup, 8192-byte stages
                (517, 9728, 256, 7),      # 74 rows, the down_proj row, 20480-byte stages
                (60, 10240, 4096, 2),     # 20480-byte stages, K + k = 14336 (60928 bytes)
                (60, 10240, 4224, 2),     # K + k = 14464: past the window, stored directly
                (45, 8320, 96, 3),        # the shortest row of the 20480-byte class
                (300, 4096, 1024, 5),     # 30 rows
                (260, 8192, 2048, 3),     # 87 rows, 16384-byte stages
                (77, 2048, 2048, 2),      # 4096-byte stages, window exactly full
                (40, 12288, 3072, 2),     # 24576-byte stages, K + k = 15360 (65280 bytes)
                (40, 12288, 4096, 2),     # K + k = 16384: past the window, stored directly
                (24, 16384, 512, 2),      # 32768-byte stages: stored directly
                (100, 2080, 32, 3)]       # K + k = 2112 = 16.5 steps


@pytest.mark.parametrize("M,K,k,cus", WINDOW_QUANT)
@pytest.mark.parametrize("kernel", [3, 4])
def test_quant_act_packed_windows(kernel, M, K, k, cus):
    """The LDS-staged packed quantizer with multi-row workgroup ranges, its
    output through the 8-row LDS window (kernel 3) or stored directly (4):
    every code and scale byte, padding included, as the oracle's quantizer laid
    out by the reference packer."""
    rng = np.random.default_rng(M * 7 + K + k + kernel)
    X = inputs.f32_to_bf16_bits((rng.standard_normal((M, K)) *
                                 rng.uniform(0.01, 30.0, K)).astype(np.float32))
    inv = rng.uniform(0.25, 4.0, K).astype(np.float32)
    perm = rng.permutation(K).astype(np.int32)
    say("packed window quant case:", kernel, M, K, k, cus)
    ap, aps = _tune_quant_packed(X, K, k, _pos(inv, perm), perm, None, 1, kernel, cus)
    ep, es = pack_rows(*pq.quant_act(X, inv, perm, k))
    np.testing.assert_array_equal(aps, es, err_msg="packed scales")
    np.testing.assert_array_equal(ap, ep, err_msg="packed codes")


def _tune_packed(shape, A, W, Y):
    from paper_2609_22106_amd import build
    lib = ctypes.CDLL(build.PROBE_LIB)
    P, I = ctypes.c_void_p, ctypes.c_int
    lib.prq_tune_gemm_tile_packed.argtypes = [P, P, I, P, P, I, I, P, I, P]
    lib.prq_tune_gemm_tile_packed.restype = I
    return lib.prq_tune_gemm_tile_packed(A.Ap.data_ptr(), A.Aps.data_ptr(), A.M, W.Wp.data_ptr(),
                                         W.Wps.data_ptr(), W.N, W.K_aug, Y.data_ptr(), shape,
                                         torch.cuda.current_stream().cuda_stream)


GEMM = [(300, 384, 1024), (513, 272, 1152), (40, 512, 9984), (257, 272, 1088), (130, 144, 4192),
        (17, 48, 96), (64, 256, 256), (1, 16, 32),
        # decode rows (AUTO: the whole-K decode kernel on the packed operand): two
        # tiles per workgroup over an odd tile count, one tile for two-tile
        # workgroups, three row groups, ragged K + k
        (49, 80, 1088), (64, 16, 2624), (33, 272, 4192)]


@pytest.mark.parametrize("M,N,K_aug", GEMM)
@pytest.mark.parametrize("shape", [None, 0, 1, 2, 3])
def test_gemm_packed(shape, M, N, K_aug):
    prq = _prq()
    rng = np.random.default_rng(M * 31 + N + K_aug)
    Aq, Asc = inputs.random_mxfp4(rng, M, K_aug)
    Wq, Wsc = inputs.random_mxfp4(rng, N, K_aug)
    ap, aps = pack_rows(Aq, Asc)
    A = prq.PackedAct(dev(ap), dev(aps), M, K_aug)
    W = prq.prq_pack_weight(dev(Wq), dev(Wsc))
    say("packed gemm case:", shape, M, N, K_aug)
    if shape is None:
        Y = prq.prq_gemm_packed(A, W)
    else:
        Y = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
        assert _tune_packed(shape, A, W, Y) == 0
    torch.cuda.synchronize()
    assert_gemm_close(host(Y), pq.gemm(Aq, Asc, Wq, Wsc), f"packed shape {shape} {M}x{N}x{K_aug}")


def _staged_decode_one_tile(Aq, Asc, W):
    """The staged whole-K decode kernel on the row-major operand, forced to one
    tile per workgroup and one workgroup row (tuning entry)."""
    from paper_2609_22106_amd import build
    lib = ctypes.CDLL(build.PROBE_LIB)
    P, I = ctypes.c_void_p, ctypes.c_int
    lib.prq_tune_gemm_decode.argtypes = [P, P, I, P, I, P, P, I, I, P, I, I, P]
    A, S = dev(Aq), dev(Asc)
    M = Aq.shape[0]
    Y = nan_output(M, W.N)
    st = lib.prq_tune_gemm_decode(A.data_ptr(), S.data_ptr(), M, None, 1, W.Wp.data_ptr(),
                                  W.Wps.data_ptr(), W.N, W.K_aug, Y.data_ptr(), 1, 1,
                                  torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert st == 0
    return host(Y)


@pytest.mark.parametrize("M,N,K_aug", [(64, 2560, 9984), (17, 2560, 9984), (40, 2560, 9984),
                                       (32, 160, 9984), (49, 80, 1088), (64, 16, 2624),
                                       (20, 272, 4192), (33, 272, 4192), (30, 48, 2080),
                                       (48, 80, 2624), (40, 48, 10240)])
def test_packed_decode_direct_variant(M, N, K_aug):
    """prq_gemm_packed at two to four 16-row blocks runs the decode kernel's
    register-direct variant (operands loaded straight into registers; one tile
    per wave at two blocks, two tiles per wave from three): every element
    written, within the GEMM bar of the oracle, and bit for bit the staged
    kernel with one tile per workgroup (same K chunks, MFMA order and chunk
    sum).  Shapes: the down_proj at 17, 40 and 64 rows, a single tile (its
    second tile past N), an odd tile count with two tiles per wave, waves
    without K steps (1088 = 9 steps), a ragged last step (2080), rows past M
    in the last block, workgroup rows with unequal group counts, three whole
    blocks, and the longest K it takes (10240: 80 steps, five per wave)."""
    prq = _prq()
    rng = np.random.default_rng(M * 7 + N + K_aug)
    Aq, Asc = inputs.random_mxfp4(rng, M, K_aug)
    Wq, Wsc = inputs.random_mxfp4(rng, N, K_aug)
    ap, aps = pack_rows(Aq, Asc)
    A = prq.PackedAct(dev(ap), dev(aps), M, K_aug)
    W = prq.prq_pack_weight(dev(Wq), dev(Wsc))
    say("packed decode direct case:", M, N, K_aug)
    assert prq.prq_gemm_packed_workspace_bytes(M, N, K_aug) == 0
    Y = nan_output(M, N)
    prq.prq_gemm_packed(A, W, Y=Y)
    torch.cuda.synchronize()
    y = host(Y)
    assert np.all(np.isfinite(y)), "an output element was not written"
    np.testing.assert_array_equal(y.view(np.uint32), _staged_decode_one_tile(Aq, Asc, W).view(np.uint32))
    assert_gemm_close(y, pq.gemm(Aq, Asc, Wq, Wsc), f"packed decode direct {M}x{N}x{K_aug}")


@pytest.mark.parametrize("M,K,k", [(8192, 9728, 256), (4100, 9728, 224)])
def test_quant_act_packed_full_size_sampled_blocks(M, K, k):
    """The packed quantizer as the prefill benchmark launches it (the public
    entry on all CUs: 16 or more rows per workgroup of long rows, so the rows
    go through the 8-row LDS window), every code and scale byte of sampled
    16-row blocks -- the first, the last (ragged M: padded rows), blocks at
    workgroup range boundaries and random ones -- against the oracle's
    quantizer laid out by the reference packer."""
    prq = _prq()
    rng = np.random.default_rng(M + k)
    X = inputs.f32_to_bf16_bits((rng.standard_normal((M, K)) *
                                 rng.uniform(0.01, 30.0, K)).astype(np.float32))
    inv = rng.uniform(0.25, 4.0, K).astype(np.float32)
    perm = rng.permutation(K).astype(np.int32)
    say("packed quant full size case:", M, K, k)
    A = prq.prq_quant_act_packed(dev(X), K, k, dev(_pos(inv, perm)), dev(perm))
    torch.cuda.synchronize()
    ap, aps = host(A.Ap), host(A.Aps)
    nblk = -(-M // 16)
    steps = -(-(K + k) // 128)
    sgroups = -(-steps // 4)
    blocks = {0, nblk - 1, 1, nblk // 2, nblk // 2 - 1} | set(rng.choice(nblk, 6).tolist())
    for b in sorted(blocks):
        rows = np.arange(16 * b, min(16 * b + 16, M))
        ep, es = pack_rows(*pq.quant_act(X[rows], inv, perm, k))
        np.testing.assert_array_equal(ap[b * steps * 1024:(b + 1) * steps * 1024], ep,
                                      err_msg=f"codes of row block {b}")
        np.testing.assert_array_equal(aps[b * sgroups * 256:(b + 1) * sgroups * 256], es,
                                      err_msg=f"scales of row block {b}")


@pytest.mark.parametrize("M", [512, 2048, 8192])
def test_packed_pair_down_proj(M):
    """X -> prq_quant_act_packed -> prq_gemm_packed on the down_proj shape
    (K = 9728, k = 256, N = 2560), with the planner's workspace (split along K
    where it picks it) and without: every element of both outputs written (Y
    starts as NaN), and one oracle row in every 16-row block (so every row tile
    of every tile shape) within the GEMM bar."""
    prq = _prq()
    rng = np.random.default_rng(M)
    K, k, N = 9728, 256, 2560
    X = inputs.f32_to_bf16_bits((rng.standard_normal((M, K)) *
                                 rng.uniform(0.01, 30.0, K)).astype(np.float32))
    inv = rng.uniform(0.25, 4.0, K).astype(np.float32)
    perm = rng.permutation(K).astype(np.int32)
    Wq, Wsc = inputs.random_mxfp4(rng, N, K + k)
    W = prq.prq_pack_weight(dev(Wq), dev(Wsc))
    say("packed pair case:", M)
    A = prq.prq_quant_act_packed(dev(X), K, k, dev(_pos(inv, perm)), dev(perm))
    ws_n = prq.prq_gemm_packed_workspace_bytes(M, N, K + k)
    ws = torch.zeros(ws_n, dtype=torch.uint8, device="cuda") if ws_n else None
    Yd, Yd0 = nan_output(M, N), nan_output(M, N)     # both live: no reuse of one block
    prq.prq_gemm_packed(A, W, Y=Yd, workspace=ws)
    prq.prq_gemm_packed(A, W, Y=Yd0)
    Y, Y0 = host(Yd), host(Yd0)
    assert np.all(np.isfinite(Y)) and np.all(np.isfinite(Y0)), "an output element was not written"
    rows = rows_per_block(M, rng)
    rq, rs = pq.quant_act(X[rows], inv, perm, k)
    Yo = pq.gemm(rq, rs, Wq, Wsc)
    assert_gemm_close(Y[rows], Yo, f"packed pair M={M} workspace {ws_n}")
    assert_gemm_close(Y0[rows], Yo, f"packed pair M={M} without workspace")


@pytest.mark.parametrize("M", [1, 8, 17, 32, 64])
def test_packed_pair_decode_rows(M):
    """Decode rows through the packed pair on the down_proj shape: the
    quantizer's few-rows kernel writes the packed layout (codes, scales and the
    padding of the last 16-row block, byte for byte the oracle's), and the
    whole-K decode kernel reads it: every element written (Y starts as NaN),
    within the GEMM bar of the oracle, and, where both split K in the same 16
    chunks (up to two blocks; at four the row-major call takes two tiles per
    workgroup and 8 chunks), bit for bit the row-major pair's Y."""
    prq = _prq()
    rng = np.random.default_rng(M + 1000)
    K, k, N = 9728, 256, 2560
    X = inputs.f32_to_bf16_bits((rng.standard_normal((M, K)) *
                                 rng.uniform(0.01, 30.0, K)).astype(np.float32))
    inv = rng.uniform(0.25, 4.0, K).astype(np.float32)
    perm = rng.permutation(K).astype(np.int32)
    Wq, Wsc = inputs.random_mxfp4(rng, N, K + k)
    W = prq.prq_pack_weight(dev(Wq), dev(Wsc))
    say("packed decode pair case:", M)
    assert prq.prq_gemm_packed_workspace_bytes(M, N, K + k) == 0
    cb, sb = prq.prq_packed_act_bytes(M, K + k)
    A = prq.PackedAct(torch.full((cb,), 0xAB, dtype=torch.uint8, device="cuda"),
                      torch.full((sb,), 0xCD, dtype=torch.uint8, device="cuda"), M, K + k)
    prq.prq_quant_act_packed(dev(X), K, k, dev(_pos(inv, perm)), dev(perm), out=A)
    Yp = nan_output(M, N)
    prq.prq_gemm_packed(A, W, Y=Yp)
    Aq, Asc = prq.prq_quant_act(dev(X), K, k, dev(_pos(inv, perm)), dev(perm))
    Yr = nan_output(M, N)
    prq.prq_gemm(Aq, Asc, W, Y=Yr)
    torch.cuda.synchronize()
    rq, rs = pq.quant_act(X, inv, perm, k)
    ep, es = pack_rows(rq, rs)
    np.testing.assert_array_equal(host(A.Aps), es, err_msg="packed scales")
    np.testing.assert_array_equal(host(A.Ap), ep, err_msg="packed codes")
    yp = host(Yp)
    assert np.all(np.isfinite(yp)), "an output element was not written"
    if M <= 32:
        np.testing.assert_array_equal(yp.view(np.uint32), host(Yr).view(np.uint32))
    assert_gemm_close(yp, pq.gemm(rq, rs, Wq, Wsc), f"packed decode pair M={M}")
    assert_gemm_close(host(Yr), pq.gemm(rq, rs, Wq, Wsc), f"row-major decode pair M={M}")


def _random_decode_shapes(n, seed=7):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        M = int(rng.integers(17, 65))
        N = 16 * int(rng.integers(1, 41))
        K_aug = 32 * int(rng.integers(4, 321))          # up to 10240: at most 5 steps per wave
        out.append((M, N, K_aug))
    return out


@pytest.mark.parametrize("M,N,K_aug", _random_decode_shapes(12))
def test_packed_decode_direct_random_shapes(M, N, K_aug):
    """Seeded random decode shapes through prq_gemm_packed (17-64 rows: the
    direct variant): every element written, within the GEMM bar of the oracle,
    bit for bit the staged one-tile kernel."""
    prq = _prq()
    rng = np.random.default_rng(M * 131 + N * 7 + K_aug)
    Aq, Asc = inputs.random_mxfp4(rng, M, K_aug)
    Wq, Wsc = inputs.random_mxfp4(rng, N, K_aug)
    ap, aps = pack_rows(Aq, Asc)
    A = prq.PackedAct(dev(ap), dev(aps), M, K_aug)
    W = prq.prq_pack_weight(dev(Wq), dev(Wsc))
    say("packed decode random case:", M, N, K_aug)
    Y = nan_output(M, N)
    prq.prq_gemm_packed(A, W, Y=Y)
    torch.cuda.synchronize()
    y = host(Y)
    assert np.all(np.isfinite(y)), "an output element was not written"
    np.testing.assert_array_equal(y.view(np.uint32), _staged_decode_one_tile(Aq, Asc, W).view(np.uint32))
    assert_gemm_close(y, pq.gemm(Aq, Asc, Wq, Wsc), f"packed decode random {M}x{N}x{K_aug}")


@pytest.mark.parametrize("M,K,k,counts", [(1, 1024, 64, None), (40, 2080, 32, None),
                                          (100, 768, 64, None), (50, 1088, 0, [3, 0, 30, 17])])
def test_quant_act_packed_few_rows_kernel(M, K, k, counts):
    """The few-rows kernel forced (tuning entry, kernel 1) into the packed
    layout: one row per workgroup row and padding rows up to the end of the last
    16-row block, ragged K + k (2112 = 16.5 steps), more rows than AUTO gives
    it, and groups of sorted rows that share 16-row blocks."""
    rng = np.random.default_rng(M * 3 + K)
    X = inputs.f32_to_bf16_bits((rng.standard_normal((M, K)) *
                                 rng.uniform(0.01, 30.0, K)).astype(np.float32))
    if counts is None:
        inv = rng.uniform(0.25, 4.0, K).astype(np.float32)
        perm = rng.permutation(K).astype(np.int32)
        say("packed few-rows quant case:", M, K, k)
        ap, aps = _tune_quant_packed(X, K, k, _pos(inv, perm), perm, None, 1, 1, 256)
        rq, rs = pq.quant_act(X, inv, perm, k)
    else:
        G = len(counts)
        off = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
        assert off[-1] == M
        inv = rng.uniform(0.25, 4.0, (G, K)).astype(np.float32)
        perm = np.stack([rng.permutation(K) for _ in range(G)]).astype(np.int32)
        inv_pos = np.stack([inv[g][perm[g]] for g in range(G)])
        say("packed few-rows quant case: grouped", counts)
        ap, aps = _tune_quant_packed(X, K, k, inv_pos, perm, off, G, 1, 256)
        rq, rs = pq.quant_act_grouped(X, inv, perm, off, k)
    ep, es = pack_rows(rq, rs)
    np.testing.assert_array_equal(aps, es, err_msg="packed scales")
    np.testing.assert_array_equal(ap, ep, err_msg="packed codes")


@pytest.mark.parametrize("entry", ["packed", "rowmajor"])
def test_full_prefill_gemm_every_element(entry):
    """The largest down_proj prefill GEMM (8192 x 2560 over K + k = 9984) with
    random MXFP4 operands, every element of Y (which starts as NaN) against the
    oracle's float64 product: the packed pair's GEMM with its planner's
    workspace, and the row-major prq_gemm."""
    prq = _prq()
    rng = np.random.default_rng(8192)
    M, N, K_aug = 8192, 2560, 9984
    Aq, Asc = inputs.random_mxfp4(rng, M, K_aug)
    Wq, Wsc = inputs.random_mxfp4(rng, N, K_aug)
    W = prq.prq_pack_weight(dev(Wq), dev(Wsc))
    Yd = nan_output(M, N)
    say("full prefill gemm case:", entry)
    if entry == "packed":
        ap, aps = pack_rows(Aq, Asc)
        ws_n = prq.prq_gemm_packed_workspace_bytes(M, N, K_aug)
        ws = torch.zeros(ws_n, dtype=torch.uint8, device="cuda") if ws_n else None
        prq.prq_gemm_packed(prq.PackedAct(dev(ap), dev(aps), M, K_aug), W, Y=Yd, workspace=ws)
    else:
        prq.prq_gemm(dev(Aq), dev(Asc), W, Y=Yd)
    assert_gemm_close(host(Yd), pq.gemm(Aq, Asc, Wq, Wsc), f"full prefill {entry}")


@pytest.mark.parametrize("packed", [True, False])
def test_planned_column_regions(packed):
    """A GEMM whose columns the planner splits into two regions of different
    tile shapes (4096 x 9728 over K + k = 2624: 256 x 256 tiles over the first
    7680 columns, 256 x 128 over the rest), on 40 sampled rows, every column."""
    prq = _prq()
    rng = np.random.default_rng(21 + packed)
    M, N, K_aug = 4096, 9728, 2624
    Aq, Asc = inputs.random_mxfp4(rng, M, K_aug)
    Wq, Wsc = inputs.random_mxfp4(rng, N, K_aug)
    W = prq.prq_pack_weight(dev(Wq), dev(Wsc))
    say("planned regions case: packed =", packed)
    if packed:
        ap, aps = pack_rows(Aq, Asc)
        Y = prq.prq_gemm_packed(prq.PackedAct(dev(ap), dev(aps), M, K_aug), W)
    else:
        Y = prq.prq_gemm(dev(Aq), dev(Asc), W, variant=prq.GEMM_TILE)
    Y = host(Y)
    rows = np.unique(np.concatenate([rng.choice(M, 38, replace=False), [0, M - 1]]))
    assert_gemm_close(Y[rows], pq.gemm(Aq[rows], Asc[rows], Wq, Wsc), f"regions packed={packed}")



def _pos_grouped(inv, perm):
    return np.take_along_axis(np.asarray(inv), np.asarray(perm), axis=1)


# Experts sharing 16-row blocks, empty experts (first, middle and last), and
# K below (register-staged kernel) and above (LDS-staged kernel) 2048.
GROUPED_QUANT = [([3, 0, 20, 1, 13], 768, 64),
                 ([0, 37, 16, 0, 64, 5, 0], 768, 64),
                 ([40, 0, 90, 7], 4160, 160),
                 ([17, 1, 0, 33], 2048, 32)]


@pytest.mark.parametrize("counts,K,k", GROUPED_QUANT)
def test_quant_act_packed_grouped(counts, K, k):
    """Rows of several experts quantized with each expert's permutation and
    scales into one packed activation: every byte as the oracle's grouped
    quantizer laid out by the reference packer."""
    prq = _prq()
    rng = np.random.default_rng(sum(counts) + K + k)
    E = len(counts)
    off = inputs.routed_offsets(counts)
    M = int(off[-1])
    X = inputs.f32_to_bf16_bits((rng.standard_normal((M, K)) *
                                 rng.uniform(0.01, 30.0, K)).astype(np.float32))
    perm = np.stack([rng.permutation(K) for _ in range(E)]).astype(np.int32)
    inv = rng.uniform(0.1, 4.0, (E, K)).astype(np.float32)
    say("packed grouped quant case:", counts, K, k)
    A = prq.prq_quant_act_packed(dev(X), K, k, dev(_pos_grouped(inv, perm)), dev(perm),
                                 group_offsets=dev(off), G=E)
    torch.cuda.synchronize()
    ep, es = pack_rows(*pq.quant_act_grouped(X, inv, perm, off, k))
    np.testing.assert_array_equal(host(A.Aps), es, err_msg="packed scales")
    np.testing.assert_array_equal(host(A.Ap), ep, err_msg="packed codes")


# (M, K, k, num_cus) through the register-staged kernel: several rows per pass
# (each thread one unit of two rows, half a pass apart), a pass of exactly two
# rows (256 <= K/8 < 512), tiny rows, ragged ranges of many passes.
SHORT_QUANT = [(300, 768, 64, 7), (97, 2400, 96, 3), (1000, 64, 32, 5), (333, 96, 0, 2),
               (41, 4064, 32, 2)]


@pytest.mark.parametrize("M,K,k,cus", SHORT_QUANT)
def test_quant_act_packed_register_staged(M, K, k, cus):
    """The register-staged packed quantizer (forced) with multi-pass workgroup
    ranges: every code and scale byte, padding included, as the oracle's
    quantizer laid out by the reference packer."""
    rng = np.random.default_rng(M * 5 + K + k)
    X = inputs.f32_to_bf16_bits((rng.standard_normal((M, K)) *
                                 rng.uniform(0.01, 30.0, K)).astype(np.float32))
    inv = rng.uniform(0.25, 4.0, K).astype(np.float32)
    perm = rng.permutation(K).astype(np.int32)
    say("packed register-staged quant case:", M, K, k, cus)
    ap, aps = _tune_quant_packed(X, K, k, _pos(inv, perm), perm, None, 1, 2, cus)
    ep, es = pack_rows(*pq.quant_act(X, inv, perm, k))
    np.testing.assert_array_equal(aps, es, err_msg="packed scales")
    np.testing.assert_array_equal(ap, ep, err_msg="packed codes")


@pytest.mark.parametrize("counts,K,k,cus", [([5, 60, 0, 129, 1, 0, 33], 768, 64, 2),
                                            ([0, 3, 250, 7], 2400, 96, 3)])
def test_quant_act_packed_register_staged_grouped(counts, K, k, cus):
    """Grouped rows through the register-staged packed quantizer: a thread's
    two rows of a pass may belong to different experts."""
    rng = np.random.default_rng(sum(counts) + K)
    E = len(counts)
    off = inputs.routed_offsets(counts)
    M = int(off[-1])
    X = inputs.f32_to_bf16_bits((rng.standard_normal((M, K)) *
                                 rng.uniform(0.01, 30.0, K)).astype(np.float32))
    perm = np.stack([rng.permutation(K) for _ in range(E)]).astype(np.int32)
    inv = rng.uniform(0.1, 4.0, (E, K)).astype(np.float32)
    say("packed register-staged grouped quant case:", counts, K, k, cus)
    ap, aps = _tune_quant_packed(X, K, k, _pos_grouped(inv, perm), perm, off, E, 2, cus)
    ep, es = pack_rows(*pq.quant_act_grouped(X, inv, perm, off, k))
    np.testing.assert_array_equal(aps, es, err_msg="packed scales")
    np.testing.assert_array_equal(ap, ep, err_msg="packed codes")


# Experts changing inside 8-row windows and inside a workgroup's range.
GROUPED_WINDOW_QUANT = [([40, 0, 90, 7, 300], 4160, 160, 3),
                        ([17, 1, 0, 33, 250, 2], 2048, 32, 5),
                        ([5, 60, 0, 129], 9728, 256, 2)]


@pytest.mark.parametrize("counts,K,k,cus", GROUPED_WINDOW_QUANT)
@pytest.mark.parametrize("kernel", [3, 4])
def test_quant_act_packed_grouped_windows(kernel, counts, K, k, cus):
    """Grouped rows through the LDS-staged packed quantizer with multi-row
    workgroup ranges (window or direct output): every byte as the oracle's
    grouped quantizer laid out by the reference packer."""
    rng = np.random.default_rng(sum(counts) * 3 + K + k + kernel)
    E = len(counts)
    off = inputs.routed_offsets(counts)
    M = int(off[-1])
    X = inputs.f32_to_bf16_bits((rng.standard_normal((M, K)) *
                                 rng.uniform(0.01, 30.0, K)).astype(np.float32))
    perm = np.stack([rng.permutation(K) for _ in range(E)]).astype(np.int32)
    inv = rng.uniform(0.1, 4.0, (E, K)).astype(np.float32)
    say("packed grouped window quant case:", kernel, counts, K, k, cus)
    ap, aps = _tune_quant_packed(X, K, k, _pos_grouped(inv, perm), perm, off, E, kernel, cus)
    ep, es = pack_rows(*pq.quant_act_grouped(X, inv, perm, off, k))
    np.testing.assert_array_equal(aps, es, err_msg="packed scales")
    np.testing.assert_array_equal(ap, ep, err_msg="packed codes")


def _tune_grouped_packed(shape, A, off, W, Y, num_cus):
    from paper_2609_22106_amd import build
    lib = ctypes.CDLL(build.PROBE_LIB)
    P, I = ctypes.c_void_p, ctypes.c_int
    lib.prq_tune_grouped_gemm_tile_packed.argtypes = [P, P, I, P, I, P, P, I, I, P, I, I, P]
    lib.prq_tune_grouped_gemm_tile_packed.restype = I
    return lib.prq_tune_grouped_gemm_tile_packed(
        A.Ap.data_ptr(), A.Aps.data_ptr(), A.M, off.data_ptr(), W.E, W.Wp.data_ptr(),
        W.Wps.data_ptr(), W.N, W.K_aug, Y.data_ptr(), shape, num_cus,
        torch.cuda.current_stream().cuda_stream)


# Expert row ranges starting inside 16-row blocks, experts spanning more than
# one 256-row tile, empty experts, ragged N and K + k.
GROUPED_GEMM = [([0, 300, 0, 5, 260], 272, 1024),
                ([3, 0, 17, 1, 0], 48, 1088),
                ([0, 0, 200], 128, 832),
                ([255, 258, 1, 15, 16, 17, 600], 144, 832),
                ([7] * 40, 64, 4192),
                ([0, 3, 1, 0, 2] * 60, 32, 256)]      # 300 experts (38 per XCD), mostly one tile


@pytest.mark.parametrize("counts,N,K_aug", GROUPED_GEMM)
@pytest.mark.parametrize("shape,cus", [(None, None), (0, 0), (1, 0), (2, 0), (3, 0), (4, 256),
                                       (4, 8), (4, 1)])
def test_grouped_gemm_packed(shape, cus, counts, N, K_aug):
    """Every row of every expert stored exactly once (Y starts as NaN) and within
    1e-3 max |Y| of the oracle's grouped GEMM (Eq. 3 per expert): a workgroup per
    tile (shapes 0-3), or the persistent kernel (shape 4) in which each XCD's
    workgroups stride over its own experts' tiles with the next tile's loads in
    flight -- on all CUs, and on 8 or 1 CU(s) so that every workgroup runs many
    tiles back to back."""
    prq = _prq()
    rng = np.random.default_rng(sum(counts) * 7 + N + K_aug)
    E = len(counts)
    off = inputs.routed_offsets(counts)
    M = int(off[-1])
    Aq, Asc = inputs.random_mxfp4(rng, M, K_aug)
    Wq, Wsc = inputs.random_mxfp4(rng, (E, N), K_aug)
    A = prq.PackedAct(*map(dev, pack_rows(Aq, Asc)), M, K_aug)
    W = prq.prq_pack_weight(dev(Wq), dev(Wsc))
    offd = dev(off)
    Y = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    say("packed grouped gemm case:", shape, cus, counts, N, K_aug)
    if shape is None:
        prq.prq_grouped_gemm_packed(A, offd, W, Y)
    else:
        assert _tune_grouped_packed(shape, A, offd, W, Y, cus) == 0
    torch.cuda.synchronize()
    assert_gemm_close(host(Y), pq.grouped_gemm(Aq, Asc, off, Wq, Wsc),
                      f"grouped packed shape {shape} cus {cus} {counts} {N}x{K_aug}")


@pytest.mark.parametrize("counts", [[300], [0, 1, 0, 2] * 150, [33] * 513])
def test_grouped_gemm_packed_expert_counts(counts):
    """prq_grouped_gemm_packed's own choice at the ends of the expert range: one
    expert (persistent, all its tiles on one XCD), 600 experts and 513 experts
    (above the persistent kernel's 512: one workgroup per tile), against the
    oracle's grouped GEMM; every row stored (Y starts as NaN)."""
    prq = _prq()
    rng = np.random.default_rng(len(counts))
    E, N, K_aug = len(counts), 48, 320
    off = inputs.routed_offsets(counts)
    M = int(off[-1])
    Aq, Asc = inputs.random_mxfp4(rng, M, K_aug)
    Wq, Wsc = inputs.random_mxfp4(rng, (E, N), K_aug)
    A = prq.PackedAct(*map(dev, pack_rows(Aq, Asc)), M, K_aug)
    W = prq.prq_pack_weight(dev(Wq), dev(Wsc))
    Y = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    say("packed grouped expert-count case:", E, "experts,", M, "rows")
    prq.prq_grouped_gemm_packed(A, dev(off), W, Y)
    torch.cuda.synchronize()
    assert_gemm_close(host(Y), pq.grouped_gemm(Aq, Asc, off, Wq, Wsc), f"{E} experts")


def test_grouped_packed_pair_experts():
    """X -> prq_quant_act_packed -> prq_grouped_gemm_packed on the MoE expert
    shape (128 experts, 768 -> 2048, k = 64, 4096 tokens routed top-8 to
    distinct uniformly random experts): every element written (Y starts as
    NaN), and the first and last row of every expert plus one row of every
    16-row block against the oracle."""
    prq = _prq()
    E, K, k, N, tokens = 128, 768, 64, 2048, 4096
    rng = np.random.default_rng(2)
    routed = np.stack([rng.choice(E, 8, replace=False) for _ in range(tokens)])
    off = inputs.routed_offsets(np.bincount(routed.ravel(), minlength=E))
    M = int(off[-1])
    X = inputs.f32_to_bf16_bits((rng.standard_normal((M, K)) *
                                 rng.uniform(0.01, 30.0, K)).astype(np.float32))
    perm = np.stack([rng.permutation(K) for _ in range(E)]).astype(np.int32)
    inv = rng.uniform(0.1, 4.0, (E, K)).astype(np.float32)
    Wq, Wsc = inputs.random_mxfp4(rng, (E, N), K + k)
    W = prq.prq_pack_weight(dev(Wq), dev(Wsc))
    offd = dev(off)
    say("grouped packed pair case:", M, "rows")
    A = prq.prq_quant_act_packed(dev(X), K, k, dev(_pos_grouped(inv, perm)), dev(perm),
                                 group_offsets=offd, G=E)
    Yd = nan_output(M, N)
    prq.prq_grouped_gemm_packed(A, offd, W, Y=Yd)
    Y = host(Yd)
    assert np.all(np.isfinite(Y)), "an output element was not written"
    ends = np.concatenate([off[:-1][np.diff(off) > 0], off[1:][np.diff(off) > 0] - 1])
    rows = np.unique(np.concatenate([rows_per_block(M, rng), ends]))
    e_of = np.searchsorted(off, rows, side="right") - 1
    assert set(np.unique(e_of)) == set(np.flatnonzero(np.diff(off) > 0))
    for e in np.unique(e_of):
        r = rows[e_of == e]
        rq, rs = pq.quant_act(X[r], inv[e], perm[e], k)
        assert_gemm_close(Y[r], pq.gemm(rq, rs, Wq[e], Wsc[e]), f"expert {e} rows {r.tolist()}")


@pytest.mark.parametrize("name,N,K", inputs.LAYER_SET)
def test_packed_pair_layer_shapes(name, N, K):
    """The seven linears of a Qwen3-4B-shaped decoder layer at M = 4096 (k = K/40
    rounded down to a multiple of 32), through the packed pair as the benchmark
    launches it (the planner's tile shapes, column regions and workspace),
    every element written (Y starts as NaN), one oracle row in every 16-row
    block and every column."""
    prq = _prq()
    rng = np.random.default_rng(N + K)
    M, k = 4096, inputs.tail_width(K)
    X = inputs.f32_to_bf16_bits((rng.standard_normal((M, K)) *
                                 rng.uniform(0.01, 30.0, K)).astype(np.float32))
    inv = rng.uniform(0.25, 4.0, K).astype(np.float32)
    perm = rng.permutation(K).astype(np.int32)
    Wq, Wsc = inputs.random_mxfp4(rng, N, K + k)
    W = prq.prq_pack_weight(dev(Wq), dev(Wsc))
    say("layer shape case:", name, M, N, K, k)
    A = prq.prq_quant_act_packed(dev(X), K, k, dev(_pos(inv, perm)), dev(perm))
    ws_n = prq.prq_gemm_packed_workspace_bytes(M, N, K + k)
    ws = torch.zeros(ws_n, dtype=torch.uint8, device="cuda") if ws_n else None
    Yd = nan_output(M, N)
    prq.prq_gemm_packed(A, W, Y=Yd, workspace=ws)
    Y = host(Yd)
    assert np.all(np.isfinite(Y)), "an output element was not written"
    rows = rows_per_block(M, rng)
    rq, rs = pq.quant_act(X[rows], inv, perm, k)
    assert_gemm_close(Y[rows], pq.gemm(rq, rs, Wq, Wsc), f"{name} {M}x{N}x{K}+{k}")
