"""prq_gemm / prq_grouped_gemm (Eq. 3 over K + k) against the oracle's float64
GEMM: max |dY| <= 1e-3 max |Y|.  Both kernels (LDS-tiled and weight-streaming
split-K), ragged M, N and K_aug, the full decode/prefill down_proj shapes and
the grouped expert shapes."""
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


def _packed(Wq, Wsc):
    return _prq().prq_pack_weight(dev(Wq), dev(Wsc))


def _gpu_gemm(Aq, Asc, Wq, Wsc, variant, splits=0, workspace=None):
    prq = _prq()
    Y = prq.prq_gemm(dev(Aq), dev(Asc), _packed(Wq, Wsc), variant=variant, splits=splits,
                     workspace=workspace)
    torch.cuda.synchronize()
    return host(Y)


SHAPES = [(1, 16, 32), (5, 48, 96), (16, 512, 1088), (100, 272, 1088), (64, 2560, 9984),
          (200, 256, 2624), (130, 144, 4192), (257, 128, 832), (33, 2048, 832)]


@pytest.mark.parametrize("M,N,K_aug", SHAPES)
@pytest.mark.parametrize("variant", ["tile", "stream"])
def test_random_operands(M, N, K_aug, variant):
    prq = _prq()
    rng = np.random.default_rng(M * 7 + N + K_aug)
    Aq, Asc = inputs.random_mxfp4(rng, M, K_aug)
    Wq, Wsc = inputs.random_mxfp4(rng, N, K_aug)
    v = prq.GEMM_TILE if variant == "tile" else prq.GEMM_STREAM
    say("gemm case:", variant, M, N, K_aug)
    assert_gemm_close(_gpu_gemm(Aq, Asc, Wq, Wsc, v), pq.gemm(Aq, Asc, Wq, Wsc),
                      f"{variant} {M}x{N}x{K_aug}")


def test_stream_forced_split_that_cannot_stage_is_rejected():
    """With a forced split count above one the split-K kernel runs; at 64 rows
    it stages the activation of the split in LDS, and two splits over 9984 K
    elements would need 64 rows x 39 steps (about 175 KB): the call is refused
    and nothing is launched."""
    prq = _prq()
    rng = np.random.default_rng(0)
    Aq, Asc = inputs.random_mxfp4(rng, 64, 9984)
    Wq, Wsc = inputs.random_mxfp4(rng, 320, 9984)
    with pytest.raises(prq.PRQError) as ei:
        _gpu_gemm(Aq, Asc, Wq, Wsc, prq.GEMM_STREAM, 2)
    assert ei.value.status == prq.PRQ_EINVAL


def _tune_decode(Aq, Asc, Wq, Wsc, tiles, row_splits, off=None, E=1):
    """The decode kernel with explicit tiles per workgroup and row splits."""
    import ctypes
    from paper_2609_22106_amd import build
    lib = ctypes.CDLL(build.PROBE_LIB)
    P, I = ctypes.c_void_p, ctypes.c_int
    lib.prq_tune_gemm_decode.argtypes = [P, P, I, P, I, P, P, I, I, P, I, I, P]
    W = _packed(Wq, Wsc)
    A, S = dev(Aq), dev(Asc)
    M = Aq.shape[0]
    Y = torch.full((M, W.N), float("nan"), dtype=torch.float32, device="cuda")
    o = dev(off) if off is not None else None
    st = lib.prq_tune_gemm_decode(A.data_ptr(), S.data_ptr(), M, None if o is None else o.data_ptr(),
                                  E, W.Wp.data_ptr(), W.Wps.data_ptr(), W.N, W.K_aug, Y.data_ptr(),
                                  tiles, row_splits, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    return st, host(Y)


@pytest.mark.parametrize("M,N,K_aug", [(1, 2560, 9984), (40, 320, 2624), (64, 272, 9984),
                                       (17, 48, 1088), (100, 160, 832)])
@pytest.mark.parametrize("tiles,row_splits", [(1, 1), (1, 4), (2, 2), (4, 1), (4, 3)])
def test_decode_kernel_configs(M, N, K_aug, tiles, row_splits):
    """Every tile count and row split (a workgroup looping over several row
    groups, partial last tile group, ragged rows and K); shapes whose K needs
    more weight steps per wave than the kernel holds are refused (-1)."""
    rng = np.random.default_rng(M * 31 + tiles * 7 + row_splits)
    Aq, Asc = inputs.random_mxfp4(rng, M, K_aug)
    Wq, Wsc = inputs.random_mxfp4(rng, N, K_aug)
    say("gemm case: decode", M, N, K_aug, "tiles", tiles, "row_splits", row_splits)
    st, Y = _tune_decode(Aq, Asc, Wq, Wsc, tiles, row_splits)
    steps = -(-K_aug // 128)
    if -(-steps // (16 // tiles)) > 10:
        assert st == -1
        return
    assert st == 0
    assert_gemm_close(Y, pq.gemm(Aq, Asc, Wq, Wsc), f"decode {M}x{N}x{K_aug} t{tiles} r{row_splits}")


@pytest.mark.parametrize("M,shift", [(1, 3), (9, 1), (33, 4), (40, 7), (64, 15)])
def test_decode_scale_rows_at_any_byte_offset(M, shift):
    """Asc carries no alignment requirement: the decode kernels read a row
    group's scale bytes as one run of 16-byte pieces from the aligned address
    below it.  Asc at offsets 1..15 from a 16-byte boundary, rows of
    K_aug / 32 = 82 bytes (not a multiple of 16), K_aug not a multiple of
    128 (the last step's K parts past K_aug); Y starts as NaN."""
    prq = _prq()
    rng = np.random.default_rng(M * 16 + shift)
    N, K_aug = 160, 2624
    Aq, Asc = inputs.random_mxfp4(rng, M, K_aug)
    Wq, Wsc = inputs.random_mxfp4(rng, N, K_aug)
    buf = torch.zeros(Asc.size + 64, dtype=torch.uint8, device="cuda")
    S = buf[shift:shift + Asc.size].view(M, K_aug // 32)
    S.copy_(dev(Asc))
    assert S.data_ptr() % 16 == shift % 16
    say("gemm case: decode scale offset", M, shift)
    Y = nan_output(M, N)
    prq.prq_gemm(dev(Aq), S, _packed(Wq, Wsc), Y=Y, variant=prq.GEMM_STREAM)
    torch.cuda.synchronize()
    assert_gemm_close(host(Y), pq.gemm(Aq, Asc, Wq, Wsc), f"decode scale offset {M} {shift}")


def test_decode_kernel_longest_rows():
    """K_aug = 16384 (512 scale blocks a row): 16 staged rows take 129 KB of
    LDS at one tile per workgroup; two tiles per workgroup need 16 weight
    steps per wave and are refused."""
    rng = np.random.default_rng(5)
    M, N, K_aug = 20, 64, 16384
    Aq, Asc = inputs.random_mxfp4(rng, M, K_aug)
    Wq, Wsc = inputs.random_mxfp4(rng, N, K_aug)
    say("gemm case: decode K_aug 16384")
    st, Y = _tune_decode(Aq, Asc, Wq, Wsc, 1, 2)
    assert st == 0
    assert_gemm_close(Y, pq.gemm(Aq, Asc, Wq, Wsc), "decode K_aug 16384")
    st, _ = _tune_decode(Aq, Asc, Wq, Wsc, 2, 2)
    assert st == -1


@pytest.mark.parametrize("M,splits", [(8, 1), (24, 0), (24, 2), (24, 3), (24, 7), (24, 19), (64, 6)])
def test_stream_split_counts(M, splits):
    prq = _prq()
    rng = np.random.default_rng(splits)
    N, K_aug = 320, 9984
    Aq, Asc = inputs.random_mxfp4(rng, M, K_aug)
    Wq, Wsc = inputs.random_mxfp4(rng, N, K_aug)
    say("gemm case: stream M", M, "splits", splits)
    Y = _gpu_gemm(Aq, Asc, Wq, Wsc, prq.GEMM_STREAM, splits)
    assert_gemm_close(Y, pq.gemm(Aq, Asc, Wq, Wsc), f"splits={splits}")


def test_split_k_workspace_reuse_and_two_splits_are_deterministic():
    """Repeated calls on one workspace with fresh activations stay correct (stale
    partial sums would show); the partial sums of a forced split count are
    added in a fixed order (bitwise repeatable) and the workspace's state head
    stays zero."""
    prq = _prq()
    rng = np.random.default_rng(3)
    N, K_aug = 2560, 9984
    Wq, Wsc = inputs.random_mxfp4(rng, N, K_aug)
    for M, splits in ((16, 2), (64, 6), (64, 8)):
        need = prq.prq_gemm_workspace_bytes(M, N, K_aug, prq.GEMM_STREAM, splits)
        ws = torch.zeros(need, dtype=torch.uint8, device="cuda")
        ys = []
        for call in range(3):   # new activations each call: stale partial sums would show
            Aq, Asc = inputs.random_mxfp4(rng, M, K_aug)
            y = _gpu_gemm(Aq, Asc, Wq, Wsc, prq.GEMM_STREAM, splits, ws)
            assert_gemm_close(y, pq.gemm(Aq, Asc, Wq, Wsc), f"M={M} split {splits} call {call}")
            assert int(torch.count_nonzero(ws[:16384])) == 0
        ys = [_gpu_gemm(Aq, Asc, Wq, Wsc, prq.GEMM_STREAM, splits, ws) for _ in range(3)]
        np.testing.assert_array_equal(ys[0].view(np.uint32), ys[1].view(np.uint32))
        np.testing.assert_array_equal(ys[0].view(np.uint32), ys[2].view(np.uint32))


def _tune_stream(Aq, Asc, Wq, Wsc, splits, waves, unroll, stage, reduce, wave_tiles, off=None,
                 E=1):
    """The weight-streaming kernel with an explicit configuration (one row
    group per pass, one tile group per workgroup)."""
    import ctypes
    from paper_2609_22106_amd import build
    lib = ctypes.CDLL(build.PROBE_LIB)
    P, I = ctypes.c_void_p, ctypes.c_int
    lib.prq_tune_gemm_stream.argtypes = [P, P, I, P, I, P, P, I, I, P] + [I] * 8 + [P, P]
    W = _packed(Wq, Wsc)
    A, S = dev(Aq), dev(Asc)
    M = Aq.shape[0]
    Y = torch.full((M, W.N), float("nan"), dtype=torch.float32, device="cuda")
    ws = torch.zeros(splits * M * W.N * 4 + 4 * 65536, dtype=torch.uint8, device="cuda")
    o = dev(off) if off is not None else None
    st = lib.prq_tune_gemm_stream(A.data_ptr(), S.data_ptr(), M, None if o is None else o.data_ptr(),
                                  E, W.Wp.data_ptr(), W.Wps.data_ptr(), W.N, W.K_aug, Y.data_ptr(),
                                  splits, waves, unroll, 1, 1, stage, reduce, wave_tiles,
                                  ws.data_ptr(), torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    return st, host(Y)


# (splits, waves, unroll, stage, reduce) over 9 K steps (K + k = 1088): one
# split, and three splits under each reduction (atomic accumulator with a last
# arriver, partial sums added by a second kernel, atomics into Y zeroed first).
WAVE_TILE_CFGS = [(1, 4, 3, 0, 0), (1, 8, 2, 1, 0), (3, 4, 1, 0, 0), (3, 4, 1, 1, 1),
                  (3, 8, 1, 0, 2)]


@pytest.mark.parametrize("splits,waves,unroll,stage,reduce", WAVE_TILE_CFGS)
def test_stream_four_tiles_per_wave(splits, waves, unroll, stage, reduce):
    """Four 16-feature tiles per wave sharing its activation operands: dense
    with N = 272 (17 tiles, the last group of four cut by N) and rows in two
    passes, and grouped with empty experts and an expert past 16 rows, each
    against the oracle's float64 GEMM."""
    rng = np.random.default_rng(splits * 10 + waves + stage + reduce)
    M, N, K_aug = 21, 272, 1088
    Aq, Asc = inputs.random_mxfp4(rng, M, K_aug)
    Wq, Wsc = inputs.random_mxfp4(rng, N, K_aug)
    say("gemm case: stream four tiles per wave", splits, waves, unroll, stage, reduce)
    st, Y = _tune_stream(Aq, Asc, Wq, Wsc, splits, waves, unroll, stage, reduce, 4)
    assert st == 0
    assert_gemm_close(Y, pq.gemm(Aq, Asc, Wq, Wsc), f"dense wave tiles {splits} {waves} {unroll}")
    if splits == 1:
        counts = [3, 0, 17, 1, 0]
        off, Aq, Asc, Wq, Wsc = _grouped_case(counts, 48, K_aug, 11)
        st, Y = _tune_stream(Aq, Asc, Wq, Wsc, 1, waves, unroll, stage, 0, 4, off=off,
                             E=len(counts))
        assert st == 0
        assert_gemm_close(Y, pq.grouped_gemm(Aq, Asc, off, Wq, Wsc), "grouped wave tiles")


def test_stream_four_tiles_per_wave_rejected_past_registers():
    """Configurations whose weight registers would not fit (more than four
    steps per wave, or more than one row group) are refused, nothing launched."""
    rng = np.random.default_rng(2)
    Aq, Asc = inputs.random_mxfp4(rng, 4, 1088)
    Wq, Wsc = inputs.random_mxfp4(rng, 64, 1088)
    st, _ = _tune_stream(Aq, Asc, Wq, Wsc, 1, 4, 6, 0, 0, 4)
    assert st == -1
    st, _ = _tune_stream(Aq, Asc, Wq, Wsc, 1, 16, 1, 0, 0, 4)
    assert st == -1


def test_decode_kernel_grouped_mode():
    """The decode kernel's grouped mode (one tile per workgroup, the expert's
    16-row groups looped in one workgroup), empty experts included."""
    counts = [0, 5, 40, 0, 17, 1]
    off, Aq, Asc, Wq, Wsc = _grouped_case(counts, 64, 1088, 5)
    say("gemm case: decode grouped", counts)
    st, Y = _tune_decode(Aq, Asc, Wq, Wsc, 1, 1, off=off, E=len(counts))
    assert st == 0
    assert_gemm_close(Y, pq.grouped_gemm(Aq, Asc, off, Wq, Wsc), "decode grouped")


@pytest.mark.parametrize("M", [1, 16, 300])
def test_e8m0_search_export_end_to_end(M):
    """Weights exported with the weight-side E8M0 block-scale search through
    the GPU act-quant and GEMM (decode and tile kernels) against the oracle."""
    prq = _prq()
    c = inputs.make_dense("e", N=256, K=1024, M=M, T=64, k_tail=64, n_out=8, out_scale=40.0,
                          heavy_tail=False, seed=M)
    art = prq.prq_prepare(c.W, c.Xcal, 0.5, 64, scale_search=True)
    ref = pq.prepare(c.W, c.Xcal, 0.5, 64, scale_search=True)
    np.testing.assert_array_equal(art["Wsc"], ref["Wsc"])
    say("gemm case: E8M0-W export M", M)
    Aq, Asc = prq.prq_quant_act(dev(c.X), 1024, 64, dev(art["inv_scale_pos"]), dev(art["perm"]))
    Y = host(prq.prq_gemm(Aq, Asc, _packed(art["Wq"], art["Wsc"])))
    rq, rs = pq.quant_act(c.X, ref["inv_scale"], ref["perm"], 64)
    assert_gemm_close(Y, pq.gemm(rq, rs, ref["Wq"], ref["Wsc"]), f"E8M0-W M={M}")


def test_hand_values():
    """All-ones A block x all-halves W block = 16 (one block); a second block at
    scales (130, 126) adds 64 (Eq. 3 by hand)."""
    prq = _prq()
    A = np.full((1, 32), 0x22, np.uint8)
    W = np.full((16, 32), 0x11, np.uint8)
    Asc = np.array([[127, 130]], np.uint8)
    Wsc = np.tile(np.array([[127, 126]], np.uint8), (16, 1))
    for v in (prq.GEMM_TILE, prq.GEMM_STREAM):
        Y = _gpu_gemm(A, Asc, W, Wsc, v)
        np.testing.assert_array_equal(Y, np.full((1, 16), 80.0, np.float32))


@pytest.mark.parametrize("M", [1, 8, 32, 64])
def test_down_proj_decode_end_to_end(c1_art, M):
    """9728 -> 2560, k = 256: oracle export, GPU act-quant + GEMM (auto kernel)
    against the oracle's Eq. 3."""
    prq = _prq()
    c, art = c1_art
    X = c.X[:M]
    say("gemm case: down_proj decode M =", M)
    Aq, Asc = prq.prq_quant_act(dev(X), 9728, 256, dev(art["inv_scale"][art["perm"]]), dev(art["perm"]))
    Y = prq.prq_gemm(Aq, Asc, _packed(art["Wq"], art["Wsc"]))
    torch.cuda.synchronize()
    rq, rs = pq.quant_act(X, art["inv_scale"], art["perm"], 256)
    assert_gemm_close(host(Y), pq.gemm(rq, rs, art["Wq"], art["Wsc"]), f"decode M={M}")


@pytest.mark.parametrize("M", [512, 2048, 8192])
def test_down_proj_prefill_sampled_rows(c1_art, M):
    """The oracle's down_proj export, GPU act-quant + prq_gemm (row-major
    activation, auto kernel): every element written (Y starts as NaN), one
    oracle row in every 16-row block and every column within the GEMM bar."""
    prq = _prq()
    _, art = c1_art
    c = inputs.down_proj_prefill()
    X = c.X[:M]
    say("gemm case: down_proj prefill M =", M)
    Aq, Asc = prq.prq_quant_act(dev(X), 9728, 256, dev(art["inv_scale"][art["perm"]]), dev(art["perm"]))
    Yd = nan_output(M, 2560)
    prq.prq_gemm(Aq, Asc, _packed(art["Wq"], art["Wsc"]), Y=Yd)
    Y = host(Yd)
    assert np.all(np.isfinite(Y)), "an output element was not written"
    rows = rows_per_block(M, np.random.default_rng(M))
    rq, rs = pq.quant_act(X[rows], art["inv_scale"], art["perm"], 256)
    assert_gemm_close(Y[rows], pq.gemm(rq, rs, art["Wq"], art["Wsc"]), f"prefill M={M}")


# ------------------------------------------------------------- grouped ---
def _grouped_case(counts, N, K_aug, seed):
    rng = np.random.default_rng(seed)
    off = inputs.routed_offsets(counts)
    Aq, Asc = inputs.random_mxfp4(rng, int(off[-1]), K_aug)
    Wq, Wsc = inputs.random_mxfp4(rng, (len(counts), N), K_aug)
    return off, Aq, Asc, Wq, Wsc


def _gpu_grouped(off, Aq, Asc, Wq, Wsc, variant):
    prq = _prq()
    Y = prq.prq_grouped_gemm(dev(Aq), dev(Asc), dev(off), _packed(Wq, Wsc), variant=variant)
    torch.cuda.synchronize()
    return host(Y)


GROUPED = [([3, 0, 17, 1, 0], 48, 1088), ([0, 0, 40], 32, 832), ([1], 16, 64),
           ([200, 3, 0, 65], 144, 832), ([0, 130, 0, 0, 7, 300], 256, 2624)]


@pytest.mark.parametrize("counts,N,K_aug", GROUPED)
@pytest.mark.parametrize("variant", ["tile", "stream"])
def test_grouped_random(counts, N, K_aug, variant):
    prq = _prq()
    off, Aq, Asc, Wq, Wsc = _grouped_case(counts, N, K_aug, sum(counts) + N)
    v = prq.GEMM_TILE if variant == "tile" else prq.GEMM_STREAM
    say("grouped case:", variant, counts, N, K_aug)
    Y = _gpu_grouped(off, Aq, Asc, Wq, Wsc, v)
    assert_gemm_close(Y, pq.grouped_gemm(Aq, Asc, off, Wq, Wsc), f"grouped {variant} {counts}")


@pytest.mark.parametrize("tokens", [64, 4096])
def test_grouped_expert_shapes(tokens):
    """128 experts of 2048 x 832 (768 + 64), rows routed top-8 (512 and 32768
    routed rows): every element of Y (which starts as NaN) against the oracle's
    grouped GEMM."""
    prq = _prq()
    rng = np.random.default_rng(tokens)
    E, N, K_aug = 128, 2048, 832
    experts = np.stack([rng.choice(E, 8, replace=False) for _ in range(tokens)])
    off = inputs.routed_offsets(np.bincount(experts.ravel(), minlength=E))
    Aq, Asc = inputs.random_mxfp4(rng, int(off[-1]), K_aug)
    Wq, Wsc = inputs.random_mxfp4(rng, (E, N), K_aug)
    say("grouped case: experts", tokens, "tokens")
    Yd = nan_output(int(off[-1]), N)
    prq.prq_grouped_gemm(dev(Aq), dev(Asc), dev(off), _packed(Wq, Wsc), Y=Yd)
    assert_gemm_close(host(Yd), pq.grouped_gemm(Aq, Asc, off, Wq, Wsc), f"experts {tokens} tokens")


def test_grouped_end_to_end_prepared_experts():
    """Eight experts of the 768 -> 2048 shape exported by the oracle, GPU grouped
    act-quant + grouped GEMM against the oracle."""
    prq = _prq()
    c = inputs.make_moe("m", E=8, N=2048, K=768, tokens=40, topk=3, T=256, k_tail=64, seed=4)
    arts = [pq.prepare(c.W[e], c.Xcal[e], 0.5, 64) for e in range(8)]
    inv = np.stack([a["inv_scale"] for a in arts])
    perm = np.stack([a["perm"] for a in arts])
    Wq = np.stack([a["Wq"] for a in arts])
    Wsc = np.stack([a["Wsc"] for a in arts])
    off = c.group_offsets
    say("grouped case: end to end, counts", np.diff(off).tolist())
    inv_pos = np.take_along_axis(inv, perm.astype(np.int64), axis=1)
    Aq, Asc = prq.prq_quant_act(dev(c.X), 768, 64, dev(inv_pos), dev(perm), dev(off), 8)
    for v in (prq.GEMM_TILE, prq.GEMM_STREAM):
        Y = prq.prq_grouped_gemm(Aq, Asc, dev(off), _packed(Wq, Wsc), variant=v)
        torch.cuda.synchronize()
        rq, rs = pq.quant_act_grouped(c.X, inv, perm, off, 64)
        np.testing.assert_array_equal(host(Aq), rq)
        assert_gemm_close(host(Y), pq.grouped_gemm(rq, rs, off, Wq, Wsc), f"e2e variant {v}")


# ------------------------------------------------------------- packing ---
def _pack_reference(Wq, Wsc):
    """The packed layout written out from its definition in include/prq.h."""
    return pack_rows(Wq, Wsc)


@pytest.mark.parametrize("E,N,K_aug", [(1, 16, 32), (1, 48, 1088), (3, 32, 832), (2, 64, 544)])
def test_pack_weight_layout(E, N, K_aug):
    prq = _prq()
    rng = np.random.default_rng(E * N + K_aug)
    Wq, Wsc = inputs.random_mxfp4(rng, (E, N), K_aug)
    W = prq.prq_pack_weight(dev(Wq), dev(Wsc))
    torch.cuda.synchronize()
    ref_p, ref_s = _pack_reference(Wq, Wsc)
    np.testing.assert_array_equal(host(W.Wp), ref_p)
    np.testing.assert_array_equal(host(W.Wps), ref_s)
