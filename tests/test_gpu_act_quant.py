"""prq_quant_act (fused inverse scale, permutation gather, MXFP4 quantize and
online tail copy) against the oracle: codes and scale bytes bit for bit."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import prquant as pq                       # noqa: E402
from paper_2609_22106_amd import inputs                # noqa: E402
from tests.golden import load_hand_blocks              # noqa: E402
from tests.gpu_util import dev, host, say              # noqa: E402

pytestmark = pytest.mark.gpu


def _pos(inv, perm):
    """Inverse scales in position order, inv_s[perm[p]] (per group when 2-D)."""
    if perm is None:
        return inv
    return np.take_along_axis(np.asarray(inv), np.asarray(perm).astype(np.int64), axis=-1)


def _gpu_quant(X_bits, K, k, inv=None, perm=None, offsets=None, G=1, ld=None):
    from paper_2609_22106_amd import prq
    M = X_bits.shape[0]
    if ld is not None and ld != K:
        Xp = np.zeros((M, ld), np.uint16)
        Xp[:, :K] = X_bits
        Xd = dev(Xp)
    else:
        Xd = dev(X_bits)
    Aq, Asc = prq.prq_quant_act(Xd, K, k, None if inv is None else dev(_pos(inv, perm)),
                                None if perm is None else dev(perm),
                                None if offsets is None else dev(offsets), G)
    torch.cuda.synchronize()
    return host(Aq), host(Asc)


def _check(X_bits, K, k, inv, perm, what, **kw):
    say("act_quant case:", what, X_bits.shape, "k =", k)
    Aq, Asc = _gpu_quant(X_bits, K, k, inv, perm, **kw)
    rq, rs = pq.quant_act(X_bits, inv, perm, k)
    np.testing.assert_array_equal(Asc, rs, err_msg=f"{what}: scales")
    np.testing.assert_array_equal(Aq, rq, err_msg=f"{what}: codes")


def test_tiny_workload():
    c = inputs.tiny_case()
    art = pq.prepare(c.W, c.Xcal, 0.5, 64)
    _check(c.X, 1024, 64, art["inv_scale"], art["perm"], "tiny 16x1024 k64")


@pytest.mark.parametrize("M", [1, 3, 17, 257, 1000])
def test_ragged_rows(M):
    c = inputs.make_dense("r", N=64, K=1024, M=M, T=32, k_tail=64, n_out=8, out_scale=40.0,
                          heavy_tail=False, seed=M)
    art = pq.prepare(c.W, c.Xcal, 0.5, 64)
    _check(c.X, 1024, 64, art["inv_scale"], art["perm"], f"M={M}")


@pytest.mark.parametrize("K,k,M", [(768, 64, 131), (4096, 96, 70), (4160, 160, 97), (9728, 224, 65),
                                   (12320, 288, 66), (16384, 512, 67)])
def test_many_row_kernel_shapes(K, k, M):
    """The many-row kernel at every units-per-thread count (K/8 over 512
    threads: 1 with several rows per pass, 1, 2, 3, 4 and the largest K),
    ragged row counts, random permutation and scales."""
    rng = np.random.default_rng(K + M)
    X = inputs.f32_to_bf16_bits((rng.standard_normal((M, K)) * 3).astype(np.float32))
    perm = rng.permutation(K).astype(np.int32)
    inv = rng.uniform(0.05, 8.0, K).astype(np.float32)
    _check(X, K, k, inv, perm, f"K={K} k={k} M={M}")


def test_few_row_kernel_grouped():
    """Grouped rows through the few-rows kernel (at most 64 rows): a workgroup's
    row range crosses experts, empty experts included."""
    rng = np.random.default_rng(13)
    E, K, k = 6, 768, 64
    counts = [3, 0, 20, 1, 0, 9]
    off = inputs.routed_offsets(counts)
    X = inputs.f32_to_bf16_bits((rng.standard_normal((int(off[-1]), K)) * 3).astype(np.float32))
    perm = np.stack([rng.permutation(K) for _ in range(E)]).astype(np.int32)
    inv = rng.uniform(0.1, 4.0, (E, K)).astype(np.float32)
    say("act_quant case: grouped few rows", counts)
    Aq, Asc = _gpu_quant(X, K, k, inv, perm, offsets=off, G=E)
    rq, rs = pq.quant_act_grouped(X, inv, perm, off, k)
    np.testing.assert_array_equal(Asc, rs)
    np.testing.assert_array_equal(Aq, rq)


@pytest.mark.parametrize("M", [1, 5, 48, 64])
def test_few_row_kernel_largest_rows(M):
    """K = 16384 (four staged rows of 32 KiB per workgroup at 64 rows)."""
    rng = np.random.default_rng(M)
    K, k = 16384, 512
    X = inputs.f32_to_bf16_bits((rng.standard_normal((M, K)) * 3).astype(np.float32))
    perm = rng.permutation(K).astype(np.int32)
    inv = rng.uniform(0.05, 8.0, K).astype(np.float32)
    _check(X, K, k, inv, perm, f"K=16384 M={M}")


def test_many_row_kernel_grouped_two_units_per_thread():
    rng = np.random.default_rng(12)
    E, K, k = 4, 4160, 160
    counts = [40, 0, 90, 7]
    off = inputs.routed_offsets(counts)
    X = inputs.f32_to_bf16_bits((rng.standard_normal((int(off[-1]), K)) * 2).astype(np.float32))
    perm = np.stack([rng.permutation(K) for _ in range(E)]).astype(np.int32)
    inv = rng.uniform(0.1, 4.0, (E, K)).astype(np.float32)
    say("act_quant case: grouped K=4160", counts)
    Aq, Asc = _gpu_quant(X, K, k, inv, perm, offsets=off, G=E)
    rq, rs = pq.quant_act_grouped(X, inv, perm, off, k)
    np.testing.assert_array_equal(Asc, rs)
    np.testing.assert_array_equal(Aq, rq)


def test_no_scale_no_perm_k0():
    rng = np.random.default_rng(4)
    X = inputs.f32_to_bf16_bits(rng.standard_normal((33, 512)).astype(np.float32) * 3)
    _check(X, 512, 0, None, None, "identity k0")


def test_whole_row_is_tail():
    """k = K: every block is copied once more."""
    c = inputs.make_dense("t", N=32, K=256, M=9, T=8, k_tail=256, n_out=2, seed=3)
    art = pq.prepare(c.W, c.Xcal, 0.5, 256)
    _check(c.X, 256, 256, art["inv_scale"], art["perm"], "k = K")


def test_random_permutation_and_scales():
    rng = np.random.default_rng(9)
    K = 2048
    X = inputs.f32_to_bf16_bits((rng.standard_normal((40, K)) * 5).astype(np.float32))
    perm = rng.permutation(K).astype(np.int32)
    inv = rng.uniform(0.01, 20.0, K).astype(np.float32)
    _check(X, K, 96, inv, perm, "random perm")


@pytest.mark.parametrize("K,M", [(96, 2), (1056, 31), (4192, 64), (9728, 17)])
def test_few_row_kernel_staged_row_pads(K, M):
    """The few-rows kernel copies each row whole into LDS in 1 KiB pieces: rows
    whose byte length is not a multiple of 1 KiB (the last piece partly past
    the row), strided rows (ld = K + 32), 1 to 4 rows per workgroup."""
    rng = np.random.default_rng(K + M)
    X = inputs.f32_to_bf16_bits((rng.standard_normal((M, K)) * 3).astype(np.float32))
    perm = rng.permutation(K).astype(np.int32)
    inv = rng.uniform(0.05, 8.0, K).astype(np.float32)
    k = 32
    say("act_quant case: staged row pads", K, M)
    Aq, Asc = _gpu_quant(X, K, k, inv, perm, ld=K + 32)
    rq, rs = pq.quant_act(X, inv, perm, k)
    np.testing.assert_array_equal(Asc, rs)
    np.testing.assert_array_equal(Aq, rq)


def test_strided_rows():
    c = inputs.tiny_case()
    art = pq.prepare(c.W, c.Xcal, 0.5, 64)
    _check(c.X, 1024, 64, art["inv_scale"], art["perm"], "ld 1056", ld=1056)


def test_hand_blocks_and_edge_values():
    """The hand-derived blocks (rounded to bf16), subnormals, signed zeros,
    huge values and exact E2M1 ties, with no scaling or permutation."""
    blocks = [b["values"] for b in load_hand_blocks()]
    rng = np.random.default_rng(1)
    ties = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 7.0, -0.25, -2.5, 6.0, -6.0] * 2
                    + [7.9, -7.9, 0.0, -0.0, 2.0 ** -130, -(2.0 ** -133), 3e38, -3e38], np.float32)
    extra = [np.concatenate([ties, rng.standard_normal(32 - ties.size % 32 if ties.size % 32 else 0)
                             .astype(np.float32)])]
    row = np.concatenate(blocks + extra)
    row = row[: row.size // 32 * 32]
    X = inputs.f32_to_bf16_bits(np.stack([row, -row, row * 0.75, row * np.float32(2.0 ** -120)]))
    K = X.shape[1]
    _check(X, K, 64, None, None, "hand blocks")


def test_full_decode_rows(c1_art):
    c, art = c1_art
    _check(c.X, 9728, 256, art["inv_scale"], art["perm"], "9728 k256 M=64")


def test_full_prefill_rows_sampled(c1_art):
    """8192 rows through the kernel; 256 sampled rows checked against the oracle."""
    _, art = c1_art
    c = inputs.down_proj_prefill()
    Aq, Asc = _gpu_quant(c.X, 9728, 256, art["inv_scale"], art["perm"])
    rows = np.sort(np.random.default_rng(0).choice(c.X.shape[0], 256, replace=False))
    rows = np.unique(np.concatenate([rows, [0, c.X.shape[0] - 1]]))
    rq, rs = pq.quant_act(c.X[rows], art["inv_scale"], art["perm"], 256)
    np.testing.assert_array_equal(Asc[rows], rs)
    np.testing.assert_array_equal(Aq[rows], rq)


def test_grouped_experts_with_empty_groups():
    rng = np.random.default_rng(2)
    E, K, k = 6, 768, 64
    counts = [5, 0, 70, 1, 0, 33]
    off = inputs.routed_offsets(counts)
    X = inputs.f32_to_bf16_bits((rng.standard_normal((int(off[-1]), K)) * 4).astype(np.float32))
    perms, invs = [], []
    for e in range(E):
        c = inputs.make_dense("g", N=32, K=K, M=1, T=16, k_tail=k, n_out=4, seed=100 + e)
        a = pq.prepare(c.W, c.Xcal, 0.5, k)
        perms.append(a["perm"])
        invs.append(a["inv_scale"])
    perm, inv = np.stack(perms), np.stack(invs)
    say("act_quant case: grouped", counts)
    Aq, Asc = _gpu_quant(X, K, k, inv, perm, offsets=off, G=E)
    rq, rs = pq.quant_act_grouped(X, inv, perm, off, k)
    np.testing.assert_array_equal(Asc, rs)
    np.testing.assert_array_equal(Aq, rq)
