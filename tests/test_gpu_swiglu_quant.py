"""The gated activation quantized as it is formed (offline copy, producer
side: prq_swiglu_quant / prq_swiglu_quant_packed) against the oracle's
Q(SiLU(gate) * up) (oracle.prquant.swiglu_quant): every code and scale byte,
row-major and in the packed layout (its padding included); then the expanded
producers' outputs through it and the augmented GEMM against the oracle."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import prquant as pq                       # noqa: E402
from paper_2609_22106_amd import inputs                # noqa: E402
from tests.gpu_util import assert_gemm_close, dev, host, rows_per_block, say   # noqa: E402
from tests.packing import pack_rows                    # noqa: E402

pytestmark = pytest.mark.gpu


def _prq():
    from paper_2609_22106_amd import prq
    return prq


def _gate_up(rng, M, K, ld=None):
    """bf16 gate / up outputs: gate ~ 4 N(0,1) (SiLU's curved part, both
    tails), with some entries far into the tails (+-17..+-110, where SiLU is
    exact or -0), zeros of both signs; up ~ N(0,1) per-column scaled."""
    ld = ld or K
    gate = (rng.standard_normal((M, ld)) * 4).astype(np.float32)
    far = rng.random((M, ld)) < 0.02
    gate[far] = rng.choice([-110.0, -90.0, -88.5, -60.0, 17.0, 25.0, 95.0], far.sum())
    gate[rng.random((M, ld)) < 0.01] = 0.0
    gate[rng.random((M, ld)) < 0.01] = -0.0
    up = (rng.standard_normal((M, ld)) * rng.uniform(0.01, 8.0, ld)).astype(np.float32)
    return pq.bf16_round_bits(gate), pq.bf16_round_bits(up)


# (M, K_aug, ld): a single row; ragged rows; K_aug of one block, of whole 128
# steps and not (the packed layout's padding); strided rows; the down_proj
# width (K + k = 9728 + 256).
CASES = [(1, 32, None), (7, 96, None), (33, 2592, None), (300, 1024, 1040), (64, 9984, None),
         (17, 9984, 10000)]


@pytest.mark.parametrize("M,K_aug,ld", CASES)
def test_swiglu_quant_rows(M, K_aug, ld):
    prq = _prq()
    rng = np.random.default_rng(M * 5 + K_aug)
    g, u = _gate_up(rng, M, K_aug, ld)
    say("swiglu quant case:", M, K_aug, ld)
    Aq, Asc = prq.prq_swiglu_quant(dev(g), dev(u), K_aug)
    torch.cuda.synchronize()
    rq, rs = pq.swiglu_quant(g[:, :K_aug], u[:, :K_aug])
    np.testing.assert_array_equal(host(Asc), rs, err_msg="scales")
    np.testing.assert_array_equal(host(Aq), rq, err_msg="codes")


@pytest.mark.parametrize("M,K_aug,ld", CASES)
def test_swiglu_quant_packed(M, K_aug, ld):
    prq = _prq()
    rng = np.random.default_rng(M * 3 + K_aug + 1)
    g, u = _gate_up(rng, M, K_aug, ld)
    cb, sb = prq.prq_packed_act_bytes(M, K_aug)
    out = prq.PackedAct(torch.full((cb,), 0x5A, dtype=torch.uint8, device="cuda"),
                        torch.full((sb,), 0xA5, dtype=torch.uint8, device="cuda"), M, K_aug)
    say("swiglu quant packed case:", M, K_aug, ld)
    prq.prq_swiglu_quant(dev(g), dev(u), K_aug, packed=True, out=out)
    torch.cuda.synchronize()
    ep, es = pack_rows(*pq.swiglu_quant(g[:, :K_aug], u[:, :K_aug]))
    np.testing.assert_array_equal(host(out.Aps), es, err_msg="packed scales")
    np.testing.assert_array_equal(host(out.Ap), ep, err_msg="packed codes")


def test_swiglu_quant_full_prefill_rows_sampled():
    """The down_proj prefill size (M = 8192, K + k = 9984): every element of
    the packed output written (buffers pre-filled with other bytes), one row of
    every 16-row block against the oracle."""
    prq = _prq()
    M, K_aug = 8192, 9984
    gen = torch.Generator(device="cuda").manual_seed(7)
    gd = (torch.randn((M, K_aug), generator=gen, device="cuda") * 4).to(torch.bfloat16)
    ud = torch.randn((M, K_aug), generator=gen, device="cuda").to(torch.bfloat16)
    cb, sb = prq.prq_packed_act_bytes(M, K_aug)
    out = prq.PackedAct(torch.full((cb,), 0x5A, dtype=torch.uint8, device="cuda"),
                        torch.full((sb,), 0xA5, dtype=torch.uint8, device="cuda"), M, K_aug)
    say("swiglu quant full size case")
    prq.prq_swiglu_quant(gd, ud, K_aug, packed=True, out=out)
    Aq, Asc = prq.prq_swiglu_quant(gd, ud, K_aug)
    torch.cuda.synchronize()
    rows = rows_per_block(M, np.random.default_rng(8))
    g = host(gd.view(torch.int16)).view(np.uint16)[rows]
    u = host(ud.view(torch.int16)).view(np.uint16)[rows]
    rq, rs = pq.swiglu_quant(g, u)
    np.testing.assert_array_equal(host(Aq)[rows], rq)
    np.testing.assert_array_equal(host(Asc)[rows], rs)
    ep, es = pack_rows(host(Aq), host(Asc))       # the packed output is the row-major one laid out
    np.testing.assert_array_equal(host(out.Aps), es)
    np.testing.assert_array_equal(host(out.Ap), ep)


@pytest.mark.parametrize("M", [5, 300])
def test_offline_copy_producer_side_end_to_end(M):
    """Expanded producers (prq_expand_producer) -> their bf16 outputs -> the
    fused quantizer -> the augmented GEMM, against the oracle on the same
    producer outputs; the fused codes equal the oracle's bit for bit."""
    prq = _prq()
    f = inputs.make_ffn("f", H=256, C=1024, M=M, T=64, seed=M + 11)
    k = 64
    z_cal = pq.bf16_round_bits(pq.gated_ffn(f.X_cal, f.W_up, f.W_gate).astype(np.float32))
    art = prq.prq_prepare(f.W_down, z_cal, 0.5, k)
    up_aug, gate_aug = prq.prq_expand_producer(f.W_up, f.W_gate, art["inv_scale"], art["perm"], k)
    Xf = pq.bf16_bits_to_f32(f.X_hidden).astype(np.float64)
    up_out = pq.bf16_round_bits((Xf @ pq.bf16_bits_to_f32(up_aug).astype(np.float64).T).astype(np.float32))
    g_out = pq.bf16_round_bits((Xf @ pq.bf16_bits_to_f32(gate_aug).astype(np.float64).T).astype(np.float32))
    say("offline copy producer side case: M", M)
    A = prq.prq_swiglu_quant(dev(g_out), dev(up_out), f.C + k, packed=True)
    Aq, Asc = prq.prq_swiglu_quant(dev(g_out), dev(up_out), f.C + k)
    W = prq.prq_pack_weight(dev(art["Wq"]), dev(art["Wsc"]))
    Y = host(prq.prq_gemm_packed(A, W))
    Y2 = host(prq.prq_gemm(Aq, Asc, W))
    rq, rs = pq.swiglu_quant(g_out, up_out)
    np.testing.assert_array_equal(host(Aq), rq)
    np.testing.assert_array_equal(host(Asc), rs)
    Y_ref = pq.gemm(rq, rs, art["Wq"], art["Wsc"])
    assert_gemm_close(Y, Y_ref, f"producer side packed M={M}")
    assert_gemm_close(Y2, Y_ref, f"producer side row-major M={M}")
