"""Offline copy on the device path: the expanded producer emits [Z~, Z~_tail]
(C + k channels, bf16), prq_quant_act quantizes it as a plain MXFP4
quantizer (no permutation, no scales, no tail copy) and prq_gemm multiplies
it with the augmented weight -- against the oracle on the same inputs."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import prquant as pq                       # noqa: E402
from paper_2609_22106_amd import inputs                # noqa: E402
from tests.gpu_util import assert_gemm_close, dev, host, say   # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("M", [1, 40, 300])
def test_offline_copy_end_to_end(M):
    from paper_2609_22106_amd import prq
    f = inputs.make_ffn("f", H=256, C=1024, M=M, T=64, seed=M)
    k = 64
    z_cal = pq.bf16_round_bits(pq.gated_ffn(f.X_cal, f.W_up, f.W_gate).astype(np.float32))
    art = prq.prq_prepare(f.W_down, z_cal, 0.5, k)
    up_aug, gate_aug = prq.prq_expand_producer(f.W_up, f.W_gate, art["inv_scale"], art["perm"], k)
    z_aug = pq.bf16_round_bits(pq.gated_ffn(f.X_hidden, up_aug, gate_aug).astype(np.float32))
    say("offline copy case: M", M)
    Aq, Asc = prq.prq_quant_act(dev(z_aug), f.C + k, 0)
    torch.cuda.synchronize()
    rq, rs = pq.quant_act(z_aug, None, None, 0)
    np.testing.assert_array_equal(host(Asc), rs)
    np.testing.assert_array_equal(host(Aq), rq)
    W = prq.prq_pack_weight(dev(art["Wq"]), dev(art["Wsc"]))
    Y = host(prq.prq_gemm(Aq, Asc, W))
    Y_ref = pq.gemm(rq, rs, art["Wq"], art["Wsc"])
    assert_gemm_close(Y, Y_ref, f"offline copy M={M}")
    z = pq.bf16_round_bits(pq.gated_ffn(f.X_hidden, f.W_up, f.W_gate).astype(np.float32))
    oq, os_ = pq.quant_act(z, art["inv_scale"], art["perm"], k)
    ref = pq.reference_product(z, f.W_down)
    say(f"y-NRMSE offline copy {pq.nrmse(Y_ref, ref):.5f}, online copy "
        f"{pq.nrmse(pq.gemm(oq, os_, art['Wq'], art['Wsc']), ref):.5f}")
