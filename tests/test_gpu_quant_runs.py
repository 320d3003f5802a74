"""The quantizers with permutations of the form Algorithm 1 exports (head of
unselected channels in increasing order, then the selected ones): units of
8 consecutive channels are read as aligned 16-byte LDS pieces shifted into
place, the others channel by channel.  Every code and scale byte against the
oracle (row-major, and packed through the reference packer), for every
quantizer kernel that gathers from LDS, with runs at every alignment, runs
broken inside a wave, and the identity."""
import ctypes

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import prquant as pq                                            # noqa: E402
from paper_2609_22106_amd import inputs                                     # noqa: E402
from tests.gpu_util import dev, host, say, tail_permutation                 # noqa: E402
from tests.packing import pack_rows                                         # noqa: E402

pytestmark = pytest.mark.gpu


def _prq():
    from paper_2609_22106_amd import prq
    return prq


def _case(M, K, k, kind, seed):
    rng = np.random.default_rng(seed)
    X = inputs.f32_to_bf16_bits((rng.standard_normal((M, K)) *
                                 rng.uniform(0.01, 30.0, K)).astype(np.float32))
    inv = rng.uniform(0.25, 4.0, K).astype(np.float32)
    if kind == "identity":
        perm = np.arange(K, dtype=np.int32)
    else:
        perm = tail_permutation(rng, K, k, swaps=0 if kind == "tail" else 7)
    return X, inv, perm


KINDS = ["tail", "tail+swaps", "identity"]


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("M,K,k", [(65, 768, 64), (300, 2560, 64), (97, 4096, 96), (70, 9728, 256)])
def test_row_major_quantizer_runs(M, K, k, kind):
    prq = _prq()
    X, inv, perm = _case(M, K, k, kind, M + K)
    say("runs case: row-major", M, K, k, kind)
    Aq, Asc = prq.prq_quant_act(dev(X), K, k, dev(inv[perm]), dev(perm))
    torch.cuda.synchronize()
    rq, rs = pq.quant_act(X, inv, perm, k)
    np.testing.assert_array_equal(host(Asc), rs, err_msg="scales")
    np.testing.assert_array_equal(host(Aq), rq, err_msg="codes")


def _tune_packed(X, K, k, inv_pos, perm, off, G, kernel, num_cus):
    from paper_2609_22106_amd import build
    prq = _prq()
    lib = ctypes.CDLL(build.PROBE_LIB)
    P, I = ctypes.c_void_p, ctypes.c_int
    lib.prq_tune_act_quant_packed.argtypes = [P, ctypes.c_int64, I, I, I, P, P, P, I, P, P, I, I, P]
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


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("kernel", [0, 2, 3, 4])
@pytest.mark.parametrize("M,K,k,cus", [(97, 2400, 96, 3), (41, 9728, 256, 2), (300, 768, 64, 7),
                                       (37, 6144, 128, 2)])
def test_packed_quantizer_kernels_runs(M, K, k, cus, kernel, kind):
    """The automatic choice (0; at K = 6144 with 19 rows per workgroup, LDS
    row stages with the output window), register-staged rows (2), LDS row
    stages with the 8-row output window (3) and with direct output (4),
    multi-row workgroup ranges."""
    X, inv, perm = _case(M, K, k, kind, M * 3 + K + kernel)
    say("runs case: packed kernel", kernel, M, K, k, kind)
    ap, aps = _tune_packed(X, K, k, inv[perm], perm, None, 1, kernel, cus)
    ep, es = pack_rows(*pq.quant_act(X, inv, perm, k))
    np.testing.assert_array_equal(aps, es, err_msg="packed scales")
    np.testing.assert_array_equal(ap, ep, err_msg="packed codes")


@pytest.mark.parametrize("kind", ["tail", "tail+swaps"])
@pytest.mark.parametrize("counts,K,k", [([5, 60, 0, 129, 1, 0, 33], 768, 64),
                                        ([40, 0, 90, 7, 300], 4160, 160)])
def test_grouped_packed_quantizer_runs(counts, K, k, kind):
    """Each expert with its own tail permutation (rows of several experts in
    one pass or one workgroup range)."""
    prq = _prq()
    rng = np.random.default_rng(sum(counts) + K + len(kind))
    E = len(counts)
    off = inputs.routed_offsets(counts)
    M = int(off[-1])
    X = inputs.f32_to_bf16_bits((rng.standard_normal((M, K)) *
                                 rng.uniform(0.01, 30.0, K)).astype(np.float32))
    perm = np.stack([tail_permutation(rng, K, k, swaps=0 if kind == "tail" else 5)
                     for _ in range(E)]).astype(np.int32)
    inv = rng.uniform(0.1, 4.0, (E, K)).astype(np.float32)
    inv_pos = np.take_along_axis(inv, perm, axis=1)
    say("runs case: grouped packed", counts, K, k, kind)
    A = prq.prq_quant_act_packed(dev(X), K, k, dev(inv_pos), dev(perm), group_offsets=dev(off), G=E)
    torch.cuda.synchronize()
    ep, es = pack_rows(*pq.quant_act_grouped(X, inv, perm, off, k))
    np.testing.assert_array_equal(host(A.Aps), es, err_msg="packed scales")
    np.testing.assert_array_equal(host(A.Ap), ep, err_msg="packed codes")
