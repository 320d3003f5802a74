"""The hot path captured into a HIP graph and replayed: every replay, with the
program's own eager work and synchronizations between replays, must match the
eager result (quantized activations bit for bit, GEMM outputs to float32
summation-order noise).  Covers the stream GEMM in both reduction modes its
decode defaults use (in-kernel atomics that leave the workspace zeroed, and
per-split partial sums plus a reduction kernel), the tile GEMM and the grouped
GEMM.  Nothing on the path allocates or clears memory with a memset, so the
captured graph holds kernel nodes only."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2609_22106_amd import inputs                # noqa: E402
from tests.gpu_util import dev, say                    # noqa: E402

pytestmark = pytest.mark.gpu


def _ops(prq, rng, K, k, N, M_list):
    K_aug = K + k
    Wq, Wsc = inputs.random_mxfp4(rng, N, K_aug)
    W = prq.prq_pack_weight(dev(Wq), dev(Wsc))
    inv = torch.from_numpy(rng.uniform(0.25, 4.0, K).astype(np.float32)).cuda()
    perm = torch.from_numpy(rng.permutation(K).astype(np.int32)).cuda()
    X = dev(inputs.f32_to_bf16_bits(rng.standard_normal((max(M_list), K)).astype(np.float32)))
    ops = []
    for M in M_list:
        Aq = torch.empty((M, K_aug // 2), dtype=torch.uint8, device="cuda")
        Asc = torch.empty((M, K_aug // 32), dtype=torch.uint8, device="cuda")
        Y = torch.empty((M, N), dtype=torch.float32, device="cuda")
        n = prq.prq_gemm_workspace_bytes(M, N, K_aug)
        ws = torch.zeros(n, dtype=torch.uint8, device="cuda") if n else None

        def run(M=M, Aq=Aq, Asc=Asc, Y=Y, ws=ws):
            prq.prq_quant_act(X[:M], K, k, inv, perm, Aq=Aq, Asc=Asc)
            prq.prq_gemm(Aq, Asc, W, Y=Y, workspace=ws)
        ops.append((run, (Aq, Asc, Y)))
    return ops


def _grouped_op(prq, rng):
    counts = [0, 70, 3, 0, 300, 1]
    E, N, K, k = len(counts), 256, 768, 64
    K_aug = K + k
    off = dev(inputs.routed_offsets(counts))
    Wq, Wsc = inputs.random_mxfp4(rng, (E, N), K_aug)
    W = prq.prq_pack_weight(dev(Wq), dev(Wsc))
    inv = torch.from_numpy(rng.uniform(0.5, 2.0, (E, K)).astype(np.float32)).cuda()
    perm = torch.from_numpy(np.stack([rng.permutation(K) for _ in range(E)]).astype(np.int32)).cuda()
    M = sum(counts)
    X = dev(inputs.f32_to_bf16_bits(rng.standard_normal((M, K)).astype(np.float32)))
    Aq = torch.empty((M, K_aug // 2), dtype=torch.uint8, device="cuda")
    Asc = torch.empty((M, K_aug // 32), dtype=torch.uint8, device="cuda")
    Y = torch.empty((M, N), dtype=torch.float32, device="cuda")

    def run():
        prq.prq_quant_act(X, K, k, inv, perm, group_offsets=off, G=E, Aq=Aq, Asc=Asc)
        prq.prq_grouped_gemm(Aq, Asc, off, W, Y=Y)
    return run, (Aq, Asc, Y)


def test_graph_replays_match_eager():
    from paper_2609_22106_amd import prq
    rng = np.random.default_rng(11)
    ops = _ops(prq, rng, 9728, 256, 2560, [1, 8, 32, 64])      # stream GEMM, both reductions
    ops += _ops(prq, rng, 2560, 64, 1024, [300])                 # tile GEMM
    ops.append(_grouped_op(prq, rng))                            # grouped GEMM + grouped quant
    say("graph case: decode M=1,8,32,64; tile M=300; grouped 6 experts")
    for run, _ in ops:
        run()
    torch.cuda.synchronize()
    ref = [tuple(t.clone() for t in bufs) for _, bufs in ops]

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for run, _ in ops:
            run()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for run, _ in ops:
            run()

    for rep in range(4):
        for _, (Aq, Asc, Y) in ops:           # eager work between replays
            Aq.zero_()
            Asc.fill_(255)
            Y.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for i, ((_, (Aq, Asc, Y)), (rq, rs, ry)) in enumerate(zip(ops, ref)):
            assert torch.equal(Aq, rq) and torch.equal(Asc, rs), f"replay {rep} op {i}: activations"
            assert torch.isfinite(Y).all(), f"replay {rep} op {i}: output not written"
            err = float((Y - ry).abs().max() / ry.abs().max().clamp_min(1e-30))
            assert err <= 1e-6, f"replay {rep} op {i}: GEMM differs from eager by {err:.2e}"
        say(f"graph replay {rep}: every op matches eager")
    del g
