"""The offline evaluation calls (Algorithm 1's alpha search and the y-NRMSE of
one configuration) on the device path against the oracle: errors to the
float32-accumulation level (the reference product is float32 on the device,
float64 in the oracle) and the same selected alpha."""
import numpy as np
import pytest

pytest.importorskip("torch")

from oracle import prquant as pq                       # noqa: E402
from paper_2609_22106_amd import inputs                # noqa: E402
from tests.gpu_util import say                         # noqa: E402

pytestmark = pytest.mark.gpu

RTOL = 1e-4


@pytest.mark.parametrize("scale_search", [False, True])
def test_alpha_search_matches_oracle(scale_search):
    from paper_2609_22106_amd import prq
    c = inputs.tiny_case()
    alphas = [0.0, 0.25, 0.5, 0.75, 1.0]
    say("evaluate case: alpha search tiny, E8M0-W", scale_search)
    best, errs = prq.prq_search_alpha(c.W, c.Xcal, alphas, 64, scale_search=scale_search)
    ref_best, ref_errs = pq.search_alpha(c.W, c.Xcal, alphas, 64, scale_search=scale_search)
    say("errors", np.round(errs, 5), "oracle", np.round(ref_errs, 5))
    np.testing.assert_allclose(errs, ref_errs, rtol=RTOL)
    order = np.sort(ref_errs)
    if order[1] - order[0] > 4 * RTOL * order[0]:
        assert best == alphas[ref_best]


def test_evaluate_on_held_out_rows_matches_oracle():
    from paper_2609_22106_amd import prq
    c = inputs.make_dense("h", N=256, K=2048, M=96, T=128, k_tail=64, n_out=10, seed=21)
    for mode, k in (("smooth", 64), ("smooth", 0), ("none", 0)):
        say("evaluate case:", mode, k)
        got = prq.prq_evaluate_nrmse(c.W, c.Xcal, c.X, 0.5, k, mode)
        y, _ = pq.prquant_forward(c.X, c.W, c.Xcal, 0.5, k, mode)
        want = pq.nrmse(y, pq.reference_product(c.X, c.W))
        assert abs(got - want) <= RTOL * want, (mode, k, got, want)


def test_ablation_grid_matches_oracle():
    """The device-path ablation grid against the oracle's on a small shape."""
    from paper_2609_22106_amd import ablation
    c = inputs.make_dense("a", N=128, K=1024, M=64, T=64, k_tail=64, n_out=8, seed=31)
    got = ablation.run_grid(c.X, c.W, c.Xcal, 0.5, 64)
    want = pq.ablation_grid(c.X, c.W, c.Xcal, 0.5, 64)
    say("ablation grid", {k: round(v, 5) for k, v in got.items()}, "w/o Perm (oracle)",
        round(want["w/o Perm"], 5))
    for name, v in got.items():
        assert abs(v - want[name]) <= RTOL * want[name], (name, v, want[name])


def test_ablation_grid_full_down_proj_matches_stored_oracle():
    """The full 9728 -> 2560 workload (512 evaluation rows) against the oracle
    values written by tests/golden/make_ablation_down_proj.py."""
    import json
    import os
    from paper_2609_22106_amd import ablation
    with open(os.path.join(os.path.dirname(__file__), "golden", "ablation_down_proj.json")) as f:
        want = json.load(f)["y_nrmse"]
    c = inputs.down_proj_prefill()
    say("evaluate case: ablation grid, full down_proj")
    got = ablation.run_grid(c.X[:512], c.W, c.Xcal, c.alpha, c.k_tail)
    for name, v in got.items():
        assert abs(v - want[name]) <= RTOL * want[name], (name, v, want[name])
