"""Synthetic ablation grid of Sec. Ablation Studies on the device path.

Every variant that keeps the contiguous tail is evaluated with
``prq_evaluate_nrmse`` (host export, then pack, act-quant and GEMM on the
GPU): plain MXFP4 (no scaling, k = 0), PRQuant, w/o AWQ (no scaling), w/o Res
(k = 0) and E8M0-W (weight-side block-scale search).  The "w/o Perm" variant
appends the residual of channels scattered among the main blocks, so its
activation tail is a gather of scattered channels quantized on its own --
exactly what the permutation exists to avoid -- and has no kernel here; its
numbers come from the CPU oracle in the tests.

``python -m paper_2609_22106_amd.ablation`` prints the grid for the
down-projection shape (9728 -> 2560, k = 256) and for the expert
down-projections (768 -> 2048, k = 64, mean over experts of the y-NRMSE on
each expert's routed rows), one JSON line each.
"""
from __future__ import annotations

import json
import sys

import numpy as np

VARIANTS = {   # name -> (scale_mode, uses k_tail, E8M0 search)
    "plain MXFP4": ("none", False, False),
    "PRQuant": ("smooth", True, False),
    "w/o AWQ": ("none", True, False),
    "w/o Res": ("smooth", False, False),
    "E8M0-W": ("smooth", True, True),
}


def run_grid(X_bf16, W_bf16, Xcal_bf16, alpha, k_tail):
    """y-NRMSE of each device-path variant on the rows X."""
    from . import prq
    out = {}
    for name, (mode, use_k, search) in VARIANTS.items():
        out[name] = prq.prq_evaluate_nrmse(W_bf16, Xcal_bf16, X_bf16, alpha,
                                           k_tail if use_k else 0, mode, scale_search=search)
    return out


def main(argv=None):
    from . import inputs
    c = inputs.down_proj_prefill()
    g = run_grid(c.X[:512], c.W, c.Xcal, c.alpha, c.k_tail)
    print(json.dumps({"workload": "qwen3_4b_down_proj (512 evaluation rows)", "N": c.N, "K": c.K,
                      "k_tail": c.k_tail, "alpha": c.alpha, "y_nrmse": g}), flush=True)
    m = inputs.moe_experts(4096)
    per = {name: [] for name in VARIANTS}
    off = m.group_offsets
    for e in range(m.E):
        r0, r1 = int(off[e]), int(off[e + 1])
        if r1 == r0:
            continue
        ge = run_grid(m.X[r0:r1], m.W[e], m.Xcal[e], m.alpha, m.k_tail)
        for name, v in ge.items():
            per[name].append(v)
    print(json.dumps({"workload": "qwen3_30b_a3b expert down_proj (mean over experts, routed rows)",
                      "E": m.E, "N": m.N, "K": m.K, "k_tail": m.k_tail, "alpha": m.alpha,
                      "experts_evaluated": len(per["PRQuant"]),
                      "y_nrmse": {k: float(np.mean(v)) for k, v in per.items()}}), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
