"""Writes ablation_down_proj.json: the oracle's y-NRMSE of every ablation
variant (Sec. Ablation Studies) on the 9728 -> 2560 down-projection workload,
k = 256, alpha = 0.5, evaluated on its first 512 prefill rows.  Calls only the
oracle and the seeded input generator.  Run from the repository root:
    python tests/golden/make_ablation_down_proj.py
"""
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import prquant as pq              # noqa: E402
from paper_2609_22106_amd import inputs       # noqa: E402


def main():
    c = inputs.down_proj_prefill()
    X = c.X[:512]
    grid = pq.ablation_grid(X, c.W, c.Xcal, c.alpha, c.k_tail)
    out = {"workload": "qwen3_4b_down_proj, first 512 prefill rows", "N": c.N, "K": c.K,
           "k_tail": c.k_tail, "alpha": c.alpha, "seed": 0, "y_nrmse": grid}
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "ablation_down_proj.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
