"""Calibrate the Zipf-shaped bias of the skewed DeepSeek-V3 workload.

Finds, by bisection, the scale beta of the bias b_e = beta * ln(E * p_r(e))
for which the oracle's routing of the seeded dsv3 inputs sends ~10x the mean
load to the busiest expert, and writes tests/golden/zipf_beta.json. Calls only
the oracle and the seeded input generator. Run from the repository root:
    python tests/golden/make_zipf_beta.py
"""
import json
import os
import sys

import numpy as np
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import moe_oracle as O  # noqa: E402
from paper_2603_02376_amd import inputs  # noqa: E402


def routed_counts(logits, cfg, beta):
    bias = inputs.zipf_bias(cfg["E"], 0, beta=beta)
    idx, _ = O.route(logits, k=cfg["k"], score="sigmoid", bias=bias, n_groups=cfg["n_groups"],
                     topk_groups=cfg["topk_groups"], scale=cfg["scale"])
    return np.bincount(idx.reshape(-1), minlength=cfg["E"])


def main():
    cfg = inputs.preset("dsv3_skew")
    x, wr, _ = inputs.host_activations(cfg, 0)
    xb = inputs.oracle_view(torch.from_numpy(x).to(torch.bfloat16))
    wb = inputs.oracle_view(torch.from_numpy(wr).to(torch.bfloat16))
    logits = O.gate_logits(xb, wb)
    mean = cfg["T"] * cfg["k"] / cfg["E"]
    target = inputs.ZIPF_TARGET_MAX_OVER_MEAN
    lo, hi = 0.0, 1.0
    for _ in range(40):
        mid = 0.5 * (lo + hi)
        if routed_counts(logits, cfg, mid).max() / mean < target:
            lo = mid
        else:
            hi = mid
    beta = round(hi, 6)
    c = routed_counts(logits, cfg, beta)
    rec = dict(beta=beta, alpha=inputs.ZIPF_ALPHA, target_max_over_mean=target,
               max_over_mean=float(c.max() / mean), zero_load_experts=int((c == 0).sum()),
               max_count=int(c.max()), mean_count=mean,
               source="tests/golden/make_zipf_beta.py (oracle routing of the seeded dsv3 inputs, seed 0)")
    with open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "zipf_beta.json"), "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps(rec))


if __name__ == "__main__":
    main()
