"""The seeded workload generator: presets, determinism, the Zipf bias."""
import json
import os

import numpy as np

from paper_2603_02376_amd import inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_presets_match_the_workloads():
    p = inputs.PRESETS
    assert (p["tiny"]["T"], p["tiny"]["d"], p["tiny"]["E"], p["tiny"]["k"], p["tiny"]["I"]) == (64, 128, 8, 2, 256)
    assert (p["mixtral"]["d"], p["mixtral"]["E"], p["mixtral"]["k"], p["mixtral"]["I"]) == (4096, 8, 2, 14336)
    d = p["dsv3"]
    # GEMM1 7168 x 4096 (gate+up) and GEMM2 2048 x 7168 per expert
    assert (d["d"], 2 * d["I"], d["I"]) == (7168, 4096, 2048)
    assert (d["E"], d["n_groups"], d["topk_groups"], d["k"], d["scale"]) == (256, 8, 4, 8, 2.5)
    assert p["dsv3_decode"]["T"] == 128 and p["dsv3_skew"]["bias"] == "zipf"


def test_host_draws_are_deterministic():
    cfg = inputs.preset("dsv3", T=16)
    a = inputs.host_activations(cfg, 0)
    b = inputs.host_activations(cfg, 0)
    c = inputs.host_activations(cfg, 1)
    assert all((u == v).all() for u, v in zip(a[:2], b[:2]))
    assert not (a[0] == c[0]).all()
    assert abs(a[0].std() - 1.0) < 0.02 and abs(a[1].std() - 0.02) < 0.001


def test_tiny_inputs_on_cpu():
    cfg = inputs.preset("tiny")
    t = inputs.make_inputs(cfg, 0, "cpu")
    assert t["w_gate"].shape == (8, 256, 128) and t["w_down"].shape == (8, 128, 256)
    assert abs(float(t["w_down"].std()) - 1 / 16) < 0.003
    t2 = inputs.make_inputs(cfg, 0, "cpu")
    assert (t["w_up"] == t2["w_up"]).all()


def test_zipf_beta_matches_calibration_record():
    rec = json.load(open(os.path.join(GOLDEN, "zipf_beta.json")))
    assert rec["beta"] == inputs.ZIPF_BETA and rec["alpha"] == inputs.ZIPF_ALPHA
    assert 9.0 <= rec["max_over_mean"] <= 10.5 and rec["zero_load_experts"] >= 1
    b = inputs.zipf_bias(256)
    # the most popular expert gets the largest bias; bias is monotone in popularity rank
    order = inputs.host_rng(0, "zipf_order").permutation(256)
    assert np.argmax(b) == order[0] and np.argmin(b) == order[-1]
