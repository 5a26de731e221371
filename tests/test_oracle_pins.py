"""Pins for the CPU oracle: checks against things other than the oracle itself.

The paper prints no numeric value for the MoE layer, so every pin here is a
closed form, a hand-derived worked example, a brute-force enumeration on tiny
inputs written independently (pure Python, ``math``), a special case that
reduces to a textbook computation, or an invariant. Each is chosen so that a
plausible slip in the oracle (a dropped term, a wrong sign or index, a
transposed or swapped operand, the bias leaking into the weights, a wrong tie
rule, an unstable permutation) fails at least one of them.
"""

import itertools
import json
import math
import os
import random

import numpy as np
import pytest

from oracle import moe_oracle as O
from oracle.checks import check_dispatch, check_routing, max_rel_err

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _sig(z):
    return 1.0 / (1.0 + math.exp(-z))


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# ---------------------------------------------------------------------------
# decoding of bf16 bit patterns
# ---------------------------------------------------------------------------

def test_bf16_decode_known_bits():
    bits = np.array([0x3F80, 0xC000, 0x3E80, 0x0000, 0x8000, 0x7F7F, 0x3F81], dtype=np.uint16)
    want = [1.0, -2.0, 0.25, 0.0, -0.0, 3.3895313892515355e38, 1.0 + 2.0 ** -7]
    got = O.to_f64(bits)
    assert got.tolist() == want


# ---------------------------------------------------------------------------
# routing: worked examples (tests/golden/routing_examples.json)
# ---------------------------------------------------------------------------

def test_w1_sigmoid_group_limited_worked_example():
    ex = _load("routing_examples.json")["W1"]
    u = np.array([ex["logits"]])
    b = np.array(ex["bias"])
    idx, w, det = O.route(u, k=ex["k"], score="sigmoid", bias=b, n_groups=ex["n_groups"],
                          topk_groups=ex["topk_groups"], scale=ex["scale"], return_detail=True)
    assert idx[0].tolist() == ex["topk_idx"]
    assert sorted(det["chosen_groups"][0].tolist()) == ex["groups"]
    # weights from the unbiased sigmoid of the chosen logits, in closed form
    s = [_sig(ex["logits"][e]) for e in ex["topk_idx"]]
    want = [ex["scale"] * v / sum(s) for v in s]
    assert np.allclose(w[0], want, rtol=0, atol=1e-15)
    assert abs(w[0].sum() - ex["scale"]) < 1e-14
    # group scores: the two largest keys in each group
    keys = [_sig(v) + bb for v, bb in zip(ex["logits"], ex["bias"])]
    gs = [keys[2 * g] + keys[2 * g + 1] for g in range(4)]
    assert np.allclose(det["group_score"][0], gs, rtol=0, atol=1e-15)


def test_w2_softmax_top2_closed_form_and_tie():
    ex = _load("routing_examples.json")["W2"]
    idx, w = O.route(np.array([ex["case_a"]["logits"]]), k=2, score="softmax")
    assert idx[0].tolist() == ex["case_a"]["topk_idx"]
    # e^0.7 / (e^0.7 + e^0.4) = sigmoid(0.3)
    assert abs(w[0, 0] - _sig(0.3)) < 1e-15 and abs(w[0, 1] - _sig(-0.3)) < 1e-15
    idx, w = O.route(np.array([ex["case_b"]["logits"]]), k=2, score="softmax")
    assert idx[0].tolist() == ex["case_b"]["topk_idx"]
    assert w[0].tolist() == [0.5, 0.5]


def test_all_equal_logits_pick_lowest_indices():
    for score, scale in (("softmax", 1.0), ("sigmoid", 2.5)):
        u = np.full((3, 256), 0.37)
        kw = dict(n_groups=8, topk_groups=4) if score == "sigmoid" else {}
        idx, w = O.route(u, k=8, score=score, scale=scale, **kw)
        # groups 0..3 tie with all others and win on index; experts 0..7 lie in group 0
        assert (idx == np.arange(8)).all()
        assert np.allclose(w, scale / 8, rtol=0, atol=1e-15)


def test_large_bias_forces_expert():
    rng = np.random.default_rng(5)
    u = rng.normal(size=(50, 64))
    b = np.zeros(64)
    b[37] = 10.0
    for ng, tg in ((1, 1), (8, 2)):
        idx, w = O.route(u, k=4, score="sigmoid", bias=b, n_groups=ng, topk_groups=tg, scale=2.5)
        assert (idx[:, 0] == 37).all()
        # the weight uses the unbiased score: equal to 2.5 * s37 / sum(s)
        s = 1.0 / (1.0 + np.exp(-u))
        want = 2.5 * s[:, 37] / np.take_along_axis(s, idx, axis=1).sum(axis=1)
        assert np.allclose(w[:, 0], want, rtol=0, atol=1e-14)


# ---------------------------------------------------------------------------
# routing: brute-force enumeration on tiny inputs
# ---------------------------------------------------------------------------

def _brute_route(u, bias, k, score, n_groups, topk_groups, renorm, scale):
    E = len(u)
    if score == "softmax":
        m = max(u)
        z = [math.exp(v - m) for v in u]
        prob = [v / sum(z) for v in z]
        keys = list(u)
    else:
        prob = [_sig(v) for v in u]
        keys = [p + (bias[e] if bias is not None else 0.0) for e, p in enumerate(prob)]
    gsize = E // n_groups
    groups = [list(range(g * gsize, (g + 1) * gsize)) for g in range(n_groups)]
    if n_groups > 1:
        def gscore(g):
            mem = groups[g]
            if len(mem) == 1:
                return keys[mem[0]]
            return max(keys[a] + keys[b] for a, b in itertools.combinations(mem, 2))
        best = max(itertools.combinations(range(n_groups), topk_groups),
                   key=lambda c: sum(gscore(g) for g in c))
        eligible = [e for g in best for e in groups[g]]
    else:
        eligible = list(range(E))
    chosen = max(itertools.combinations(eligible, k), key=lambda c: sum(keys[e] for e in c))
    chosen = sorted(chosen, key=lambda e: -keys[e])
    w = [prob[e] for e in chosen]
    if renorm:
        tot = sum(w)
        w = [v / tot for v in w]
    return chosen, [scale * v for v in w]


@pytest.mark.parametrize("case", [
    dict(E=8, k=3, score="sigmoid", n_groups=4, topk_groups=2, renorm=True, scale=2.5, bias=True),
    dict(E=12, k=4, score="sigmoid", n_groups=3, topk_groups=2, renorm=True, scale=1.0, bias=True),
    dict(E=6, k=2, score="sigmoid", n_groups=6, topk_groups=3, renorm=True, scale=1.0, bias=False),
    dict(E=8, k=2, score="softmax", n_groups=1, topk_groups=1, renorm=True, scale=1.0, bias=False),
    dict(E=7, k=3, score="softmax", n_groups=1, topk_groups=1, renorm=False, scale=1.0, bias=False),
    dict(E=9, k=3, score="sigmoid", n_groups=1, topk_groups=1, renorm=False, scale=2.0, bias=True),
])
def test_route_matches_brute_force(case):
    rnd = random.Random(1234 + case["E"] * 7 + case["k"])
    T = 40
    u = [[rnd.gauss(0.0, 1.5) for _ in range(case["E"])] for _ in range(T)]
    bias = [rnd.gauss(0.0, 0.3) for _ in range(case["E"])] if case["bias"] else None
    idx, w = O.route(np.array(u), k=case["k"], score=case["score"],
                     bias=None if bias is None else np.array(bias),
                     n_groups=case["n_groups"], topk_groups=case["topk_groups"],
                     renorm=case["renorm"], scale=case["scale"])
    for t in range(T):
        want_idx, want_w = _brute_route(u[t], bias, case["k"], case["score"], case["n_groups"],
                                        case["topk_groups"], case["renorm"], case["scale"])
        assert idx[t].tolist() == want_idx, t
        assert np.allclose(w[t], want_w, rtol=1e-13, atol=1e-15), t


def test_k_equals_E_softmax_is_dense_softmax():
    rnd = random.Random(3)
    u = [rnd.gauss(0, 1) for _ in range(6)]
    idx, w = O.route(np.array([u]), k=6, score="softmax")
    m = max(u)
    z = [math.exp(v - m) for v in u]
    p = [v / sum(z) for v in z]
    assert sorted(idx[0].tolist()) == list(range(6))
    for j, e in enumerate(idx[0]):
        assert abs(w[0, j] - p[e]) < 1e-15


def test_route_margin_marks_ties():
    u = np.array([[0.0, 1.0, 1.0, -1.0],      # the two selected keys tie; next key is 1 lower
                  [2.0, 1.0, 1.0, -1.0],      # 2nd and 3rd keys tie -> margin 0
                  [3.0, 2.0, 1.0, 0.0]])
    _, _, det = O.route(u, k=2, score="softmax", return_detail=True)
    assert det["margin"].tolist() == [1.0, 0.0, 1.0]


# ---------------------------------------------------------------------------
# dispatch
# ---------------------------------------------------------------------------

def test_w3_dispatch_worked_example():
    ex = _load("routing_examples.json")["W3"]
    counts, offsets, st, sa, inv = O.dispatch(np.array(ex["topk_idx"]), ex["E"])
    assert counts.tolist() == ex["counts"]
    assert offsets.tolist() == ex["offsets"]
    assert st.tolist() == ex["sorted_token"]
    assert sa.tolist() == ex["sorted_assign"]
    assert inv.tolist() == ex["inv_perm"]


def _brute_dispatch(idx, E):
    T, k = len(idx), len(idx[0])
    triples = sorted((idx[t][j], t, t * k + j) for t in range(T) for j in range(k))
    counts = [sum(1 for tr in triples if tr[0] == e) for e in range(E)]
    offsets = [0]
    for c in counts:
        offsets.append(offsets[-1] + c)
    st = [tr[1] for tr in triples]
    sa = [tr[2] for tr in triples]
    inv = [0] * (T * k)
    for r, a in enumerate(sa):
        inv[a] = r
    return counts, offsets, st, sa, inv


@pytest.mark.parametrize("T,E,k", [(0, 4, 2), (1, 8, 8), (3, 5, 2), (17, 16, 4), (64, 8, 2), (50, 256, 8)])
def test_dispatch_matches_brute_force(T, E, k):
    rnd = random.Random(T * 131 + E * 7 + k)
    idx = [rnd.sample(range(E), k) for _ in range(T)]
    arr = np.array(idx, dtype=np.int32).reshape(T, k)
    got = O.dispatch(arr, E)
    want = _brute_dispatch(idx, E) if T else ([0] * E, [0] * (E + 1), [], [], [])
    for g, w in zip(got, want):
        assert g.tolist() == list(w)
    check_dispatch(arr, got[0], got[1], got[2], got[4], got[3])


def test_dispatch_hot_expert_and_empty_experts():
    T, k, E = 40, 2, 16
    idx = np.stack([np.full(T, 3), np.arange(T) % 2 + 10], axis=1).astype(np.int32)
    counts, offsets, st, sa, inv = O.dispatch(idx, E)
    assert counts[3] == T and counts[10] == 20 and counts[11] == 20
    assert counts.sum() == T * k and (counts[[0, 1, 2, 4, 5, 15]] == 0).all()
    check_dispatch(idx, counts, offsets, st, inv, sa)


def test_checker_detects_planted_mistakes():
    rnd = random.Random(9)
    idx = np.array([rnd.sample(range(8), 2) for _ in range(20)], dtype=np.int32)
    counts, offsets, st, sa, inv = O.dispatch(idx, 8)
    check_dispatch(idx, counts, offsets, st, inv, sa)
    # swap two rows inside one segment -> order no longer stable
    e = int(np.argmax(counts))
    lo = offsets[e]
    st2, inv2 = st.copy(), inv.copy()
    st2[[lo, lo + 1]] = st2[[lo + 1, lo]]
    a, b = sa[lo], sa[lo + 1]
    inv2[a], inv2[b] = inv2[b], inv2[a]
    with pytest.raises(AssertionError):
        check_dispatch(idx, counts, offsets, st2, inv2)
    # corrupt one count
    c2 = counts.copy()
    c2[0] += 1
    c2[1] -= 1
    with pytest.raises(AssertionError):
        check_dispatch(idx, c2, offsets, st, inv)
    # non-bijective inverse
    inv3 = inv.copy()
    inv3[0] = inv3[1]
    with pytest.raises(AssertionError):
        check_dispatch(idx, counts, offsets, st, inv3)
    # routing: duplicate expert and wrong weight sum
    with pytest.raises(AssertionError):
        check_routing(np.array([[1, 1]]), np.array([[0.5, 0.5]]), 4)
    with pytest.raises(AssertionError):
        check_routing(np.array([[1, 2]]), np.array([[0.5, 0.6]]), 4)


# ---------------------------------------------------------------------------
# expert FFN
# ---------------------------------------------------------------------------

def test_silu_closed_forms():
    assert O.silu(1.0) == pytest.approx(0.7310585786300049, abs=1e-16)
    assert O.silu(-1.0) == pytest.approx(-0.2689414213699951, abs=1e-16)
    assert O.silu(0.0) == 0.0
    assert O.silu(-800.0) == 0.0          # exp overflow must not produce nan


def test_swiglu_scalar_closed_form_distinguishes_gate_and_up():
    # d = I = 1: y = w_d * silu(w_g * a) * (w_u * a)
    a, wg, wu, wd = 1.0, 2.0, 3.0, 5.0
    y = O.swiglu_ffn(np.array([[a]]), np.array([[wg]]), np.array([[wu]]), np.array([[wd]]))
    want = wd * (wg * a * _sig(wg * a)) * (wu * a)
    swapped = wd * (wu * a * _sig(wu * a)) * (wg * a)
    assert y[0, 0] == pytest.approx(want, rel=1e-15)
    assert abs(want - swapped) > 1.0


def _loop_ffn(x, wg, wu, wd):
    M, d = len(x), len(x[0])
    I = len(wg)
    out = [[0.0] * d for _ in range(M)]
    for m in range(M):
        h = []
        for i in range(I):
            g = sum(x[m][c] * wg[i][c] for c in range(d))
            u = sum(x[m][c] * wu[i][c] for c in range(d))
            h.append(g * _sig(g) * u)
        for c in range(d):
            out[m][c] = sum(h[i] * wd[c][i] for i in range(I))
    return out


def _rand_mat(rnd, r, c, s=1.0):
    return [[rnd.gauss(0, s) for _ in range(c)] for _ in range(r)]


def test_swiglu_matches_loops_on_nonsquare_shapes():
    rnd = random.Random(11)
    M, d, I = 3, 5, 4
    x, wg, wu, wd = _rand_mat(rnd, M, d), _rand_mat(rnd, I, d), _rand_mat(rnd, I, d), _rand_mat(rnd, d, I)
    got = O.swiglu_ffn(np.array(x), np.array(wg), np.array(wu), np.array(wd))
    assert np.allclose(got, _loop_ffn(x, wg, wu, wd), rtol=1e-13, atol=1e-14)


def test_expert_ffn_segments_and_zero_weights():
    rnd = random.Random(12)
    T, d, I, E, k = 6, 4, 3, 3, 2
    x = _rand_mat(rnd, T, d)
    W = [(_rand_mat(rnd, I, d), _rand_mat(rnd, I, d), _rand_mat(rnd, d, I)) for _ in range(E)]
    idx = np.array([rnd.sample(range(E), k) for _ in range(T)], dtype=np.int32)
    counts, offsets, st, sa, inv = O.dispatch(idx, E)
    y = O.expert_ffn(np.array(x), st, offsets, np.array([w[0] for w in W]),
                     np.array([w[1] for w in W]), np.array([w[2] for w in W]))
    for r in range(T * k):
        e = int(np.searchsorted(offsets, r, side="right") - 1)
        want = _loop_ffn([x[st[r]]], *W[e])[0]
        assert np.allclose(y[r], want, rtol=1e-13, atol=1e-14)
    z = np.zeros((E, I, d))
    y0 = O.expert_ffn(np.array(x), st, offsets, z, z, np.zeros((E, d, I)))
    assert (y0 == 0).all()


# ---------------------------------------------------------------------------
# combine and whole layer
# ---------------------------------------------------------------------------

def test_combine_identity_experts_returns_scaled_input():
    rnd = np.random.default_rng(2)
    T, d, E, k = 30, 16, 32, 8
    x = rnd.normal(size=(T, d))
    u = rnd.normal(size=(T, E))
    idx, w = O.route(u, k=k, score="sigmoid", n_groups=4, topk_groups=2, scale=2.5)
    counts, offsets, st, sa, inv = O.dispatch(idx, E)
    y_perm = x[st]                       # every expert is the identity map
    out = O.combine(y_perm, inv, w)
    assert np.allclose(out, 2.5 * x, rtol=1e-14, atol=1e-14)
    sh = rnd.normal(size=(T, d))
    assert np.allclose(O.combine(y_perm, inv, w, sh), 2.5 * x + sh, rtol=1e-14, atol=1e-14)


def test_combine_matches_loops():
    rnd = random.Random(4)
    T, k, d = 5, 3, 4
    n = T * k
    perm = list(range(n))
    rnd.shuffle(perm)
    Y = _rand_mat(rnd, n, d)
    W = _rand_mat(rnd, T, k)
    out = O.combine(np.array(Y), np.array(perm), np.array(W))
    for t in range(T):
        for c in range(d):
            want = sum(W[t][j] * Y[perm[t * k + j]][c] for j in range(k))
            assert abs(out[t, c] - want) < 1e-14


def test_layer_single_expert_is_dense_swiglu():
    rnd = random.Random(21)
    T, d, I = 5, 4, 6
    x, wg, wu, wd = _rand_mat(rnd, T, d), _rand_mat(rnd, I, d), _rand_mat(rnd, I, d), _rand_mat(rnd, d, I)
    wr = _rand_mat(rnd, 1, d)
    cfg = dict(E=1, k=1, score="softmax", n_shared=0)
    r = O.layer(cfg, np.array(x), np.array(wr), None, np.array([wg]), np.array([wu]), np.array([wd]))
    assert np.allclose(r["out"], _loop_ffn(x, wg, wu, wd), rtol=1e-13, atol=1e-14)


def test_layer_k_equals_E_is_dense_softmax_mixture_plus_shared():
    rnd = random.Random(22)
    T, d, I, E = 4, 3, 5, 3
    x = _rand_mat(rnd, T, d)
    wr = _rand_mat(rnd, E, d)
    W = [(_rand_mat(rnd, I, d), _rand_mat(rnd, I, d), _rand_mat(rnd, d, I)) for _ in range(E)]
    S = (_rand_mat(rnd, I, d), _rand_mat(rnd, I, d), _rand_mat(rnd, d, I))
    cfg = dict(E=E, k=E, score="softmax", n_shared=1)
    r = O.layer(cfg, np.array(x), np.array(wr), None, np.array([w[0] for w in W]),
                np.array([w[1] for w in W]), np.array([w[2] for w in W]),
                np.array(S[0]), np.array(S[1]), np.array(S[2]))
    for t in range(T):
        u = [sum(x[t][c] * wr[e][c] for c in range(d)) for e in range(E)]
        m = max(u)
        z = [math.exp(v - m) for v in u]
        p = [v / sum(z) for v in z]
        ys = [_loop_ffn([x[t]], *W[e])[0] for e in range(E)]
        sh = _loop_ffn([x[t]], *S)[0]
        want = [sum(p[e] * ys[e][c] for e in range(E)) + sh[c] for c in range(d)]
        assert np.allclose(r["out"][t], want, rtol=1e-12, atol=1e-13)


def test_layer_rows_agrees_with_full_layer():
    rnd = np.random.default_rng(8)
    T, d, I, E, k = 24, 8, 6, 16, 4
    x = rnd.normal(size=(T, d))
    wr = rnd.normal(size=(E, d))
    wg, wu = rnd.normal(size=(E, I, d)), rnd.normal(size=(E, I, d))
    wd = rnd.normal(size=(E, d, I))
    s = [rnd.normal(size=(I, d)), rnd.normal(size=(I, d)), rnd.normal(size=(d, I))]
    cfg = dict(E=E, k=k, score="sigmoid", n_groups=4, topk_groups=2, scale=2.5, n_shared=1)
    full = O.layer(cfg, x, wr, np.zeros(E), wg, wu, wd, *s)
    rows = np.array([0, 5, 23, 7])
    part = O.layer_rows(x, rows, full["topk_idx"][rows], full["topk_w"][rows], wg, wu, wd, *s)
    assert np.allclose(part, full["out"][rows], rtol=1e-13, atol=1e-13)


def test_dsv3_shaped_routing_invariants():
    rnd = np.random.default_rng(0)
    T, E = 512, 256
    u = rnd.normal(scale=1.7, size=(T, E))
    bias = rnd.normal(scale=0.05, size=E)
    idx, w, det = O.route(u, k=8, score="sigmoid", bias=bias, n_groups=8, topk_groups=4,
                          scale=2.5, return_detail=True)
    check_routing(idx, w, E, scale=2.5)
    # every chosen expert lies in one of the chosen groups
    assert np.isin(idx // 32, det["chosen_groups"]).reshape(T, 8).all()
    counts, offsets, st, sa, inv = O.dispatch(idx, E)
    check_dispatch(idx, counts, offsets, st, inv, sa)


def test_max_rel_err_metric():
    want = np.array([1.0, -2.0, 0.0, 4.0])
    rms = math.sqrt((1 + 4 + 0 + 16) / 4)
    got = want + np.array([0.01, 0.0, 0.05, 0.0])
    assert max_rel_err(got, want) == pytest.approx(max(0.01 / rms, 0.05 / rms))


# ---------------------------------------------------------------------------
# token quantization (App. F pipeline: int8 codes, one scale per token)
# ---------------------------------------------------------------------------

def _bf16_bits(a):
    """float32 values that bf16 represents exactly -> their bf16 bit patterns."""
    b = np.asarray(a, dtype=np.float32).view(np.uint32)
    assert (b & 0xFFFF == 0).all(), "value not exact in bf16"
    return (b >> 16).astype(np.uint16)


def test_quantize_worked_examples():
    ex = json.load(open(os.path.join(GOLDEN, "quant_examples.json")))
    for name in ("Q1", "Q2", "Q3", "Q4"):
        e = ex[name]
        for x in (np.asarray([e["x"]], np.float32), _bf16_bits([e["x"]])):
            codes, scales = O.quantize_tokens(x)
            assert codes.dtype == np.int8 and scales.dtype == np.float32
            assert codes[0].tolist() == e["codes"], name
            assert float(scales[0]) == e["scale"], name


def test_quantize_invariants_and_error_bound():
    rng = np.random.default_rng(7)
    x = (rng.standard_normal((64, 300)) * rng.uniform(0.01, 50, (64, 1))).astype(np.float32)
    x[3] = 0.0
    codes, scales = O.quantize_tokens(x)
    assert np.abs(codes.astype(np.int32)).max() <= 127
    nz = scales > 0
    # the largest |x| of every non-zero row maps to +-127
    assert (np.abs(codes[nz].astype(np.int32)).max(axis=1) == 127).all()
    assert scales[3] == 0 and (codes[3] == 0).all()
    # scale is max|x|/127 to float32 rounding
    np.testing.assert_allclose(scales[nz], np.abs(x[nz]).max(axis=1) / 127.0, rtol=2 ** -23)
    # round to nearest: every element within half a step (plus float32 rounding)
    err = np.abs(O.dequantize_tokens(codes, scales) - x)
    assert (err <= scales[:, None] * (0.5 + 2 ** -20) + 1e-30).all()
    # a power-of-two rescaling of a row changes only its scale
    c2, s2 = O.quantize_tokens(x * np.float32(8.0))
    assert np.array_equal(c2, codes) and np.array_equal(s2, scales * np.float32(8.0))
    # per token: quantizing a subset of rows gives the same rows
    c3, s3 = O.quantize_tokens(x[10:20])
    assert np.array_equal(c3, codes[10:20]) and np.array_equal(s3, scales[10:20])


def test_quantize_rounding_is_half_even_not_half_away():
    # max |x| = 127 gives scale 1: ties at .5 go to the even integer
    x = np.asarray([[127.0, 0.5, 1.5, 2.5, -1.5, -126.5]], np.float32)
    codes, _ = O.quantize_tokens(x)
    assert codes[0].tolist() == [127, 0, 2, 2, -2, -126]


def test_quantize_bound_catches_planted_off_by_one():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((8, 64)).astype(np.float32)
    codes, scales = O.quantize_tokens(x)
    bad = codes.copy()
    frac = np.abs(x[2] / scales[2]) % 1
    r, c = 2, int(np.argmax(np.abs(frac - 0.5)))  # the element farthest from a rounding tie
    bad[r, c] += 1 if bad[r, c] < 127 else -1
    err = np.abs(O.dequantize_tokens(bad, scales) - x)
    assert (err > scales[:, None] * (0.5 + 2 ** -20)).any()


def test_quantized_layer_equals_plain_layer_on_exact_tokens():
    # tokens that are integers times max|x|/127 (a power of two) survive the
    # quantization exactly, so the quantized layer is the plain layer
    rng = np.random.default_rng(11)
    T, d, E, I = 20, 32, 4, 16
    x = (rng.integers(-127, 128, (T, d)).astype(np.float32) * np.float32(0.25))
    x[:, 0] = 127 * 0.25
    wr = rng.standard_normal((E, d)) * 0.1
    wg, wu = rng.standard_normal((E, I, d)) * 0.2, rng.standard_normal((E, I, d)) * 0.2
    wd = rng.standard_normal((E, d, I)) * 0.2
    cfg = dict(E=E, k=2, score="softmax", n_groups=1, topk_groups=1, renorm=True, scale=1.0, n_shared=0)
    a = O.layer(cfg, x, wr, None, wg, wu, wd)
    b = O.layer(dict(cfg, quant="int8"), x, wr, None, wg, wu, wd)
    assert np.array_equal(a["out"], b["out"])
    # and a non-exact token changes it, by no more than the quantization step allows
    x2 = x.copy()
    x2[5, 3] += np.float32(0.1)
    c = O.layer(dict(cfg, quant="int8"), x2, wr, None, wg, wu, wd)
    d_ = O.layer(cfg, x2, wr, None, wg, wu, wd)
    assert not np.array_equal(c["out"], d_["out"])
    assert max_rel_err(c["out"], d_["out"]) < 0.05


def test_layer_rows_quantized_agrees_with_full_layer():
    rng = np.random.default_rng(12)
    T, d, E, I = 24, 64, 8, 16
    x = rng.standard_normal((T, d)).astype(np.float32)
    wr = rng.standard_normal((E, d)) * 0.1
    wg, wu = rng.standard_normal((E, I, d)) * 0.2, rng.standard_normal((E, I, d)) * 0.2
    wd = rng.standard_normal((E, d, I)) * 0.2
    sg, su, sd = rng.standard_normal((I, d)) * 0.2, rng.standard_normal((I, d)) * 0.2, rng.standard_normal((d, I)) * 0.2
    cfg = dict(E=E, k=3, score="sigmoid", n_groups=4, topk_groups=2, renorm=True, scale=2.5, n_shared=1,
               quant="int8")
    bias = np.zeros(E)
    full = O.layer(cfg, x, wr, bias, wg, wu, wd, sg, su, sd)
    rows = np.array([0, 5, 23])
    part = O.layer_rows(x, rows, full["topk_idx"][rows], full["topk_w"][rows], wg, wu, wd, sg, su, sd, quant="int8")
    np.testing.assert_allclose(part, full["out"][rows], rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------------------
# expert parallelism, receive side
# ---------------------------------------------------------------------------

def test_ep_receive_plan_worked_examples():
    ex = json.load(open(os.path.join(GOLDEN, "ep_plan_examples.json")))
    s = O.dispatch(np.asarray(ex["self_topk"]), ex["E"])
    p = O.dispatch(np.asarray(ex["peer_topk"]), ex["E"])
    for name in ("P1", "P2"):
        e = ex[name]
        rt, off, se = O.ep_receive_plan(s[1], s[2], p[1], p[2], e["e_first"], e["e_count"])
        assert rt.tolist() == e["row_token"], name
        assert off.tolist() == e["offsets"], name
        assert se.tolist() == e["self_end"], name


def _ep_plan_brute(self_topk, peer_topk, e_first, e_count):
    """The receive plan by enumeration: for each local expert, scan the
    tokens of each rank in order and keep those that chose it."""
    rows, offsets, self_end = [], [0], []
    for e in range(e_first, e_first + e_count):
        mine = [t for t, r in enumerate(self_topk) if e in list(r)]
        theirs = [t for t, r in enumerate(peer_topk) if e in list(r)]
        rows += mine
        self_end.append(offsets[-1] + len(mine))
        rows += theirs
        offsets.append(offsets[-1] + len(mine) + len(theirs))
    return rows, offsets, self_end


@pytest.mark.parametrize("ratio", [1.0, 3.0, 5.0])
def test_ep_receive_plan_matches_enumeration_and_invariants(ratio):
    from paper_2603_02376_amd import inputs
    T, E, k = 40, 16, 3
    st = inputs.ep_topk(T, E, k, ratio, "self", seed=1)
    pt = inputs.ep_topk(T, E, k, ratio, "peer", seed=1)
    s, p = O.dispatch(st, E), O.dispatch(pt, E)
    for e_first, e_count in ((0, E // 2), (E // 2, E // 2), (3, 5)):
        rt, off, se = O.ep_receive_plan(s[1], s[2], p[1], p[2], e_first, e_count)
        rows, offsets, self_end = _ep_plan_brute(st, pt, e_first, e_count)
        assert rt.tolist() == rows and off.tolist() == offsets and se.tolist() == self_end
        # every local assignment of either rank appears exactly once
        local = lambda tk: sorted((t, int(e)) for t, r in enumerate(tk) for e in r if e_first <= e < e_first + e_count)
        got_self = sorted((int(rt[r]), e_first + e) for e in range(e_count) for r in range(off[e], se[e]))
        got_peer = sorted((int(rt[r]), e_first + e) for e in range(e_count) for r in range(se[e], off[e + 1]))
        assert got_self == local(st) and got_peer == local(pt)


def test_ep_topk_ratio_and_distinct_experts():
    from paper_2603_02376_amd import inputs
    T, E, k = 4096, 256, 8
    for r in inputs.EP_RATIOS:
        tk = inputs.ep_topk(T, E, k, r, "self")
        assert tk.dtype == np.int32 and tk.shape == (T, k)
        assert all(len(set(row)) == k for row in tk)
        assert tk.min() >= 0 and tk.max() < E
        frac = (tk < E // 2).mean()
        # binomial mean r/(r+1); 32768 draws: standard error < 0.003
        assert abs(frac - r / (r + 1)) < 0.015, (r, frac)
    assert not np.array_equal(inputs.ep_topk(64, E, k, 3, "self"), inputs.ep_topk(64, E, k, 3, "peer"))


def test_ep_receive_ffn_reduces_to_each_ranks_expert_ffn():
    # every received row is the single-GPU expert FFN of its token, whichever
    # rank it came from
    from paper_2603_02376_amd import inputs
    rng = np.random.default_rng(5)
    T, Tp, E, k, d, I = 12, 5, 8, 2, 16, 8   # the peer has fewer tokens than this GPU
    xs, xp = rng.standard_normal((T, d)), rng.standard_normal((Tp, d))
    wg, wu = rng.standard_normal((E, I, d)) * 0.3, rng.standard_normal((E, I, d)) * 0.3
    wd = rng.standard_normal((E, d, I)) * 0.3
    st, pt = inputs.ep_topk(T, E, k, 2.0, "self", 2), inputs.ep_topk(Tp, E, k, 2.0, "peer", 2)
    s, p = O.dispatch(st, E), O.dispatch(pt, E)
    ys = O.expert_ffn(xs, s[2], s[1], wg, wu, wd)
    yp = O.expert_ffn(xp, p[2], p[1], wg, wu, wd)
    e0, ne = E // 2, E // 2
    rt, off, se = O.ep_receive_plan(s[1], s[2], p[1], p[2], e0, ne)
    y = O.ep_receive_ffn(xs, xp, rt, off, se, wg[e0:], wu[e0:], wd[e0:])
    # (fp64 matrix products of differently batched rows may differ in the last bits)
    for e in range(ne):
        g = e0 + e
        np.testing.assert_allclose(y[off[e]:se[e]], ys[s[1][g]:s[1][g + 1]], rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(y[se[e]:off[e + 1]], yp[p[1][g]:p[1][g + 1]], rtol=1e-12, atol=1e-12)
    sub = [0, int(off[-1]) - 1, int(se[1])]
    np.testing.assert_allclose(O.ep_receive_ffn(xs, xp, rt, off, se, wg[e0:], wu[e0:], wd[e0:], rows=sub), y[sub],
                               rtol=1e-12, atol=1e-12)
    # a planted swap of the row sources (self rows read from the peer's tokens) is caught
    xs2 = xs.copy()
    xs2[:Tp] = xp
    bad = O.ep_receive_ffn(xs2, xp, rt, off, se, wg[e0:], wu[e0:], wd[e0:])
    assert not np.allclose(bad, y, rtol=1e-6)


# ---------------------------------------------------------------------------
# FP8 (OCP E4M3) token quantization
# ---------------------------------------------------------------------------

def test_fp8_worked_examples():
    ex = json.load(open(os.path.join(GOLDEN, "fp8_examples.json")))
    for name in ("F1", "F2", "F3"):
        e = ex[name]
        for x in (np.asarray([e["x"]], np.float32), _bf16_bits([e["x"]])):
            codes, scales = O.quantize_tokens_fp8(x)
            assert codes.dtype == np.uint8 and scales.dtype == np.float32
            assert codes[0].tolist() == e["codes"], (name, codes[0].tolist())
            assert float(scales[0]) == e["scale"], name


def test_e4m3_code_table_properties():
    v = O.e4m3_values()
    nan = np.isnan(v)
    assert nan.sum() == 2 and nan[0x7F] and nan[0xFF]
    pos = v[:0x7F]
    assert pos[0] == 0.0 and pos[0x7E] == 448.0 and v[0x38] == 1.0
    assert (np.diff(pos) > 0).all()                       # codes order the values
    np.testing.assert_array_equal(v[0x80:0xFF], -pos)    # the sign bit only negates
    assert np.signbit(v[0x80])
    # subnormals: 7 equal steps of 2^-9 up to the smallest normal 2^-6
    np.testing.assert_array_equal(pos[:9], np.arange(9) * 2.0 ** -9)
    # every binade [2^e, 2^(e+1)) of the normals holds 8 values 2^(e-3) apart (the top
    # one 7: its eighth code is NaN)
    for e in range(-6, 9):
        b = pos[(pos >= 2.0 ** e) & (pos < 2.0 ** (e + 1))]
        assert b.size == (7 if e == 8 else 8)
        np.testing.assert_allclose(np.diff(b), 2.0 ** (e - 3))


def test_fp8_quantize_invariants():
    rng = np.random.default_rng(17)
    x = (rng.standard_normal((48, 200)) * rng.uniform(0.01, 40, (48, 1))).astype(np.float32)
    x[5] = 0.0
    codes, scales = O.quantize_tokens_fp8(x)
    v = O.e4m3_values()
    assert not np.isnan(v[codes]).any()
    nz = scales > 0
    # the largest |x| of every non-zero row maps to +-448
    assert (np.abs(v[codes[nz]]).max(axis=1) == 448.0).all()
    assert scales[5] == 0 and (codes[5] == 0).all()
    np.testing.assert_allclose(scales[nz], np.abs(x[nz]).max(axis=1) / 448.0, rtol=2 ** -23)
    # round to nearest: within half a step of the grid at that magnitude (2^-4 relative for
    # normals, 2^-10 absolute below the smallest normal), plus float32 rounding of the quotient
    q = x[nz] / scales[nz, None]
    err = np.abs(v[codes[nz]] - q)
    step = np.where(np.abs(q) >= 2.0 ** -6, 2.0 ** (np.floor(np.log2(np.maximum(np.abs(q), 2.0 ** -6))) - 3), 2.0 ** -9)
    assert (err <= step / 2 * (1 + 2 ** -20) + 1e-30).all()
    # quantizing the grid values themselves changes nothing
    c2, s2 = O.quantize_tokens_fp8(O.dequantize_tokens_fp8(codes, scales).astype(np.float32))
    assert np.array_equal(c2[nz], codes[nz])
    # per token: a subset of rows quantizes the same
    c3, s3 = O.quantize_tokens_fp8(x[10:20])
    assert np.array_equal(c3, codes[10:20]) and np.array_equal(s3, scales[10:20])


def test_fp8_layer_equals_plain_layer_on_exact_tokens():
    # tokens that are E4M3 values times a power of two, with max |x| = 448 times
    # it, survive the quantization exactly, so the quantized layer is the plain one
    rng = np.random.default_rng(13)
    T, d, E, I = 16, 32, 4, 16
    grid = O.e4m3_values()[:0x7F]
    x = (rng.choice(grid, (T, d)) * rng.choice([-1.0, 1.0], (T, d)) * 0.125).astype(np.float32)
    x[:, 0] = 448 * 0.125
    wr = rng.standard_normal((E, d)) * 0.1
    wg, wu = rng.standard_normal((E, I, d)) * 0.2, rng.standard_normal((E, I, d)) * 0.2
    wd = rng.standard_normal((E, d, I)) * 0.2
    cfg = dict(E=E, k=2, score="softmax", n_groups=1, topk_groups=1, renorm=True, scale=1.0, n_shared=0)
    a = O.layer(cfg, x, wr, None, wg, wu, wd)
    b = O.layer(dict(cfg, quant="fp8"), x, wr, None, wg, wu, wd)
    assert np.array_equal(a["out"], b["out"])
    x2 = x.copy()
    x2[3, 5] = np.float32(1.03)   # between two grid values
    assert not np.array_equal(O.layer(dict(cfg, quant="fp8"), x2, wr, None, wg, wu, wd)["out"],
                              O.layer(cfg, x2, wr, None, wg, wu, wd)["out"])
