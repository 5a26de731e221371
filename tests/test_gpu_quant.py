"""GPU parity of the quantized token paths (App. F pipeline: quantize the
tokens before the dispatch exchange, dequantize them before GEMM1; int8, and
FP8 (OCP E4M3) as Table 5 names), through the C ABI.

moe_quantize: codes and scales bit-exact against the oracle (codes decided in
fp32 on both sides). moe_expert_ffn_q8 and moe_layer with quantized tokens:
the oracle's FFN on the dequantized tokens, within the bf16 tolerance;
integer results of the layer bit-exact.
"""
import numpy as np
import pytest
import torch

from oracle import moe_oracle as O
from oracle.checks import max_rel_err
from paper_2603_02376_amd import inputs, moe
from tests import gpu_util as G
from tests.gpu_util import BF16_TOL, host, log

pytestmark = pytest.mark.gpu


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _bf16(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16).cuda()


def _oracle_quant(mode):
    return (O.quantize_tokens, O.dequantize_tokens) if mode == "int8" else (O.quantize_tokens_fp8,
                                                                            O.dequantize_tokens_fp8)


def _codes_buf(mode, T, d):
    return torch.empty((T, d), dtype=torch.int8 if mode == "int8" else torch.uint8, device="cuda")


@pytest.mark.parametrize("mode", ["int8", "fp8"])
@pytest.mark.parametrize("T,d", [(1, 64), (37, 256), (300, 7168), (4096, 7168), (5, 8192), (7, 8256)])
def test_quantize_bit_exact(T, d, mode):
    log("quantize", mode, T, d)
    rng = np.random.default_rng(T + d)
    x = (rng.standard_normal((T, d)) * rng.uniform(0.05, 20, (T, 1))).astype(np.float32)
    if T > 2:
        x[1] = 0.0                                    # zero row: scale 0, codes 0
        if mode == "int8":
            # a row of exact halves: max |x| = 127 * 2^-3, scale 2^-3, codes = x * 8 with .5 ties
            x[2] = (rng.integers(-254, 255, d) * 0.0625).astype(np.float32)
            x[2, 0] = 127 * 0.125
        else:
            # a row of E4M3 grid values and midpoints between neighbours (ties), max |x| = 448:
            # scale 1, every tie rule and the subnormals exercised
            g = O.e4m3_values()[:0x7F]
            pts = np.concatenate([g, (g[1:] + g[:-1]) / 2])
            x[2] = (rng.choice(pts, d) * rng.choice([-1.0, 1.0], d)).astype(np.float32)
            x[2, 0] = 448.0
    xb = _bf16(x)
    cfg = moe.MoeConfig(d=d, E=8, k=2, I=128, dtype="bf16", weight_layout="packed", token_quant=mode)
    codes = _codes_buf(mode, T, d)
    scales = torch.empty(T, dtype=torch.float32, device="cuda")
    moe.moe_quantize(cfg, T, xb, codes, scales)
    torch.cuda.synchronize()
    want_c, want_s = _oracle_quant(mode)[0](inputs.oracle_view(xb))
    assert np.array_equal(host(scales), want_s)
    got_c = host(codes)
    if not np.array_equal(got_c, want_c):
        bad = np.argwhere(got_c != want_c)
        raise AssertionError(f"{len(bad)} codes differ, first at {bad[:3].tolist()}")


QCASES = [
    # T, d, E, k, I, hot
    (300, 256, 16, 4, 128, None),    # ~75 rows per expert
    (200, 512, 8, 4, 256, 0),        # a hot expert: passes of 192 + 8 rows
    (1, 256, 8, 2, 128, None),
    (700, 256, 4, 2, 128, None),     # 350 rows per expert
    (513, 768, 32, 8, 384, None),    # ragged rows, several column tiles
]


def _topk(T, E, k, rng, hot):
    idx = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    if hot is not None:
        for t in range(T):
            if hot not in idx[t]:
                idx[t, 0] = hot
    return idx


@pytest.mark.parametrize("mode", ["int8", "fp8"])
@pytest.mark.parametrize("case", QCASES, ids=lambda c: "T{}_d{}_E{}_k{}_I{}".format(*c[:5]))
def test_expert_ffn_q8(case, mode):
    T, d, E, k, I, hot = case
    log("expert_ffn_q8", mode, case)
    p = dict(T=T, d=d, E=E, k=k, I=I, dtype="bf16", n_shared=0, bias="none")
    t = inputs.make_inputs(p, 0, "cuda")
    idx = _topk(T, E, k, np.random.default_rng(T), hot)
    counts, offsets, st, sa, inv = O.dispatch(idx, E)
    cfg = moe.MoeConfig(d=d, E=E, k=k, I=I, dtype="bf16", weight_layout="packed", token_quant=mode)
    gu, dn = moe.pack_weights(cfg, t["w_gate"], t["w_up"], t["w_down"])
    codes = _codes_buf(mode, T, d)
    scales = torch.empty(T, dtype=torch.float32, device="cuda")
    moe.moe_quantize(cfg, T, t["x"], codes, scales)
    ws = moe.alloc_workspace(cfg, T)
    y = torch.full((T * k, d), float("nan"), dtype=torch.bfloat16, device="cuda")
    moe.moe_expert_ffn_q8(cfg, T, codes, scales, _dev(st), _dev(offsets), gu, dn, y, ws)
    torch.cuda.synchronize()
    quant, dequant = _oracle_quant(mode)
    xq = dequant(host(codes), host(scales))
    want = O.expert_ffn(xq, st, offsets, inputs.ExpertView(t["w_gate"]), inputs.ExpertView(t["w_up"]),
                        inputs.ExpertView(t["w_down"]))
    got = host(y.float())
    assert np.isfinite(got).all(), "rows left unwritten"
    err = max_rel_err(got, want)
    log("  max_rel_err", err)
    assert err <= BF16_TOL
    # the codes fed to the GEMM are the oracle's codes
    wc, ws_ = quant(inputs.oracle_view(t["x"]))
    assert np.array_equal(host(codes), wc) and np.array_equal(host(scales), ws_)


def test_expert_ffn_q8_rejects_unpacked_and_f32():
    cfg = moe.MoeConfig(d=256, E=8, k=2, I=128, dtype="bf16")  # row-major weights
    z8 = torch.zeros((4, 256), dtype=torch.int8, device="cuda")
    zs = torch.zeros(4, dtype=torch.float32, device="cuda")
    zi = torch.zeros(8, dtype=torch.int32, device="cuda")
    zw = torch.zeros(8 * 128 * 256 * 2, dtype=torch.bfloat16, device="cuda")
    y = torch.zeros((8, 256), dtype=torch.bfloat16, device="cuda")
    ws = moe.alloc_workspace(cfg, 4)
    offsets = torch.zeros(9, dtype=torch.int32, device="cuda")
    with pytest.raises(moe.MoeError) as e:
        moe.moe_expert_ffn_q8(cfg, 4, z8, zs, zi, offsets, zw, zw, y, ws)
    assert e.value.status == -2
    for mode in ("int8", "fp8"):   # quantized tokens in the layer need packed weights too
        with pytest.raises(moe.MoeError) as e:
            moe.alloc_workspace(moe.MoeConfig(d=256, E=8, k=2, I=128, dtype="bf16", token_quant=mode), 4)
        assert e.value.status in (-1, -2)


LAYER_CASES = {
    "dsv3_like": dict(T=300, d=512, E=32, k=4, n_groups=4, topk_groups=2, I=256, n_shared=1, I_shared=256,
                      score="sigmoid", renorm=True, scale=2.5, dtype="bf16", bias="zipf"),
    "mixtral_like": dict(T=257, d=256, E=8, k=2, n_groups=1, topk_groups=1, I=384, n_shared=0, I_shared=0,
                         score="softmax", renorm=True, scale=1.0, dtype="bf16", bias="none"),
}


@pytest.mark.parametrize("mode", ["int8", "fp8"])
@pytest.mark.parametrize("name", list(LAYER_CASES))
def test_layer_quantized_tokens(name, mode):
    p = dict(LAYER_CASES[name], weight_layout="packed", token_quant=mode)
    log("layer quantized tokens", mode, name)
    t = G.device_inputs(p, seed=3)
    r = G.run_layer(p, t)
    G.check_logits(p, t, r)
    routing = G.check_routing_and_dispatch_exact(p, t, r)
    x = inputs.oracle_view(t["x"])
    quant, dequant = _oracle_quant(mode)
    xq = dequant(*quant(x))
    y = O.expert_ffn(xq, host(r["sorted_token"]), host(r["offsets"]), inputs.ExpertView(t["w_gate"]),
                     inputs.ExpertView(t["w_up"]), inputs.ExpertView(t["w_down"]))
    sh = None
    if p["n_shared"]:
        sh = O.swiglu_ffn(x, inputs.oracle_view(t["ws_gate"]), inputs.oracle_view(t["ws_up"]),
                          inputs.oracle_view(t["ws_down"]))
        assert max_rel_err(host(r["shared_out"].float()), sh) <= BF16_TOL
    out = O.combine(y, host(r["inv_perm"]), routing["topk_w"], sh)
    assert max_rel_err(host(r["y_perm"].float()), y) <= BF16_TOL
    err = max_rel_err(host(r["out"].float()), out)
    log("  out max_rel_err", err)
    assert err <= BF16_TOL
    # one stream or two: same bits
    r2 = G.run_layer(p, t, s_aux=None)
    assert torch.equal(r2["out"], r["out"])


@pytest.mark.parametrize("mode", ["int8", "fp8"])
def test_layer_quantized_tokens_full_size_sampled(mode):
    p = dict(inputs.preset("dsv3"), weight_layout="packed", token_quant=mode)
    log("full-size layer, quantized tokens", mode)
    t = G.device_inputs(p, seed=0, cache_weights=True)
    r = G.run_layer(p, t)
    G.check_logits(p, t, r)
    routing = G.check_routing_and_dispatch_exact(p, t, r)
    rng = np.random.default_rng(0)
    rows = np.unique(np.concatenate([[0, p["T"] - 1], rng.choice(p["T"], 8, replace=False)]))
    want = O.layer_rows(inputs.oracle_view(t["x"]), rows, routing["topk_idx"][rows], routing["topk_w"][rows],
                        inputs.ExpertView(t["w_gate"]), inputs.ExpertView(t["w_up"]), inputs.ExpertView(t["w_down"]),
                        *(inputs.oracle_view(t[n]) for n in ("ws_gate", "ws_up", "ws_down")), quant=mode)
    err = max_rel_err(host(r["out"].float())[rows], want)
    log("  sampled out max_rel_err", err)
    assert err <= BF16_TOL
    # whole segments of the first and the busiest expert (GEMM1 on the codes at
    # K = 7168, every column tile), and the shared expert over every token (its
    # GEMM1 runs on its own, its GEMM2 inside the routed GEMM2)
    x = inputs.oracle_view(t["x"])
    st, off, counts = host(r["sorted_token"]), host(r["offsets"]), host(r["counts"])
    G.check_expert_segments(x, st, off, inputs.ExpertView(t["w_gate"]), inputs.ExpertView(t["w_up"]),
                            inputs.ExpertView(t["w_down"]), [0, int(np.argmax(counts))], {mode: r["y_perm"]},
                            BF16_TOL, quant=mode)
    want_sh = O.swiglu_ffn(x, *(inputs.oracle_view(t[n]) for n in ("ws_gate", "ws_up", "ws_down")))
    err = max_rel_err(host(r["shared_out"].float()), want_sh)
    log("  shared_out (all tokens) max_rel_err", err)
    assert err <= BF16_TOL
    G.release_cached_weights()
