"""Helpers for the GPU parity tests (not a test module).

They run the HIP path through the C ABI (via the ctypes binding) and hand the
same input bits to the CPU oracle. Nothing here computes any part of the
method: the only arithmetic is in the library and in the oracle.
"""
from __future__ import annotations

import functools
import sys

import numpy as np
import torch

from oracle import moe_oracle as O
from oracle.checks import check_dispatch, check_routing, max_rel_err
from paper_2603_02376_amd import inputs, moe

BF16_TOL = 2e-2
F32_TOL = 1e-5
LOGIT_TOL = 1e-5
WEIGHT_TOL = 1e-6
NEAR_TIE = 1e-5


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def moe_cfg(p: dict) -> moe.MoeConfig:
    return moe.MoeConfig(d=p["d"], E=p["E"], k=p["k"], I=p["I"], n_groups=p.get("n_groups", 1),
                         topk_groups=p.get("topk_groups", 1), n_shared=p.get("n_shared", 0),
                         I_shared=p.get("I_shared", 0), score=p["score"], renorm=p.get("renorm", True),
                         scale=p.get("scale", 1.0), dtype=p["dtype"], weight_layout=p.get("weight_layout", "rowmajor"),
                         token_quant=p.get("token_quant", "none"))


def oracle_cfg(p: dict) -> dict:
    return dict(E=p["E"], k=p["k"], score=p["score"], n_groups=p.get("n_groups", 1),
                topk_groups=p.get("topk_groups", 1), renorm=p.get("renorm", True),
                scale=p.get("scale", 1.0), n_shared=p.get("n_shared", 0))


def route_kwargs(p: dict) -> dict:
    c = oracle_cfg(p)
    c.pop("E")
    c.pop("n_shared")
    return c


def tol(p: dict) -> float:
    return BF16_TOL if p["dtype"] == "bf16" else F32_TOL


@functools.lru_cache(maxsize=1)
def _weights_cached(key):
    d, E, I, n_shared, I_shared, dtype, seed = key
    p = dict(d=d, E=E, I=I, n_shared=n_shared, I_shared=I_shared, dtype=dtype, T=1, bias="none")
    t = inputs.make_inputs(p, seed, "cuda")
    return {k: v for k, v in t.items() if k not in ("x", "w_router", "bias")}


def device_inputs(p: dict, seed: int = 0, cache_weights: bool = False) -> dict:
    """Inputs on cuda:0; the large expert weights optionally shared between presets."""
    if not cache_weights:
        return inputs.make_inputs(p, seed, "cuda")
    key = (p["d"], p["E"], p["I"], p.get("n_shared", 0), p.get("I_shared", 0), p["dtype"], seed)
    w = _weights_cached(key)
    dt = torch.bfloat16 if p["dtype"] == "bf16" else torch.float32
    x, wr, b = inputs.host_activations(p, seed)
    out = dict(w)
    out["x"] = torch.from_numpy(x).to(device="cuda", dtype=dt)
    out["w_router"] = torch.from_numpy(wr).to(device="cuda", dtype=dt)
    out["bias"] = None if b is None else torch.from_numpy(b).cuda()
    return out


def release_cached_weights():
    _weights_cached.cache_clear()
    torch.cuda.empty_cache()


def run_layer(p: dict, t: dict, s_main=None, s_aux="new", with_debug=True) -> dict:
    """Run moe_layer; returns the output and every intermediate (device tensors)."""
    cfg = moe_cfg(p)
    T, k, E, d = p["T"], p["k"], p["E"], p["d"]
    dev = "cuda"
    dt = cfg.torch_dtype
    ws = moe.alloc_workspace(cfg, T)
    # outputs start as NaN, so a row the kernels never write fails every check
    nan = float("nan")
    out = torch.full((T, d), nan, dtype=dt, device=dev)
    dbg = None
    if with_debug:
        dbg = dict(logits=torch.empty((T, E), dtype=torch.float32, device=dev),
                   topk_idx=torch.empty((T, k), dtype=torch.int32, device=dev),
                   topk_w=torch.empty((T, k), dtype=torch.float32, device=dev),
                   counts=torch.empty(E, dtype=torch.int32, device=dev),
                   offsets=torch.empty(E + 1, dtype=torch.int32, device=dev),
                   sorted_token=torch.empty(T * k, dtype=torch.int32, device=dev),
                   sorted_assign=torch.empty(T * k, dtype=torch.int32, device=dev),
                   inv_perm=torch.empty(T * k, dtype=torch.int32, device=dev),
                   y_perm=torch.full((T * k, d), nan, dtype=dt, device=dev))
        if p.get("n_shared", 0):
            dbg["shared_out"] = torch.full((T, d), nan, dtype=dt, device=dev)
    if s_aux == "new":
        s_aux = torch.cuda.Stream()
    wg, wu, wd = t["w_gate"], t["w_up"], t["w_down"]
    sg, su, sd = t.get("ws_gate"), t.get("ws_up"), t.get("ws_down")
    if cfg.packed:
        wg, wd = moe.pack_weights(cfg, wg, wu, wd)
        wu = None
        if p.get("n_shared", 0):
            sg, sd = moe.pack_shared_weights(cfg, sg, su, sd)
            su = None
    moe.moe_layer(cfg, T, t["x"], t["w_router"], t["bias"], wg, wu, wd,
                  sg, su, sd, out, ws, s_main=s_main, s_aux=s_aux, dbg=dbg)
    torch.cuda.synchronize()
    res = dict(out=out)
    if dbg:
        res.update(dbg)
    return res


def host(t):
    return None if t is None else t.detach().cpu().numpy()


def check_routing_and_dispatch_exact(p: dict, t: dict, r: dict) -> dict:
    """Oracle re-routes from the GPU's fp32 logits: indices, counts, offsets and
    permutation must match bit for bit; weights to WEIGHT_TOL."""
    logits = host(r["logits"])
    bias = None if p["score"] == "softmax" else inputs.oracle_view(t["bias"])
    idx_o, w_o = O.route(logits, bias=bias, **route_kwargs(p))
    idx_g = host(r["topk_idx"])
    assert np.array_equal(idx_g, idx_o), f"routing differs on {int((idx_g != idx_o).any(axis=1).sum())} tokens"
    w_g = host(r["topk_w"])
    werr = float(np.abs(w_g - w_o).max()) if w_o.size else 0.0
    assert werr <= WEIGHT_TOL * max(1.0, p.get("scale", 1.0)), f"weights differ by {werr}"
    check_routing(idx_g, w_g, p["E"], scale=p.get("scale", 1.0), renorm=p.get("renorm", True), atol=2e-6)
    want = O.dispatch(idx_o, p["E"])
    names = ("counts", "offsets", "sorted_token", "sorted_assign", "inv_perm")
    for n, wv in zip(names, want):
        gv = host(r[n])
        assert np.array_equal(gv, wv), f"{n} differs"
    check_dispatch(idx_g, host(r["counts"]), host(r["offsets"]), host(r["sorted_token"]),
                   host(r["inv_perm"]), host(r["sorted_assign"]))
    return dict(topk_idx=idx_o, topk_w=w_o, weight_err=werr)


def check_logits(p: dict, t: dict, r: dict, rows=None) -> float:
    x = inputs.oracle_view(t["x"])
    wr = inputs.oracle_view(t["w_router"])
    if rows is not None:
        x = x[rows]
    want = O.gate_logits(x, wr)
    got = host(r["logits"]) if rows is None else host(r["logits"])[rows]
    rms = float(np.sqrt(np.mean(want * want))) if want.size else 1.0
    err = float(np.abs(got - want).max() / rms) if want.size else 0.0
    assert err <= LOGIT_TOL, f"logits max|d|/rms = {err}"
    return err


def near_tie_report(p: dict, t: dict, r: dict, rows=None) -> int:
    """Route from the oracle's own fp64 logits; a token whose selection differs
    from the GPU's is accepted only if the oracle's selection margin is below
    NEAR_TIE. Returns how many tokens differ."""
    x = inputs.oracle_view(t["x"])
    if rows is not None:
        x = x[rows]
    logits = O.gate_logits(x, inputs.oracle_view(t["w_router"]))
    bias = None if p["score"] == "softmax" else inputs.oracle_view(t["bias"])
    idx, _, det = O.route(logits, bias=bias, return_detail=True, **route_kwargs(p))
    g = host(r["topk_idx"]) if rows is None else host(r["topk_idx"])[rows]
    diff = np.nonzero((np.sort(idx, axis=1) != np.sort(g, axis=1)).any(axis=1))[0]
    if diff.size:
        assert (det["margin"][diff] < NEAR_TIE).all(), \
            f"tokens {diff[:5]} differ from the fp64 routing without a near tie"
    return int(diff.size)


def check_expert_segments(x, st, off, wg, wu, wd, experts, ys, tol, quant=None) -> float:
    """Every row of the listed experts' segments of y_perm against the oracle's
    SwiGLU FFN of that expert on the same gathered tokens (whole segments, so
    every pass, column tile and K step of those experts is covered).
    x: the oracle view of the tokens; st, off: host sorted_token and offsets;
    wg, wu, wd: per-expert accessors; experts: expert ids; ys: {label: y_perm
    device tensor} (each compared with the same oracle rows). quant:
    "int8"/"fp8" when the experts saw quantized tokens."""
    worst = 0.0
    for e in experts:
        lo, hi = int(off[e]), int(off[e + 1])
        if hi == lo:
            continue
        rows = np.asarray(x)[st[lo:hi]]
        if quant == "int8":
            rows = O.dequantize_tokens(*O.quantize_tokens(rows))
        elif quant == "fp8":
            rows = O.dequantize_tokens_fp8(*O.quantize_tokens_fp8(rows))
        want = O.swiglu_ffn(rows, wg[e], wu[e], wd[e])
        for label, y in ys.items():
            got = host(y[lo:hi].float())
            assert np.isfinite(got).all(), f"{label} expert {e}: rows left unwritten"
            err = max_rel_err(got, want)
            log(f"  {label} expert {e}: {hi - lo} rows, max_rel_err {err:.3e}")
            assert err <= tol, f"{label} expert {e} ({hi - lo} rows): max_rel_err {err}"
            worst = max(worst, err)
    return worst
