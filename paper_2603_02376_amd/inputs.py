"""Seeded synthetic inputs and the workload presets.

This module holds no arithmetic of the MoE method: it only names the workload
shapes and draws random tensors. It is the one piece both the HIP path's
tests/benchmark and the CPU oracle's callers share.

Presets (one GPU's share of the layer; tokens N(0,1), router N(0, 0.02),
expert weights N(0, 1/sqrt(fan_in)), seed 0):

* ``tiny``        fp32: T=64, d=128, E=8, top-2 softmax renormalised, I=256.
* ``mixtral``     bf16: T=4096, d=4096, E=8, top-2 softmax renormalised, I=14336.
* ``dsv3``        bf16: T=4096, d=7168, 256 experts in 8 groups, sigmoid
                  scores + per-expert bias (0), top-4 groups then top-8
                  experts, weights normalised and scaled by 2.5, I=2048, one
                  shared expert with I=2048 (the DeepSeek-V3 layer whose
                  GEMM1 7168x4096 and GEMM2 2048x7168 the paper runs, App. M).
* ``dsv3_skew``   as ``dsv3`` with a Zipf(1.2)-shaped per-expert bias over a
                  seeded random expert order, so a few experts receive ~10x the
                  mean load and some receive none (the single-GPU stand-in for
                  the paper's 2:1-5:1 routing imbalance, §4 Workloads).
* ``dsv3_decode`` as ``dsv3`` with T=128.

Expert parallelism over two GPUs (the paper's MoE evaluation, §4 and App. M:
two ranks, 4096 tokens each, routing imbalance ratios 2:1 to 5:1): the 256
experts split into two halves, this GPU owning the first. :func:`ep_topk`
draws each rank's top-k directly (the routing is an input here): each of a
token's k experts lies in the first half with probability r/(r+1), so that
half receives r/(r+1) of all assignments; the experts are drawn uniformly
without replacement within each half. :func:`ep_peer_tokens` draws the peer
rank's tokens.

Random streams: host tensors use ``numpy.random.Generator(PCG64(SeedSequence(
[seed, tensor_id, expert])))``, draws in float32; the multi-GB expert
weights are drawn on the target device with ``torch.randn`` from a generator
seeded with ``seed * 1000 + tensor_id`` (deterministic per device type).
bf16 tensors are the round-to-nearest-even cast of those float32 draws.
Tensor ids: x 0, router 1, expert gate 3, up 4, down 5, shared gate 6, up 7,
down 8, Zipf expert order 9, expert-parallel top-k of this rank 10 and of
the peer 11, peer tokens 12.
"""
from __future__ import annotations

import math

import numpy as np
import torch

_DSV3 = dict(T=4096, d=7168, E=256, k=8, n_groups=8, topk_groups=4, I=2048, n_shared=1, I_shared=2048,
             score="sigmoid", renorm=True, scale=2.5, dtype="bf16", bias="zero")

PRESETS = {
    "tiny": dict(T=64, d=128, E=8, k=2, n_groups=1, topk_groups=1, I=256, n_shared=0, I_shared=0,
                 score="softmax", renorm=True, scale=1.0, dtype="f32", bias="none"),
    "mixtral": dict(T=4096, d=4096, E=8, k=2, n_groups=1, topk_groups=1, I=14336, n_shared=0, I_shared=0,
                    score="softmax", renorm=True, scale=1.0, dtype="bf16", bias="none"),
    "dsv3": dict(_DSV3),
    "dsv3_skew": dict(_DSV3, bias="zipf"),
    "dsv3_decode": dict(_DSV3, T=128),
}

# Zipf-shaped bias b_e = ZIPF_BETA * ln(E * p_{r(e)}), p_r proportional to
# r^-ZIPF_ALPHA, r(e) the 1-based rank of expert e in a seeded random order.
# ZIPF_BETA is fixed by tests/golden/make_zipf_beta.py (bisection on the
# oracle's routing of the dsv3 inputs so that the busiest expert receives
# ~10x the mean load) and recorded in tests/golden/zipf_beta.json.
ZIPF_ALPHA = 1.2
ZIPF_BETA = 0.050971
ZIPF_TARGET_MAX_OVER_MEAN = 10.0

TENSOR_IDS = dict(x=0, w_router=1, bias=2, w_gate=3, w_up=4, w_down=5, ws_gate=6, ws_up=7, ws_down=8, zipf_order=9,
                  ep_topk_self=10, ep_topk_peer=11, x_peer=12)
EP_RATIOS = (2, 3, 4, 5)  # routing imbalance ratios r:1 of the paper's MoE evaluation


def preset(name: str, **overrides) -> dict:
    cfg = dict(PRESETS[name])
    cfg.update(overrides)
    cfg["name"] = name
    return cfg


def host_rng(seed: int, tensor: str, expert: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, TENSOR_IDS[tensor], expert])))


def zipf_bias(E: int, seed: int = 0, alpha: float = ZIPF_ALPHA, beta: float | None = None) -> np.ndarray:
    """Per-expert bias with a Zipf-shaped popularity over a seeded expert order."""
    beta = ZIPF_BETA if beta is None else beta
    order = host_rng(seed, "zipf_order").permutation(E)
    rank = np.empty(E, dtype=np.int64)
    rank[order] = np.arange(1, E + 1)
    p = rank.astype(np.float64) ** (-alpha)
    p /= p.sum()
    return (beta * np.log(E * p)).astype(np.float32)


def ep_topk(T: int, E: int, k: int, ratio: float, side: str = "self", seed: int = 0) -> np.ndarray:
    """int32 [T, k]: every token's k distinct experts, each in [0, E/2) with
    probability ratio/(ratio+1) (binomial count per token, capped by the half's
    size), uniform without replacement within each half; slots in a random
    order. side: "self" or "peer" (independent streams)."""
    if E % 2 or k > E // 2:
        raise ValueError("need an even E and k <= E/2")
    rng = host_rng(seed, "ep_topk_self" if side == "self" else "ep_topk_peer", int(round(ratio * 1000)))
    half = E // 2
    p = ratio / (ratio + 1.0)
    n0 = np.minimum(rng.binomial(k, p, size=T), half)
    out = np.empty((T, k), dtype=np.int32)
    for t in range(T):
        a = rng.choice(half, size=int(n0[t]), replace=False)
        b = half + rng.choice(half, size=k - int(n0[t]), replace=False)
        out[t] = rng.permutation(np.concatenate([a, b]))
    return out


def ep_peer_tokens(T: int, d: int, seed: int = 0) -> np.ndarray:
    """float32 [T, d] N(0, 1): the peer rank's tokens."""
    return host_rng(seed, "x_peer").standard_normal((T, d), dtype=np.float32)


def host_activations(cfg: dict, seed: int = 0):
    """x [T, d], router [E, d] and bias [E] (or None) as float32 numpy arrays."""
    T, d, E = cfg["T"], cfg["d"], cfg["E"]
    x = host_rng(seed, "x").standard_normal((T, d), dtype=np.float32)
    w_router = host_rng(seed, "w_router").standard_normal((E, d), dtype=np.float32) * np.float32(0.02)
    if cfg.get("bias") == "zipf":
        bias = zipf_bias(E, seed)
    elif cfg.get("bias") == "zero":
        bias = np.zeros(E, dtype=np.float32)
    else:
        bias = None
    return x, w_router, bias


def _device_weights(shape, std, seed, tensor, device, dtype):
    g = torch.Generator(device=device)
    g.manual_seed(seed * 1000 + TENSOR_IDS[tensor])
    out = torch.empty(shape, dtype=dtype, device=device)
    # draw one expert at a time so the float32 staging buffer stays small
    flat = out.view(-1, *shape[-2:]) if len(shape) == 3 else out.view(1, *shape)
    for e in range(flat.shape[0]):
        w = torch.randn(shape[-2:], generator=g, device=device, dtype=torch.float32)
        w.mul_(std)
        flat[e].copy_(w)
    return out


def make_inputs(cfg: dict, seed: int = 0, device="cpu") -> dict:
    """All layer inputs as torch tensors on ``device`` in the preset's dtype.

    Keys: x, w_router, bias (fp32 or None), w_gate, w_up [E, I, d], w_down
    [E, d, I], and ws_gate, ws_up [I_s, d], ws_down [d, I_s] (or None).
    """
    dt = torch.bfloat16 if cfg["dtype"] == "bf16" else torch.float32
    x, w_router, bias = host_activations(cfg, seed)
    out = dict(
        x=torch.from_numpy(x).to(device=device, dtype=dt),
        w_router=torch.from_numpy(w_router).to(device=device, dtype=dt),
        bias=None if bias is None else torch.from_numpy(bias).to(device),
    )
    E, I, d = cfg["E"], cfg["I"], cfg["d"]
    out["w_gate"] = _device_weights((E, I, d), 1 / math.sqrt(d), seed, "w_gate", device, dt)
    out["w_up"] = _device_weights((E, I, d), 1 / math.sqrt(d), seed, "w_up", device, dt)
    out["w_down"] = _device_weights((E, d, I), 1 / math.sqrt(I), seed, "w_down", device, dt)
    if cfg.get("n_shared", 0):
        Is = cfg["I_shared"]
        out["ws_gate"] = _device_weights((Is, d), 1 / math.sqrt(d), seed, "ws_gate", device, dt)
        out["ws_up"] = _device_weights((Is, d), 1 / math.sqrt(d), seed, "ws_up", device, dt)
        out["ws_down"] = _device_weights((d, Is), 1 / math.sqrt(Is), seed, "ws_down", device, dt)
    else:
        out["ws_gate"] = out["ws_up"] = out["ws_down"] = None
    return out


def oracle_view(t: torch.Tensor | None):
    """Host numpy view of a tensor as the oracle reads it: bf16 as uint16 bits,
    fp32 as float32 (a copy when the tensor lives on a device)."""
    if t is None:
        return None
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


class ExpertView:
    """Per-expert host accessor for a [E, ...] device tensor (decoded lazily)."""

    def __init__(self, t: torch.Tensor):
        self.t = t

    def __getitem__(self, e):
        return oracle_view(self.t[int(e)])

    def __len__(self):
        return self.t.shape[0]
