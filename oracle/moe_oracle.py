"""Plain fp64 CPU oracle for the MoE-layer hot path.

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import, call or
execute this module: only the test suite, the smoke check in
``__graft_entry__`` and the CPU-baseline leg of ``bench.py`` use it. It shares
no code with the HIP library and imports nothing from the package.

What it computes is one GPU's share of the DeepSeek-V3 Mixture-of-Experts
layer that the paper reproduces (App. M, "DeepSeek-V3 MoE Dispatch and
Combine"; §4 Workloads): route every token to experts, dispatch the tokens to
their experts, run each expert's GEMM1 (gate/up) + SwiGLU + GEMM2 (down), and
combine the expert outputs back into token order (App. F, host MoE pipeline
listing). On one GPU the two all-to-all exchanges become a permutation and its
inverse. The paper never writes down the gate, the scores, the top-k rule or
the combine weights; this module takes the public DeepSeek-V3 rule (sigmoid
scores, per-expert selection bias, group-limited top-k, weights normalised and
scaled) and the Mixtral rule (softmax, top-k, renormalised), the two MoE
families the workload presets name. Every reading that had to be chosen is
listed in the design notes of the repository.

Conventions
-----------
* Every arithmetic operation runs in float64.
* bf16 inputs are passed as ``uint16`` arrays holding the bf16 bit patterns;
  float32/float64 arrays are taken as they are. :func:`to_f64` decodes both.
* Selection ties are broken by the lower index, both for experts and for
  groups; the output slots of a token are ordered by key descending, then
  index ascending.
* Routing keys: softmax routing selects on the logit itself (softmax is
  monotone in it); sigmoid routing selects on ``sigmoid(logit) + bias``, and
  the bias never enters the weights.

Parity status: every function here is pinned by the CPU tests (closed forms,
brute-force enumeration on tiny inputs, special cases that reduce to a dense
SwiGLU or a dense softmax mixture, and invariants; the token quantization by
hand-derived examples with exact power-of-two scales, its error bound and the
quantized layer's reduction to the plain one on exactly representable
tokens; the FP8 codes by hand-derived examples, the code table's defining
properties and the same reduction; the expert-parallel receive plan by
hand-derived examples and
invariants, its FFN by its reduction to the single-GPU expert FFN). The layer
as a whole has no value printed in the paper; it is pinned only through those
pieces.
"""

from __future__ import annotations

import numpy as np

__all__ = [
    "to_f64",
    "gate_logits",
    "route",
    "dispatch",
    "silu",
    "swiglu_ffn",
    "expert_ffn",
    "combine",
    "layer",
    "layer_rows",
    "quantize_tokens",
    "dequantize_tokens",
    "e4m3_values",
    "quantize_tokens_fp8",
    "dequantize_tokens_fp8",
    "ep_receive_plan",
    "ep_receive_ffn",
]


# ---------------------------------------------------------------------------
# input decoding
# ---------------------------------------------------------------------------

def to_f64(a) -> np.ndarray:
    """Decode an input array to float64.

    ``uint16`` arrays are bf16 bit patterns: the 16 bits are the high half of
    an IEEE float32, so shifting them up by 16 gives the float32 bits exactly.
    """
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    if a.dtype.kind != "f":
        raise TypeError(f"oracle input must be float or bf16 bits, got {a.dtype}")
    return a.astype(np.float64)


# ---------------------------------------------------------------------------
# gating (App. M: each token is routed to experts; the gate is the router GEMM)
# ---------------------------------------------------------------------------

def gate_logits(x, w_router) -> np.ndarray:
    """Router logits ``u[t, e] = sum_c x[t, c] * w_router[e, c]`` in fp64.

    x: [T, d]; w_router: [E, d] (each expert's router vector is a row).
    """
    return to_f64(x) @ to_f64(w_router).T


# ---------------------------------------------------------------------------
# routing: scores, group-limited top-k, weights
# ---------------------------------------------------------------------------

def _sigmoid(z: np.ndarray) -> np.ndarray:
    with np.errstate(over="ignore"):
        return 1.0 / (1.0 + np.exp(-z))


def route(logits, *, k: int, score: str = "softmax", bias=None,
          n_groups: int = 1, topk_groups: int = 1, renorm: bool = True,
          scale: float = 1.0, return_detail: bool = False):
    """Select ``k`` experts per token and their combine weights.

    logits: [T, E] router logits (any float dtype; decoded to fp64).
    score: ``"softmax"`` (Mixtral family) or ``"sigmoid"`` (DeepSeek-V3).
    bias: [E] per-expert selection bias, sigmoid routing only.

    Steps, one token at a time (vectorised over tokens):

    1. Scores. softmax: ``p = exp(u - max u) / sum``; the selection key is
       ``u``. sigmoid: ``s = 1 / (1 + exp(-u))``; the key is ``s + bias``.
    2. Group limit (``n_groups > 1``): experts are split into ``n_groups``
       contiguous groups of ``E / n_groups``; a group's score is the sum of its
       two largest keys (its only key if a group has one expert); the
       ``topk_groups`` best groups (score descending, lower group index first
       on ties) stay eligible and every other expert is dropped.
    3. Top-k: the ``k`` eligible experts with the largest keys, lower expert
       index first on ties, stored in that order.
    4. Weights: the selected experts' scores (``p`` or the unbiased ``s``),
       divided by their sum when ``renorm``, then multiplied by ``scale``.

    Returns ``(topk_idx int32 [T, k], topk_w float64 [T, k])``; with
    ``return_detail`` a dict that also holds the keys, group scores, chosen
    groups and the selection margin of every token (the gap between the last
    selected and the first unselected key, or group score, whichever is
    smaller; +inf where nothing was left out).
    """
    u = to_f64(logits)
    if u.ndim != 2:
        raise ValueError("logits must be [T, E]")
    T, E = u.shape
    if not (1 <= k <= E):
        raise ValueError("need 1 <= k <= E")
    if n_groups < 1 or E % n_groups:
        raise ValueError("E must be a multiple of n_groups")
    if not (1 <= topk_groups <= n_groups):
        raise ValueError("need 1 <= topk_groups <= n_groups")
    gsize = E // n_groups
    if n_groups > 1 and k > topk_groups * gsize:
        raise ValueError("k exceeds the experts left by the group limit")

    # step 1: scores and selection keys
    if score == "softmax":
        if bias is not None:
            raise ValueError("bias is defined for sigmoid routing only")
        z = np.exp(u - u.max(axis=1, keepdims=True))
        prob = z / z.sum(axis=1, keepdims=True)
        keys = u.copy()
    elif score == "sigmoid":
        prob = _sigmoid(u)
        keys = prob.copy()
        if bias is not None:
            keys = keys + to_f64(bias)[None, :]
    else:
        raise ValueError(f"unknown score function {score!r}")

    # step 2: group limit
    group_score = None
    chosen_groups = None
    group_margin = np.full(T, np.inf)
    eligible = keys
    if n_groups > 1:
        grouped = keys.reshape(T, n_groups, gsize)
        top2 = np.sort(grouped, axis=2)[:, :, ::-1][:, :, : min(2, gsize)]
        group_score = top2.sum(axis=2)
        gorder = np.argsort(-group_score, axis=1, kind="stable")
        chosen_groups = gorder[:, :topk_groups]
        keep = np.zeros((T, n_groups), dtype=bool)
        np.put_along_axis(keep, chosen_groups, True, axis=1)
        eligible = np.where(np.repeat(keep, gsize, axis=1), keys, -np.inf)
        if topk_groups < n_groups:
            gs_sorted = np.take_along_axis(group_score, gorder, axis=1)
            group_margin = gs_sorted[:, topk_groups - 1] - gs_sorted[:, topk_groups]

    # step 3: top-k by (key descending, index ascending)
    order = np.argsort(-eligible, axis=1, kind="stable")
    topk_idx = order[:, :k]
    n_eligible = (topk_groups * gsize) if n_groups > 1 else E
    expert_margin = np.full(T, np.inf)
    if k < n_eligible:
        ks = np.take_along_axis(eligible, order[:, : k + 1], axis=1)
        expert_margin = ks[:, k - 1] - ks[:, k]

    # step 4: weights from the unbiased scores
    w = np.take_along_axis(prob, topk_idx, axis=1)
    if renorm:
        w = w / w.sum(axis=1, keepdims=True)
    w = w * float(scale)

    topk_idx = topk_idx.astype(np.int32)
    if not return_detail:
        return topk_idx, w
    return topk_idx, w, {
        "keys": keys,
        "prob": prob,
        "group_score": group_score,
        "chosen_groups": chosen_groups,
        "margin": np.minimum(expert_margin, group_margin),
    }


# ---------------------------------------------------------------------------
# dispatch: the single-GPU form of the all-to-all that sends tokens to experts
# ---------------------------------------------------------------------------

def dispatch(topk_idx, E: int):
    """Group the ``T*k`` token-to-expert assignments by expert.

    Assignment ``a = t*k + j`` sends token ``t`` to expert ``topk_idx[t, j]``.
    The expert segments are variable-sized and unpadded (App. M: transfers of
    variable size per peer). Rows are ordered by (expert ascending, token
    ascending); a token holds at most one slot per expert, so the order is
    total.

    Returns ``counts [E]``, ``offsets [E+1]`` (exclusive prefix sum, so
    ``offsets[E] == T*k``), ``sorted_token [T*k]`` (token of each row),
    ``sorted_assign [T*k]`` (assignment of each row) and ``inv_perm [T*k]``
    (row of each assignment), all int32.
    """
    idx = np.asarray(topk_idx)
    if idx.ndim != 2:
        raise ValueError("topk_idx must be [T, k]")
    T, k = idx.shape
    flat = idx.reshape(-1).astype(np.int64)
    if flat.size and (flat.min() < 0 or flat.max() >= E):
        raise ValueError("expert index out of range")
    counts = np.bincount(flat, minlength=E)
    offsets = np.zeros(E + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(counts)
    token_of = np.arange(T * k) // max(k, 1)
    rows = np.lexsort((token_of, flat))  # primary key expert, then token
    inv = np.empty(T * k, dtype=np.int64)
    inv[rows] = np.arange(T * k)
    return (counts.astype(np.int32), offsets.astype(np.int32),
            token_of[rows].astype(np.int32), rows.astype(np.int32),
            inv.astype(np.int32))


# ---------------------------------------------------------------------------
# expert FFN (App. M: GEMM1 up/gate projection, SwiGLU, GEMM2 down projection)
# ---------------------------------------------------------------------------

def silu(z) -> np.ndarray:
    """SiLU(z) = z * sigmoid(z)."""
    z = np.asarray(z, dtype=np.float64)
    return z * _sigmoid(z)


def swiglu_ffn(xrows, w_gate, w_up, w_down) -> np.ndarray:
    """One SwiGLU expert on a block of rows, in fp64.

    xrows: [M, d]; w_gate, w_up: [I, d]; w_down: [d, I] (every weight matrix
    holds one output feature per row). Returns ``(silu(X Wg^T) * (X Wu^T)) Wd^T``
    of shape [M, d].
    """
    X = to_f64(xrows)
    g = X @ to_f64(w_gate).T
    up = X @ to_f64(w_up).T
    return (silu(g) * up) @ to_f64(w_down).T


def expert_ffn(x, sorted_token, offsets, w_gate, w_up, w_down) -> np.ndarray:
    """Run every expert on its segment of dispatched rows.

    x: [T, d]; ``w_gate[e]``/``w_up[e]``: [I, d]; ``w_down[e]``: [d, I]. The
    weights may be any object indexable by expert (an array, or a lazy
    per-expert accessor for resident multi-GB tensors). Returns ``y_perm``
    [T*k, d] in fp64, row ``r`` being expert(r)'s output for token
    ``sorted_token[r]``. No intermediate is rounded.
    """
    X = to_f64(x)
    offsets = np.asarray(offsets, dtype=np.int64)
    sorted_token = np.asarray(sorted_token, dtype=np.int64)
    E = offsets.size - 1
    y = np.zeros((int(offsets[-1]), X.shape[1]))
    for e in range(E):
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        if hi > lo:
            y[lo:hi] = swiglu_ffn(X[sorted_token[lo:hi]], w_gate[e], w_up[e], w_down[e])
    return y


# ---------------------------------------------------------------------------
# token quantization around the dispatch exchange (App. F pipeline: quantize
# tokens to int8 with per-token scales, send, dequantize before GEMM1; App. M
# steps (1)-(3))
# ---------------------------------------------------------------------------

def quantize_tokens(x):
    """Per-token symmetric int8 quantization of the token rows.

    ``scale[t] = max_c |x[t, c]| / 127`` and ``codes[t, c] = x[t, c] / scale[t]``
    rounded half to even and clamped to [-127, 127]; a row of zeros gets scale
    0 and codes 0. The paper fixes int8 codes and one scale per token but no
    precision; because the divisions decide integers, they run in float32 (the
    kernel's precision), on the same float32 inputs the kernel reads. Returns
    (codes int8 [T, d], scales float32 [T]).
    """
    xf = to_f64(x).astype(np.float32)  # bf16 and fp32 inputs are exact in float32
    if xf.ndim != 2:
        raise ValueError("x must be [T, d]")
    absmax = np.abs(xf).max(axis=1) if xf.shape[1] else np.zeros(xf.shape[0], np.float32)
    scales = (absmax / np.float32(127.0)).astype(np.float32)
    safe = np.where(scales > 0, scales, np.float32(1.0)).astype(np.float32)
    q = np.rint(xf / safe[:, None])  # float32 division, round half to even
    q = np.clip(q, -127, 127)
    q[scales == 0] = 0
    return q.astype(np.int8), scales


def dequantize_tokens(codes, scales) -> np.ndarray:
    """``codes[t, c] * scales[t]`` in fp64 (the tokens GEMM1 sees)."""
    return np.asarray(codes, dtype=np.float64) * np.asarray(scales, dtype=np.float64)[:, None]


# FP8 (Table 5 names an FP8 quantize phase): the OCP E4M3 format, 1 sign,
# 4 exponent (bias 7) and 3 mantissa bits; exponent field 0 holds the
# subnormals m/8 * 2^-6, fields 1..15 the normals (1 + m/8) * 2^(e-7), and
# only code 0x7F (with its sign) is NaN, so the largest finite value is 448.
E4M3_MAX = 448.0


def e4m3_values() -> np.ndarray:
    """float64 [256]: the value of every E4M3 code (NaN for 0x7F and 0xFF)."""
    out = np.empty(256)
    for code in range(256):
        sign = -1.0 if code & 0x80 else 1.0
        e, m = (code >> 3) & 0xF, code & 0x7
        if e == 0xF and m == 0x7:
            out[code] = np.nan
        elif e == 0:
            out[code] = sign * (m / 8.0) * 2.0 ** -6
        else:
            out[code] = sign * (1.0 + m / 8.0) * 2.0 ** (e - 7)
    return out


def _e4m3_encode(f) -> np.ndarray:
    """Codes of float values: the nearest finite E4M3 magnitude (ties to the
    even mantissa, which is the even code), magnitudes above 448 taken as 448,
    and the sign bit of the value (so -0 and negatives that round to 0 give
    0x80)."""
    f = np.asarray(f, dtype=np.float64)
    mags = e4m3_values()[:0x7F]            # codes 0x00..0x7E, increasing
    a = np.minimum(np.abs(f), E4M3_MAX)
    hi = np.clip(np.searchsorted(mags, a, side="left"), 0, 0x7E)   # first magnitude >= a
    lo = np.clip(hi - 1, 0, 0x7E)
    dlo, dhi = a - mags[lo], mags[hi] - a
    pick_hi = (dhi < dlo) | ((dhi == dlo) & (hi % 2 == 0))
    code = np.where(pick_hi, hi, lo)
    return (code | np.where(np.signbit(f), 0x80, 0)).astype(np.uint8)


def quantize_tokens_fp8(x):
    """Per-token FP8 (E4M3) quantization of the token rows.

    ``scale[t] = max_c |x[t, c]| / 448`` and ``codes[t, c]`` the E4M3 code of
    ``x[t, c] / scale[t]``, rounded to the nearest value, ties to even; a row
    of zeros gets scale 0 and codes 0. The divisions run in float32, as for
    the int8 codes (they decide the codes). Returns (codes uint8 [T, d],
    scales float32 [T]).
    """
    xf = to_f64(x).astype(np.float32)
    if xf.ndim != 2:
        raise ValueError("x must be [T, d]")
    absmax = np.abs(xf).max(axis=1) if xf.shape[1] else np.zeros(xf.shape[0], np.float32)
    scales = (absmax / np.float32(E4M3_MAX)).astype(np.float32)
    safe = np.where(scales > 0, scales, np.float32(1.0)).astype(np.float32)
    codes = _e4m3_encode(xf / safe[:, None])  # float32 quotient, then exact rounding to E4M3
    codes[scales == 0] = 0
    return codes, scales


def dequantize_tokens_fp8(codes, scales) -> np.ndarray:
    """``value(codes[t, c]) * scales[t]`` in fp64 (the tokens GEMM1 sees)."""
    return e4m3_values()[np.asarray(codes, dtype=np.int64)] * np.asarray(scales, dtype=np.float64)[:, None]


def _dequantized(x, quant):
    """The tokens the routed experts see under a token quantization."""
    if quant == "int8":
        return dequantize_tokens(*quantize_tokens(x))
    if quant == "fp8":
        return dequantize_tokens_fp8(*quantize_tokens_fp8(x))
    return x


# ---------------------------------------------------------------------------
# expert parallelism, receive side (App. M: each GPU owns some experts; the
# dispatch exchange brings it the rows of its own tokens and of its peer's
# tokens routed to those experts; §4.3: the self rows are ready at once, the
# remote rows once the exchange has delivered them)
# ---------------------------------------------------------------------------

def ep_receive_plan(self_offsets, self_sorted_token, peer_offsets, peer_sorted_token, e_first: int, e_count: int):
    """Rows a GPU owning global experts [e_first, e_first + e_count) receives.

    Inputs are the two ranks' dispatches over the global experts (``offsets``
    and ``sorted_token`` as returned by :func:`dispatch`). Local expert ``e``
    (global ``e_first + e``) gets this GPU's rows of that expert, then the
    peer's, each in dispatch order. Returns ``row_token`` (token of each row
    in its own rank's input), ``offsets [e_count+1]`` and ``self_end
    [e_count]`` (rows ``[offsets[e], self_end[e])`` are this GPU's tokens),
    all int32.
    """
    so = np.asarray(self_offsets, dtype=np.int64)
    po = np.asarray(peer_offsets, dtype=np.int64)
    st = np.asarray(self_sorted_token, dtype=np.int64)
    pt = np.asarray(peer_sorted_token, dtype=np.int64)
    rows = []
    offsets = [0]
    self_end = []
    for e in range(e_count):
        g = e_first + e
        mine = list(st[so[g]:so[g + 1]])
        theirs = list(pt[po[g]:po[g + 1]])
        rows += mine
        self_end.append(offsets[-1] + len(mine))
        rows += theirs
        offsets.append(offsets[-1] + len(mine) + len(theirs))
    return (np.asarray(rows, dtype=np.int32), np.asarray(offsets, dtype=np.int32),
            np.asarray(self_end, dtype=np.int32))


def ep_receive_ffn(x_self, x_peer, row_token, offsets, self_end, w_gate, w_up, w_down, rows=None) -> np.ndarray:
    """Expert FFN of received rows, in fp64: row ``r`` of local expert ``e`` is
    token ``row_token[r]`` of ``x_self`` (below ``self_end[e]``) or of
    ``x_peer``; the weights are indexable by local expert. ``rows``: compute
    only these rows (all if None); returns ``[len(rows), d]``."""
    offsets = np.asarray(offsets, dtype=np.int64)
    self_end = np.asarray(self_end, dtype=np.int64)
    row_token = np.asarray(row_token, dtype=np.int64)
    n = int(offsets[-1])
    rows = np.arange(n) if rows is None else np.asarray(rows, dtype=np.int64)
    Xs, Xp = to_f64(x_self), to_f64(x_peer)
    out = np.zeros((rows.size, Xs.shape[1]))
    expert = np.searchsorted(offsets, rows, side="right") - 1
    for e in np.unique(expert):
        sel = np.nonzero(expert == e)[0]
        r = rows[sel]
        mine = r < self_end[e]
        src = np.empty((r.size, Xs.shape[1]))
        src[mine] = Xs[row_token[r[mine]]]
        src[~mine] = Xp[row_token[r[~mine]]]
        out[sel] = swiglu_ffn(src, w_gate[e], w_up[e], w_down[e])
    return out


# ---------------------------------------------------------------------------
# combine: the single-GPU form of the reverse all-to-all
# ---------------------------------------------------------------------------

def combine(y_perm, inv_perm, topk_w, shared_out=None) -> np.ndarray:
    """``out[t] = sum_j topk_w[t, j] * y_perm[inv_perm[t*k + j]] (+ shared_out[t])``.

    The sum runs over the slots j in ascending order; the shared expert, when
    present, is added with weight 1.
    """
    W = np.asarray(topk_w, dtype=np.float64)
    T, k = W.shape
    Y = to_f64(y_perm)
    inv = np.asarray(inv_perm, dtype=np.int64).reshape(T, k)
    out = np.zeros((T, Y.shape[1]))
    for j in range(k):
        out += W[:, j : j + 1] * Y[inv[:, j]]
    if shared_out is not None:
        out += to_f64(shared_out)
    return out


# ---------------------------------------------------------------------------
# whole layer
# ---------------------------------------------------------------------------

def _route_kwargs(cfg: dict) -> dict:
    return dict(k=cfg["k"], score=cfg["score"], n_groups=cfg.get("n_groups", 1),
                topk_groups=cfg.get("topk_groups", 1), renorm=cfg.get("renorm", True),
                scale=cfg.get("scale", 1.0))


def layer(cfg: dict, x, w_router, bias, w_gate, w_up, w_down,
          ws_gate=None, ws_up=None, ws_down=None, logits=None) -> dict:
    """The full layer: gate, route, dispatch, expert FFN, shared expert, combine.

    cfg holds ``E, k, score, n_groups, topk_groups, renorm, scale`` and
    ``n_shared`` (0 or 1), and optionally ``quant`` ("int8": the routed
    experts see the tokens after :func:`quantize_tokens` and
    :func:`dequantize_tokens`; "fp8": after :func:`quantize_tokens_fp8` and
    :func:`dequantize_tokens_fp8`; the gate and the shared expert, which stay
    on the sending side in the paper's pipeline, see the original tokens).
    ``logits`` replaces the gate when given (used to re-route from logits
    computed elsewhere). The shared-expert weights are [I_s, d], [I_s, d] and
    [d, I_s]. Returns every intermediate.
    """
    if logits is None:
        logits = gate_logits(x, w_router)
    rb = None if cfg["score"] == "softmax" else bias
    topk_idx, topk_w, det = route(logits, bias=rb, return_detail=True, **_route_kwargs(cfg))
    counts, offsets, sorted_token, sorted_assign, inv_perm = dispatch(topk_idx, cfg["E"])
    x_routed = _dequantized(x, cfg.get("quant"))
    y_perm = expert_ffn(x_routed, sorted_token, offsets, w_gate, w_up, w_down)
    shared = None
    if cfg.get("n_shared", 0):
        shared = swiglu_ffn(x, ws_gate, ws_up, ws_down)
    out = combine(y_perm, inv_perm, topk_w, shared)
    return dict(logits=to_f64(logits), topk_idx=topk_idx, topk_w=topk_w,
                margin=det["margin"], counts=counts, offsets=offsets,
                sorted_token=sorted_token, sorted_assign=sorted_assign,
                inv_perm=inv_perm, y_perm=y_perm, shared=shared, out=out)


def layer_rows(x, rows, topk_idx, topk_w, w_gate, w_up, w_down,
               ws_gate=None, ws_up=None, ws_down=None, quant=None) -> np.ndarray:
    """Layer outputs for a subset of tokens, given their routing.

    The FFN acts on each row independently, so ``out[t]`` needs only token
    ``t``, its selected experts and their weights:
    ``out[t] = sum_j topk_w[t, j] * FFN_{topk_idx[t, j]}(x[t]) (+ shared(x[t]))``.
    rows: token indices; ``topk_idx``/``topk_w``: [len(rows), k] for those
    tokens. Experts are visited once each, so a large resident weight tensor
    is decoded one expert at a time. ``quant="int8"`` or ``"fp8"``: the routed
    experts see the quantized tokens (the quantization is per token, so a subset of rows
    quantizes as it would inside the whole batch). Returns [len(rows), d] in
    fp64.
    """
    X = to_f64(np.asarray(x)[np.asarray(rows, dtype=np.int64)])
    Xr = _dequantized(np.asarray(x)[np.asarray(rows, dtype=np.int64)], quant) if quant in ("int8", "fp8") else X
    idx = np.asarray(topk_idx, dtype=np.int64)
    W = np.asarray(topk_w, dtype=np.float64)
    R, k = idx.shape
    y = np.zeros((R, k, X.shape[1]))
    for e in np.unique(idx):
        sel_r, sel_j = np.nonzero(idx == e)
        y[sel_r, sel_j] = swiglu_ffn(Xr[sel_r], w_gate[e], w_up[e], w_down[e])
    out = np.zeros((R, X.shape[1]))
    for j in range(k):
        out += W[:, j : j + 1] * y[:, j]
    if ws_gate is not None:
        out += swiglu_ffn(X, ws_gate, ws_up, ws_down)
    return out
