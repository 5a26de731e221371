"""Invariant checks for routing and dispatch results, and the output metric.

TEST INFRASTRUCTURE ONLY (same rule as :mod:`oracle.moe_oracle`): used by the
test suite, the smoke check and the benchmark's parity sampling, never by the
product path.

The invariants follow from the definitions in :mod:`oracle.moe_oracle`:

* routing: indices in range, distinct within a token; weights non-negative
  and summing to the routing scale when they are renormalised;
* dispatch: ``sum(counts) == T*k``; ``offsets`` is the exclusive prefix sum of
  ``counts``; the row permutation is a bijection on ``[0, T*k)``;
  ``sorted_token[inv_perm[t*k + j]] == t``; the row of assignment ``(t, j)``
  lies in the segment of expert ``topk_idx[t, j]``; tokens strictly increase
  inside every segment (stable order).

Every check raises ``AssertionError`` with a message naming the first
violation, so a planted mistake is reported, not silently accepted.
"""

from __future__ import annotations

import numpy as np

__all__ = ["check_routing", "check_dispatch", "max_rel_err", "rel_err_report"]


def check_routing(topk_idx, topk_w, E: int, *, scale: float = 1.0,
                  renorm: bool = True, atol: float = 1e-6) -> None:
    idx = np.asarray(topk_idx, dtype=np.int64)
    w = np.asarray(topk_w, dtype=np.float64)
    assert idx.ndim == 2 and idx.shape == w.shape, "topk_idx/topk_w shape mismatch"
    if idx.size == 0:
        return
    assert idx.min() >= 0 and idx.max() < E, "expert index out of range"
    srt = np.sort(idx, axis=1)
    dup = np.nonzero((srt[:, 1:] == srt[:, :-1]).any(axis=1))[0]
    assert dup.size == 0, f"token {dup[:1]} selects an expert twice"
    assert (w >= 0).all(), "negative routing weight"
    if renorm:
        err = np.abs(w.sum(axis=1) - scale)
        bad = np.nonzero(err > atol * max(1.0, scale))[0]
        assert bad.size == 0, f"weights of token {bad[0]} sum to {w[bad[0]].sum()}, want {scale}"


def check_dispatch(topk_idx, counts, offsets, sorted_token, inv_perm,
                   sorted_assign=None) -> None:
    idx = np.asarray(topk_idx, dtype=np.int64)
    T, k = idx.shape
    n = T * k
    counts = np.asarray(counts, dtype=np.int64)
    offsets = np.asarray(offsets, dtype=np.int64)
    st = np.asarray(sorted_token, dtype=np.int64)
    inv = np.asarray(inv_perm, dtype=np.int64)
    E = counts.size
    assert offsets.size == E + 1, "offsets must have E+1 entries"
    assert counts.sum() == n, f"counts sum to {counts.sum()}, want T*k = {n}"
    assert (counts >= 0).all(), "negative count"
    assert offsets[0] == 0 and (np.diff(offsets) == counts).all(), \
        "offsets are not the exclusive prefix sum of counts"
    assert st.size == n and inv.size == n, "permutation arrays must hold T*k entries"
    if n == 0:
        return
    assert inv.min() >= 0 and inv.max() < n, "inv_perm out of range"
    assert np.unique(inv).size == n, "inv_perm is not a bijection"
    t_of = np.arange(n) // k
    assert (st[inv] == t_of).all(), "sorted_token[inv_perm[t*k+j]] != t"
    seg = np.searchsorted(offsets, inv, side="right") - 1
    assert (seg == idx.reshape(-1)).all(), "a row sits outside its expert's segment"
    for e in range(E):
        lo, hi = offsets[e], offsets[e + 1]
        if hi - lo > 1:
            assert (np.diff(st[lo:hi]) > 0).all(), f"tokens not increasing in expert {e}"
    if sorted_assign is not None:
        sa = np.asarray(sorted_assign, dtype=np.int64)
        assert (sa[inv] == np.arange(n)).all(), "sorted_assign is not the inverse of inv_perm"


def max_rel_err(got, want) -> float:
    """``max_i |got_i - want_i| / max(|want_i|, rms(want))``.

    Element-wise relative error with an rms floor, so outputs near zero do not
    dominate; 0 for empty inputs.
    """
    g = np.asarray(got, dtype=np.float64)
    w = np.asarray(want, dtype=np.float64)
    assert g.shape == w.shape, f"shape {g.shape} vs {w.shape}"
    if w.size == 0:
        return 0.0
    rms = float(np.sqrt(np.mean(w * w)))
    floor = np.maximum(np.abs(w), rms if rms > 0 else 1.0)
    return float(np.max(np.abs(g - w) / floor))


def rel_err_report(got, want) -> dict:
    g = np.asarray(got, dtype=np.float64)
    w = np.asarray(want, dtype=np.float64)
    if w.size == 0:
        return dict(max_rel=0.0, norm_inf=0.0, frob=0.0)
    d = g - w
    return dict(
        max_rel=max_rel_err(g, w),
        norm_inf=float(np.abs(d).max() / max(np.abs(w).max(), 1e-300)),
        frob=float(np.linalg.norm(d) / max(np.linalg.norm(w), 1e-300)),
    )
