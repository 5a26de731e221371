"""GPU parity of the receive side of expert parallelism (App. M: every GPU owns
some experts and receives its own and its peer's rows of them; §4.3: the self
rows are there at once, the remote rows once the exchange delivers them),
through the C ABI.

moe_ep_plan: bit-exact against the oracle's receive plan (integer work).
moe_ep_copy_rows: received rows equal their source rows bit for bit; rows of
the other source stay untouched. moe_expert_ffn_segments and
moe_ep_expert_ffn: every row against the oracle's receive-side FFN within the
bf16 tolerance; the segment FFN gives the same bits as moe_expert_ffn on the
same rows, and every schedule (chunk counts, workgroup caps, one or two
streams) gives the same bits.
"""
import numpy as np
import pytest
import torch

from oracle import moe_oracle as O
from oracle.checks import max_rel_err
from paper_2603_02376_amd import inputs, moe
from tests.gpu_util import BF16_TOL, host, log

pytestmark = pytest.mark.gpu


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _bf16(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16).cuda()


def _dispatch(T, Eg, k, d, I, topk):
    """moe_dispatch over the global experts on the GPU: (offsets, sorted_token)."""
    cfg = moe.MoeConfig(d=d, E=Eg, k=k, I=I, dtype="bf16")
    ws = moe.alloc_workspace(cfg, T)
    n = T * k
    z = lambda m: torch.empty(m, dtype=torch.int32, device="cuda")
    counts, offsets, st, sa, inv = z(Eg), z(Eg + 1), z(n), z(n), z(n)
    moe.moe_dispatch(cfg, T, _dev(topk), counts, offsets, st, sa, inv, ws)
    return offsets, st


def _setup(T, d, Eg, k, I, ratio, seed=0, peer_T=None, topk_self=None, topk_peer=None):
    """One GPU owning global experts [0, Eg/2) of a two-GPU pair."""
    E = Eg // 2
    peer_T = T if peer_T is None else peer_T
    p = dict(T=T, d=d, E=E, k=k, I=I, dtype="bf16", n_shared=0, bias="none")
    t = inputs.make_inputs(p, seed, "cuda")  # x: this GPU's tokens; weights of the E local experts
    xp = _bf16(inputs.ep_peer_tokens(max(peer_T, 1), d, seed))
    st = inputs.ep_topk(T, Eg, k, ratio, "self", seed) if topk_self is None else topk_self
    pt = inputs.ep_topk(max(peer_T, 1), Eg, k, ratio, "peer", seed)[:peer_T] if topk_peer is None else topk_peer
    so, ss = _dispatch(T, Eg, k, d, I, st)
    if peer_T:
        po, ps = _dispatch(peer_T, Eg, k, d, I, pt)
    else:
        po, ps = torch.zeros(Eg + 1, dtype=torch.int32, device="cuda"), torch.zeros(1, dtype=torch.int32,
                                                                                    device="cuda")
    cfg = moe.MoeConfig(d=d, E=E, k=k, I=I, dtype="bf16", weight_layout="packed")
    n_rows = int(host(so)[E]) + int(host(po)[E])
    rt = torch.full((max(n_rows, 1),), -7, dtype=torch.int32, device="cuda")
    off = torch.empty(E + 1, dtype=torch.int32, device="cuda")
    se = torch.empty(E, dtype=torch.int32, device="cuda")
    moe.moe_ep_plan(cfg, 0, so, ss, T * k, po, ps, peer_T * k, rt, n_rows, off, se)
    torch.cuda.synchronize()
    # the plan, bit-exact against the oracle's (from the oracle's own dispatch)
    ods = O.dispatch(st, Eg)
    odp = O.dispatch(pt, Eg) if peer_T else (None, np.zeros(Eg + 1, np.int32), np.zeros(0, np.int32))
    w_rt, w_off, w_se = O.ep_receive_plan(ods[1], ods[2], odp[1], odp[2], 0, E)
    assert np.array_equal(host(off), w_off) and np.array_equal(host(se), w_se)
    assert np.array_equal(host(rt)[:n_rows], w_rt)
    gu, dn = moe.pack_weights(cfg, t["w_gate"], t["w_up"], t["w_down"])
    return dict(cfg=cfg, T=T, peer_T=peer_T, E=E, d=d, k=k, n_rows=n_rows, x=t["x"], xp=xp, rt=rt, off=off, se=se,
                gu=gu, dn=dn, t=t, plan=(w_rt, w_off, w_se))


def _expected_recv(s):
    rt, off, se = s["plan"]
    xs, xp = host(s["x"].float()), host(s["xp"].float())
    want = np.empty((s["n_rows"], s["d"]), np.float32)
    for e in range(s["E"]):
        want[off[e]:se[e]] = xs[rt[off[e]:se[e]]]
        want[se[e]:off[e + 1]] = xp[rt[se[e]:off[e + 1]]]
    return want


def _oracle_y(s, rows=None):
    rt, off, se = s["plan"]
    t = s["t"]
    return O.ep_receive_ffn(inputs.oracle_view(s["x"]), inputs.oracle_view(s["xp"]), rt, off, se,
                            inputs.ExpertView(t["w_gate"]), inputs.ExpertView(t["w_up"]),
                            inputs.ExpertView(t["w_down"]), rows=rows)


CASES = [
    # T, d, global experts, k, I, ratio
    (50, 256, 16, 2, 128, 3.0),
    (333, 512, 32, 4, 256, 2.0),   # several column tiles, ragged segments
    (400, 256, 8, 4, 128, 5.0),    # ~330 rows per expert: passes of 192 + the rest
]
IDS = ["T{}_d{}_E{}_k{}_I{}_r{}".format(*c) for c in CASES]


@pytest.mark.parametrize("case", CASES, ids=IDS)
def test_plan_and_copy_rows(case):
    log("ep plan + copy", case)
    s = _setup(*case)
    n, d, E = s["n_rows"], s["d"], s["E"]
    recv = torch.full((n, d), -3.0, dtype=torch.bfloat16, device="cuda")
    want = _expected_recv(s)
    se, off = host(s["se"]), host(s["off"])
    self_rows = np.concatenate([np.arange(off[e], se[e]) for e in range(E)])
    remote_rows = np.concatenate([np.arange(se[e], off[e + 1]) for e in range(E)])
    moe.moe_ep_copy_rows(s["cfg"], moe.MOE_EP_SELF, n, s["x"], s["T"], s["rt"], s["off"], s["se"], 0, E, recv)
    torch.cuda.synchronize()
    got = host(recv.float())
    assert np.array_equal(got[self_rows], want[self_rows])
    assert (got[remote_rows] == -3.0).all(), "remote rows written by the self copy"
    # the remote rows in two expert ranges, with a small workgroup cap
    for e0, e1 in ((0, E // 2), (E // 2, E)):
        moe.moe_ep_copy_rows(s["cfg"], moe.MOE_EP_REMOTE, n, s["xp"], s["peer_T"], s["rt"], s["off"], s["se"], e0,
                             e1, recv, max_workgroups=3)
    torch.cuda.synchronize()
    assert np.array_equal(host(recv.float()), want)
    # the other half of the experts (a GPU owning global experts [E, 2E))
    so, ss = _dispatch(s["T"], 2 * E, s["k"], d, 128, inputs.ep_topk(s["T"], 2 * E, s["k"], case[5], "self", 0))
    po, ps = _dispatch(s["T"], 2 * E, s["k"], d, 128, inputs.ep_topk(s["T"], 2 * E, s["k"], case[5], "peer", 0))
    cap = s["T"] * s["k"] * 2
    rt2 = torch.empty(cap, dtype=torch.int32, device="cuda")
    off2 = torch.empty(E + 1, dtype=torch.int32, device="cuda")
    se2 = torch.empty(E, dtype=torch.int32, device="cuda")
    moe.moe_ep_plan(s["cfg"], E, so, ss, s["T"] * s["k"], po, ps, s["T"] * s["k"], rt2, cap, off2, se2)
    torch.cuda.synchronize()
    w = O.ep_receive_plan(host(so), host(ss), host(po), host(ps), E, E)
    assert np.array_equal(host(off2), w[1]) and np.array_equal(host(se2), w[2])
    assert np.array_equal(host(rt2)[:len(w[0])], w[0])


def _recv_filled(s):
    n, d, E = s["n_rows"], s["d"], s["E"]
    recv = torch.empty((n, d), dtype=torch.bfloat16, device="cuda")
    moe.moe_ep_copy_rows(s["cfg"], moe.MOE_EP_SELF, n, s["x"], s["T"], s["rt"], s["off"], s["se"], 0, E, recv)
    moe.moe_ep_copy_rows(s["cfg"], moe.MOE_EP_REMOTE, n, s["xp"], s["peer_T"], s["rt"], s["off"], s["se"], 0, E,
                         recv)
    return recv


@pytest.mark.parametrize("case", CASES, ids=IDS)
def test_ffn_segments(case):
    log("ep ffn segments", case)
    s = _setup(*case)
    n, d, E, k = s["n_rows"], s["d"], s["E"], s["k"]
    cfg = s["cfg"]
    recv = _recv_filled(s)
    ws = moe.ep_workspace(cfg, n)
    y = torch.full((n, d), float("nan"), dtype=torch.bfloat16, device="cuda")
    se, off = host(s["se"]), host(s["off"])
    # self segments only: the remote rows stay untouched
    moe.moe_expert_ffn_segments(cfg, n, recv, s["off"], s["se"], 0, E, s["gu"], s["dn"], y, ws)
    torch.cuda.synchronize()
    got = host(y.float())
    remote_rows = np.concatenate([np.arange(se[e], off[e + 1]) for e in range(E)])
    assert np.isnan(got[remote_rows]).all()
    # then the remote segments, in two expert ranges, with a workgroup cap
    moe.moe_expert_ffn_segments(cfg, n, recv, s["se"], s["off"][1:], 0, E // 2, s["gu"], s["dn"], y, ws,
                                max_workgroups=16)
    moe.moe_expert_ffn_segments(cfg, n, recv, s["se"], s["off"][1:], E // 2, E, s["gu"], s["dn"], y, ws)
    torch.cuda.synchronize()
    got = host(y.float())
    assert np.isfinite(got).all()
    err = max_rel_err(got, _oracle_y(s))
    log("  max_rel_err", err)
    assert err <= BF16_TOL
    # the same rows through moe_expert_ffn (recv as n tokens, gathered in order) give the same bits
    st = torch.zeros(n * k, dtype=torch.int32, device="cuda")
    st[:n] = torch.arange(n, dtype=torch.int32, device="cuda")
    y2 = torch.empty((n * k, d), dtype=torch.bfloat16, device="cuda")
    moe.moe_expert_ffn(cfg, n, recv, st, s["off"], s["gu"], None, s["dn"], y2, moe.alloc_workspace(cfg, n))
    # and one call over whole segments (seg_end NULL)
    y3 = torch.empty((n, d), dtype=torch.bfloat16, device="cuda")
    moe.moe_expert_ffn_segments(cfg, n, recv, s["off"], None, 0, E, s["gu"], s["dn"], y3, ws)
    torch.cuda.synchronize()
    assert torch.equal(y2[:n], y) and torch.equal(y3, y)


@pytest.mark.parametrize("case", CASES, ids=IDS)
def test_ep_expert_ffn_schedules(case):
    log("ep schedules", case)
    s = _setup(*case)
    n, d, E = s["n_rows"], s["d"], s["E"]
    cfg = s["cfg"]
    ws = moe.ep_workspace(cfg, n)
    want_recv = _expected_recv(s)
    link = torch.cuda.Stream()
    ref = None
    runs = [("sequential", 1, 0, 0, True), ("sequential", 1, 2, 0, False), ("self_remote", 1, 2, 16, True),
            ("self_remote", 1, 0, 0, False), ("expert_chunks", 1, 0, 0, True), ("expert_chunks", 3, 2, 16, True),
            ("expert_chunks", E, 1, 8, True), ("expert_chunks", 2, 0, 0, False)]
    for sched, chunks, lw, gw, two in runs:
        recv = torch.full((n, d), -5.0, dtype=torch.bfloat16, device="cuda")
        y = torch.full((n, d), float("nan"), dtype=torch.bfloat16, device="cuda")
        moe.moe_ep_expert_ffn(cfg, sched, n, s["x"], s["T"], s["xp"], s["peer_T"], s["rt"], s["off"], s["se"],
                              s["gu"], s["dn"], recv, y, ws, chunks=chunks, link_workgroups=lw, gemm_workgroups=gw,
                              s_link=link if two else None)
        torch.cuda.current_stream().synchronize()  # the call's end on s_compute covers the transfer
        assert np.array_equal(host(recv.float()), want_recv), sched
        if ref is None:
            ref = y.clone()
            err = max_rel_err(host(y.float()), _oracle_y(s))
            log("  max_rel_err", err)
            assert err <= BF16_TOL
        else:
            assert torch.equal(y, ref), (sched, chunks, lw, gw, two)
    torch.cuda.synchronize()


def test_ep_edge_cases():
    log("ep edge cases")
    T, d, Eg, k, I = 40, 256, 8, 2, 128
    # no peer tokens: every row is a self row
    s = _setup(T, d, Eg, k, I, 2.0, seed=4, peer_T=0)
    assert np.array_equal(host(s["se"]), host(s["off"])[1:])  # no remote rows
    ws = moe.ep_workspace(s["cfg"], s["n_rows"])
    for sched in ("sequential", "self_remote", "expert_chunks"):
        recv = torch.empty((s["n_rows"], d), dtype=torch.bfloat16, device="cuda")
        y = torch.full((s["n_rows"], d), float("nan"), dtype=torch.bfloat16, device="cuda")
        moe.moe_ep_expert_ffn(s["cfg"], sched, s["n_rows"], s["x"], T, s["xp"], 0, s["rt"], s["off"], s["se"],
                              s["gu"], s["dn"], recv, y, ws, chunks=2, s_link=torch.cuda.Stream())
        torch.cuda.synchronize()
        assert max_rel_err(host(y.float()), _oracle_y(s)) <= BF16_TOL
    # a local expert that receives no row (expert 1 never chosen by this rank or the peer)
    rng = np.random.default_rng(9)
    pick = lambda: np.stack([rng.choice([e for e in range(Eg) if e != 1], k, replace=False)
                             for _ in range(T)]).astype(np.int32)
    s = _setup(T, d, Eg, k, I, 2.0, seed=5, topk_self=pick(), topk_peer=pick())
    off = host(s["off"])
    assert off[2] == off[1]
    ws = moe.ep_workspace(s["cfg"], s["n_rows"])
    recv = torch.empty((s["n_rows"], d), dtype=torch.bfloat16, device="cuda")
    y = torch.full((s["n_rows"], d), float("nan"), dtype=torch.bfloat16, device="cuda")
    moe.moe_ep_expert_ffn(s["cfg"], "expert_chunks", s["n_rows"], s["x"], T, s["xp"], T, s["rt"], s["off"], s["se"],
                          s["gu"], s["dn"], recv, y, ws, chunks=4, s_link=torch.cuda.Stream())
    torch.cuda.synchronize()
    assert max_rel_err(host(y.float()), _oracle_y(s)) <= BF16_TOL
    log("  expert 1 rows", off[2] - off[1])
    # zero rows: a no-op
    moe.moe_ep_expert_ffn(s["cfg"], "sequential", 0, s["x"], T, s["xp"], T, s["rt"], s["off"], s["se"], s["gu"],
                          s["dn"], recv, y, ws)
    # invalid arguments
    cfg = s["cfg"]
    bad = [dict(schedule="expert_chunks", chunks=0), dict(schedule="expert_chunks", chunks=17),
           dict(schedule="sequential", link_workgroups=-1)]
    for kw in bad:
        sched = kw.pop("schedule")
        with pytest.raises(moe.MoeError) as e:
            moe.moe_ep_expert_ffn(cfg, sched, s["n_rows"], s["x"], T, s["xp"], T, s["rt"], s["off"], s["se"],
                                  s["gu"], s["dn"], recv, y, ws, **kw)
        assert e.value.status == -1
    with pytest.raises(moe.MoeError) as e:
        moe.moe_expert_ffn_segments(cfg, s["n_rows"], recv, s["off"], None, 1, 0, s["gu"], s["dn"], y, ws)
    assert e.value.status == -1
    with pytest.raises(moe.MoeError) as e:  # row-major weights are not supported here
        moe.moe_expert_ffn_segments(moe.MoeConfig(d=d, E=Eg // 2, k=k, I=I, dtype="bf16"), s["n_rows"], recv,
                                    s["off"], None, 0, 1, s["gu"], s["dn"], y, ws)
    assert e.value.status == -2
    with pytest.raises(moe.MoeError) as e:
        moe.moe_ep_copy_rows(cfg, 2, s["n_rows"], s["x"], T, s["rt"], s["off"], s["se"], 0, 1, recv)
    assert e.value.status == -1


def test_ep_full_size_sampled():
    """The benchmark's configuration: DeepSeek-V3 layer (d 7168, I 2048) split
    over two GPUs, this one owning 128 of the 256 experts, 4096 tokens per
    rank, imbalance 3:1; the chunked and split schedules against the
    sequential one (same bits) and sampled rows against the oracle."""
    T, d, Eg, k, I, r = 4096, 7168, 256, 8, 2048, 3.0
    log("ep full size", T, d, Eg, k, I, r)
    s = _setup(T, d, Eg, k, I, r)
    n, E = s["n_rows"], s["E"]
    log("  rows", n)
    ws = moe.ep_workspace(s["cfg"], n)
    link = torch.cuda.Stream()
    outs = {}
    for sched, chunks in (("sequential", 1), ("self_remote", 1), ("expert_chunks", 4)):
        recv = torch.empty((n, d), dtype=torch.bfloat16, device="cuda")
        y = torch.full((n, d), float("nan"), dtype=torch.bfloat16, device="cuda")
        moe.moe_ep_expert_ffn(s["cfg"], sched, n, s["x"], T, s["xp"], T, s["rt"], s["off"], s["se"], s["gu"],
                              s["dn"], recv, y, ws, chunks=chunks, link_workgroups=8,
                              gemm_workgroups=248, s_link=link)
        torch.cuda.synchronize()
        outs[sched] = y
        del recv
    assert torch.equal(outs["sequential"], outs["self_remote"])
    assert torch.equal(outs["sequential"], outs["expert_chunks"])
    assert not torch.isnan(outs["sequential"]).any(), "rows left unwritten"
    off, se = host(s["off"]), host(s["se"])
    rows = []
    for e in (0, 1, 63, 127):
        rows += [int(off[e]), int(se[e]) - 1, int(se[e]), int(off[e + 1]) - 1]  # first/last self and remote rows
    rows = sorted(set(rows))
    want = _oracle_y(s, rows=rows)
    got = host(outs["sequential"][rows].float())
    err = max_rel_err(got, want)
    log("  sampled max_rel_err", err)
    assert err <= BF16_TOL
    # two whole experts (their self and remote rows: every pass and column tile)
    for e in (0, int(np.argmax(np.diff(off)))):
        seg = np.arange(int(off[e]), int(off[e + 1]))
        want = _oracle_y(s, rows=seg)
        got = host(outs["sequential"][int(off[e]):int(off[e + 1])].float())
        err = max_rel_err(got, want)
        log(f"  expert {e}: {seg.size} rows, max_rel_err {err:.3e}")
        assert err <= BF16_TOL
    del outs
    torch.cuda.empty_cache()
