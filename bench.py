"""Benchmark of the MoE-layer hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload dsv3]

A step is one moe_layer call (gate, route, dispatch, grouped expert FFN with
the shared expert, combine) over the workload's T tokens, with inputs and
weights already resident in HBM. By default the routed-expert weights are
converted once, before any timing, into the packed layout of
moe_pack_weights (a load-time conversion, like reading a checkpoint); the
weight-streaming expert GEMMs then read them, and the shared expert runs
inside them as one more group. --layout rowmajor times the tiled GEMMs on
the plain [E][I][d] weights instead. Prints ONE JSON line: tokens/s of the
layer, the roofline of the dominant kernel pair (the grouped expert FFN,
timed with HIP events on its own stream), the CPU oracle timed on the same
workload (all tokens routed and combined, a seeded subset of whole experts
run and the rest of the expert FFN scaled from them) as a baseline, the per-layer time of 1, 4 and 16
layer calls run back to back, the layer with the shared expert inside the
routed GEMMs against the same layer composed from the public calls with the
shared expert on one or two streams, the receive side of two-GPU expert parallelism
under the three schedules of moe_ep_expert_ffn for imbalance ratios 2:1 to
5:1 (the exchange emulated by a copy with a fixed workgroup budget), and side
measurements of the skewed-routing, decode-sized and Mixtral-shaped
workloads (--no-extra skips these).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix cores
METRIC = "MoE layer tokens/s at DeepSeek-V3 shape; % bf16 MFMA peak / % HBM BW"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def algorithmic(p: dict, counts) -> dict:
    """Algorithmic bytes and flops (activated experts only, each byte once)."""
    T, d, E, k, I = p["T"], p["d"], p["E"], p["k"], p["I"]
    es = 2 if p["dtype"] == "bf16" else 4
    touched = int((counts > 0).sum())
    w_expert = 3 * I * d * es
    ffn_bytes = touched * w_expert + T * d * es + T * k * d * es       # weights + x in + y_perm out
    ffn_flops = 6.0 * T * k * d * I
    Is = p.get("I_shared", 0) if p.get("n_shared", 0) else 0
    layer_bytes = touched * w_expert + 3 * Is * d * es + E * d * es + 2 * T * d * es
    layer_flops = 2.0 * T * d * E + ffn_flops + 6.0 * T * d * Is
    return dict(touched_experts=touched, ffn_bytes=ffn_bytes, ffn_flops=ffn_flops, layer_bytes=layer_bytes,
                layer_flops=layer_flops, bytes_per_expert=w_expert)


GEMM_SOURCES = {"packed": ("gemm_stream.hip", "gemm_dense.hip"), "rowmajor": ("gemm_bf16.hip",)}


def kernel_source_hash(layout: str = "packed") -> str:
    """Hash of the expert-GEMM kernel sources of a weight layout: a traffic
    record taken on other sources is not reported."""
    h = hashlib.sha256()
    for f in GEMM_SOURCES[layout]:
        with open(os.path.join(ROOT, "paper_2603_02376_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(workload: str, layout: str):
    """HBM bytes per expert-FFN call from the rocprofv3 counter runs committed
    under profiles/, or None when absent or taken on another kernel source."""
    path = os.path.join(ROOT, "profiles", f"traffic_expert_ffn_{workload}_{layout}.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("kernel_source_hash") != kernel_source_hash(layout):
        return None
    return rec.get("bytes_per_call")


CPU_EXPERTS = 0  # whole experts the CPU baseline runs (0: every touched expert, i.e. the whole layer)
EP_LINK_WORKGROUPS = 16  # workgroups of the emulated exchange (~77 GB/s measured: about one xGMI link, one way)
EP_CHUNKS = (4, 8, 16)


def ep_split(p: dict, x, gate_up, down, steps: int, warmup: int) -> dict:
    """Receive side of two-GPU expert parallelism (App. M; §4.3, Table 5) on
    one GPU: this GPU owns experts [0, E/2) of the workload, each rank has T
    tokens, and a fraction r/(r+1) of all assignments goes to this GPU's
    experts (r = 2..5). The remote rows arrive through a copy limited to
    EP_LINK_WORKGROUPS workgroups on its own stream (the emulated link); the
    expert GEMMs keep the other compute units while rows still arrive.
    Times moe_ep_expert_ffn under each schedule, plus the link and the FFN
    alone, and the FFN of the self rows and of the remote rows as two calls
    (the split's two passes over every expert's weights)."""
    import torch

    from paper_2603_02376_amd import inputs, moe

    T, d, Eg, k, I = p["T"], p["d"], p["E"], p["k"], p["I"]
    E = Eg // 2
    cfg = moe.MoeConfig(d=d, E=E, k=k, I=I, dtype="bf16", weight_layout="packed")
    gcfg = moe.MoeConfig(d=d, E=Eg, k=k, I=I, dtype="bf16")
    xp = torch.from_numpy(inputs.ep_peer_tokens(T, d)).to(device="cuda", dtype=torch.bfloat16)
    s_c = torch.cuda.current_stream()
    link = torch.cuda.Stream()
    gemm_wg = torch.cuda.get_device_properties(0).multi_processor_count - EP_LINK_WORKGROUPS // 2
    gemm_wg -= gemm_wg % 8
    n_steps = max(3, min(steps, 10))

    def timed(fn):
        for _ in range(max(2, warmup // 2)):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(s_c)
        for _ in range(n_steps):
            fn()
        b.record(s_c)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / n_steps

    def dispatch(tk):
        ws = moe.alloc_workspace(gcfg, T)
        z = lambda m: torch.empty(m, dtype=torch.int32, device="cuda")
        c, o, st, sa, inv = z(Eg), z(Eg + 1), z(T * k), z(T * k), z(T * k)
        moe.moe_dispatch(gcfg, T, torch.from_numpy(tk).cuda(), c, o, st, sa, inv, ws)
        return o, st

    ratios = []
    link_gbs = []
    for r in inputs.EP_RATIOS:
        so, ss = dispatch(inputs.ep_topk(T, Eg, k, r, "self"))
        po, ps = dispatch(inputs.ep_topk(T, Eg, k, r, "peer"))
        n_self, n = int(so[E].item()), int(so[E].item()) + int(po[E].item())
        rt = torch.empty(n, dtype=torch.int32, device="cuda")
        off = torch.empty(E + 1, dtype=torch.int32, device="cuda")
        se = torch.empty(E, dtype=torch.int32, device="cuda")
        moe.moe_ep_plan(cfg, 0, so, ss, T * k, po, ps, T * k, rt, n, off, se)
        recv = torch.empty((n, d), dtype=torch.bfloat16, device="cuda")
        y = torch.empty_like(recv)
        ws = moe.ep_workspace(cfg, n)
        remote_bytes = (n - n_self) * d * 2

        def run(sched, chunks=1):
            moe.moe_ep_expert_ffn(cfg, sched, n, x, T, xp, T, rt, off, se, gate_up, down, recv, y, ws,
                                  chunks=chunks, link_workgroups=EP_LINK_WORKGROUPS, gemm_workgroups=gemm_wg,
                                  s_compute=s_c, s_link=link)

        link_ms = timed(lambda: moe.moe_ep_copy_rows(cfg, moe.MOE_EP_REMOTE, n, xp, T, rt, off, se, 0, E, recv,
                                                     max_workgroups=EP_LINK_WORKGROUPS, stream=s_c))
        link_gbs.append(remote_bytes / (link_ms / 1e3) / 1e9)
        ffn_all = timed(lambda: moe.moe_expert_ffn_segments(cfg, n, recv, off, None, 0, E, gate_up, down, y, ws,
                                                            stream=s_c))
        ffn_two = timed(lambda: (moe.moe_expert_ffn_segments(cfg, n, recv, off, se, 0, E, gate_up, down, y, ws,
                                                             stream=s_c),
                                 moe.moe_expert_ffn_segments(cfg, n, recv, se, off[1:], 0, E, gate_up, down, y, ws,
                                                             stream=s_c)))
        seq = timed(lambda: run("sequential"))
        split = timed(lambda: run("self_remote"))
        chunked = {c: timed(lambda c=c: run("expert_chunks", c)) for c in EP_CHUNKS}
        best_c = min(chunked, key=chunked.get)
        ratios.append(dict(
            ratio=f"{r}:1", rows=n, self_rows=n_self, remote_rows=n - n_self,
            remote_mb=round(remote_bytes / 1e6, 1), link_ms=round(link_ms, 3),
            ffn_all_rows_ms=round(ffn_all, 3), ffn_self_then_remote_ms=round(ffn_two, 3),
            sequential_ms=round(seq, 3), self_remote_ms=round(split, 3),
            expert_chunks_ms={str(c): round(v, 3) for c, v in chunked.items()},
            self_remote_speedup=round(seq / split, 3), expert_chunks_speedup=round(seq / chunked[best_c], 3),
            best_chunks=best_c))
        del recv, y, ws, rt
        torch.cuda.empty_cache()
    return dict(local_experts=E, tokens_per_rank=T, link_workgroups=EP_LINK_WORKGROUPS,
                link_gbs=round(sum(link_gbs) / len(link_gbs), 1), gemm_workgroups=gemm_wg, ratios=ratios,
                note="one GPU of a two-GPU expert-parallel pair; the exchange of remote rows is a copy limited to "
                     "link_workgroups workgroups on its own stream; speedups are over the sequential schedule")


def run_workload(name: str, steps: int, warmup: int, want_cpu: bool, cpu_experts: int = CPU_EXPERTS,
                 ffn_only: bool = False, layout: str = "packed", multilayer: tuple = (), int8: bool = False,
                 ep: bool = False):
    import numpy as np
    import torch

    from paper_2603_02376_amd import inputs, moe

    p = inputs.preset(name)
    cfg = moe.MoeConfig(d=p["d"], E=p["E"], k=p["k"], I=p["I"], n_groups=p["n_groups"],
                        topk_groups=p["topk_groups"], n_shared=p["n_shared"], I_shared=p["I_shared"],
                        score=p["score"], renorm=p["renorm"], scale=p["scale"], dtype=p["dtype"],
                        weight_layout=layout)
    T = p["T"]
    log(f"[bench] {name}: generating inputs on device")
    t = inputs.make_inputs(p, 0, "cuda")
    w_ffn = (t["w_gate"], t["w_up"], t["w_down"])
    w_sh = (t["ws_gate"], t["ws_up"], t["ws_down"])
    if cfg.packed:  # one-time load-time conversion, outside every timed region
        gu, dn = moe.pack_weights(cfg, *w_ffn)
        w_ffn = (gu, None, dn)
        if p["n_shared"]:
            sg, sd = moe.pack_shared_weights(cfg, *w_sh)
            w_sh = (sg, None, sd)
    ws = moe.alloc_workspace(cfg, T)
    out = torch.empty((T, p["d"]), dtype=cfg.torch_dtype, device="cuda")
    s_main = torch.cuda.current_stream()
    s_aux = torch.cuda.Stream()

    def layer(dbg=None):
        moe.moe_layer(cfg, T, t["x"], t["w_router"], t["bias"], *w_ffn, *w_sh, out, ws, s_main=s_main, s_aux=s_aux, dbg=dbg)

    # untimed call that exports the routing, for the algorithmic byte count
    dbg = dict(counts=torch.empty(p["E"], dtype=torch.int32, device="cuda"),
               offsets=torch.empty(p["E"] + 1, dtype=torch.int32, device="cuda"),
               sorted_token=torch.empty(T * p["k"], dtype=torch.int32, device="cuda"),
               topk_idx=torch.empty((T, p["k"]), dtype=torch.int32, device="cuda"),
               topk_w=torch.empty((T, p["k"]), dtype=torch.float32, device="cuda"),
               logits=torch.empty((T, p["E"]), dtype=torch.float32, device="cuda"))
    layer(dbg)
    torch.cuda.synchronize()
    counts = dbg["counts"].cpu().numpy()
    alg = algorithmic(p, counts)

    ms = wall = float("nan")
    if not ffn_only:
        for _ in range(warmup):
            layer()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        log(f"[bench] {name}: timing {steps} layer steps")
        wall0 = time.perf_counter()
        e0.record(s_main)
        for _ in range(steps):
            layer()
        e1.record(s_main)
        torch.cuda.synchronize()
        wall = time.perf_counter() - wall0
        ms = e0.elapsed_time(e1) / steps

    # multi-layer steady state: L layer calls back to back on the same input
    # and weights (feeding each output to the next layer would change the
    # routing, hence the work, from layer to layer), each into its own output
    ml = {}
    if multilayer and not ffn_only:
        outs = [torch.empty_like(out) for _ in range(max(multilayer))]

        def chain(L):
            for i in range(L):
                moe.moe_layer(cfg, T, t["x"], t["w_router"], t["bias"], *w_ffn, *w_sh, outs[i], ws,
                              s_main=s_main, s_aux=s_aux)

        for L in multilayer:
            chain(L)
            reps = max(1, steps // L)
            m0, m1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            m0.record(s_main)
            for _ in range(reps):
                chain(L)
            m1.record(s_main)
            torch.cuda.synchronize()
            ml[L] = m0.elapsed_time(m1) / (reps * L)
        del outs

    # dominant kernel pair: the grouped expert FFN, timed alone on its stream
    y = torch.empty((T * p["k"], p["d"]), dtype=cfg.torch_dtype, device="cuda")

    def ffn():
        moe.moe_expert_ffn(cfg, T, t["x"], dbg["sorted_token"], dbg["offsets"], *w_ffn, y, ws, stream=s_main)

    log(f"[bench] {name}: timing {steps} expert-FFN calls")
    for _ in range(max(2, warmup)):
        ffn()
    torch.cuda.synchronize()
    f0, f1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    f0.record(s_main)
    for _ in range(steps):
        ffn()
    f1.record(s_main)
    torch.cuda.synchronize()
    ffn_ms = f0.elapsed_time(f1) / steps

    # quantized tokens (the pipeline's quantize-before-dispatch, int8 and
    # FP8): the quantize kernel, the expert FFN on the codes and the layer
    # with quantized tokens
    qres = {}
    if int8 and cfg.packed and not ffn_only:
        import dataclasses

        def timed(fn, n):
            for _ in range(max(2, warmup)):
                fn()
            torch.cuda.synchronize()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(s_main)
            for _ in range(n):
                fn()
            b.record(s_main)
            torch.cuda.synchronize()
            return a.elapsed_time(b) / n

        for mode in ("int8", "fp8"):
            codes = torch.empty((T, p["d"]), dtype=torch.uint8, device="cuda")
            scales = torch.empty(T, dtype=torch.float32, device="cuda")
            cfgq = dataclasses.replace(cfg, token_quant=mode)
            wsq = moe.alloc_workspace(cfgq, T)
            q_ms = timed(lambda: moe.moe_quantize(cfgq, T, t["x"], codes, scales, stream=s_main), steps)
            fq_ms = timed(lambda: moe.moe_expert_ffn_q8(cfgq, T, codes, scales, dbg["sorted_token"], dbg["offsets"],
                                                         w_ffn[0], w_ffn[2], y, wsq, stream=s_main), steps)
            lq_ms = timed(lambda: moe.moe_layer(cfgq, T, t["x"], t["w_router"], t["bias"], *w_ffn, *w_sh, out, wsq,
                                                s_main=s_main, s_aux=s_aux), steps)
            # token bytes the GEMM1 operand loads gather (every column tile reads its rows again)
            nt1 = p["I"] // 128
            rows = T * p["k"]
            qres[mode] = dict(quantize_ms=round(q_ms, 4), expert_ffn_ms=round(fq_ms, 4),
                              expert_ffn_speedup=round(ffn_ms / fq_ms, 4), layer_ms=round(lq_ms, 4),
                              tokens_per_s=round(T / (lq_ms / 1e3), 1),
                              gathered_token_bytes_gemm1={"bf16": nt1 * rows * p["d"] * 2,
                                                          mode: nt1 * rows * p["d"]},
                              note="layer with quantized tokens runs the shared expert's GEMM1 on its own (bf16 input) and its GEMM2 inside the routed GEMM2")
            del codes, scales, wsq

    # where the shared expert runs: inside the routed GEMMs (moe_layer with
    # packed weights), or as its own FFN composed from the public calls, on
    # the routing stream after the routed FFN, or on a second stream forked
    # before the router GEMM (the paper's two-stream overlap: it runs beside
    # routing, dispatch and the routed FFN; the combine waits for it)
    sh_res = None
    if ep and cfg.packed and p["n_shared"] and not ffn_only:
        log(f"[bench] {name}: shared expert fused vs composed on one or two streams")
        E, k = p["E"], p["k"]
        i32 = dict(dtype=torch.int32, device="cuda")
        b = dict(logits=torch.empty((T, E), dtype=torch.float32, device="cuda"),
                 idx=torch.empty((T, k), **i32), w=torch.empty((T, k), dtype=torch.float32, device="cuda"),
                 counts=torch.empty(E, **i32), offsets=torch.empty(E + 1, **i32), st=torch.empty(T * k, **i32),
                 inv=torch.empty(T * k, **i32), y=torch.empty((T * k, p["d"]), dtype=cfg.torch_dtype, device="cuda"),
                 sh=torch.empty((T, p["d"]), dtype=cfg.torch_dtype, device="cuda"), out=torch.empty_like(out))
        fork, join = torch.cuda.Event(), torch.cuda.Event()

        def shared(stream):
            moe.moe_shared_ffn(cfg, T, t["x"], *w_sh, b["sh"], ws, stream=stream)

        def composed(two):
            if two:
                fork.record(s_main)
                s_aux.wait_event(fork)
                shared(s_aux)
                join.record(s_aux)
            moe.moe_route(cfg, T, t["x"], t["w_router"], t["bias"], b["logits"], b["idx"], b["w"], ws, stream=s_main)
            moe.moe_dispatch(cfg, T, b["idx"], b["counts"], b["offsets"], b["st"], None, b["inv"], ws, stream=s_main)
            moe.moe_expert_ffn(cfg, T, t["x"], b["st"], b["offsets"], *w_ffn, b["y"], ws, stream=s_main)
            if two:
                s_main.wait_event(join)
            else:
                shared(s_main)
            moe.moe_combine(cfg, T, b["y"], b["inv"], b["w"], b["sh"], b["out"], stream=s_main)

        def timed_main(fn):
            for _ in range(max(2, warmup)):
                fn()
            torch.cuda.synchronize()
            a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(s_main)
            for _ in range(steps):
                fn()
            z.record(s_main)
            torch.cuda.synchronize()
            return a.elapsed_time(z) / steps

        one_ms = timed_main(lambda: composed(False))
        two_ms = timed_main(lambda: composed(True))
        sh_ms = timed_main(lambda: shared(s_main))
        layer()
        torch.cuda.synchronize()
        sh_res = dict(fused_layer_ms=round(ms, 4), composed_one_stream_ms=round(one_ms, 4),
                      composed_two_streams_ms=round(two_ms, 4), shared_ffn_alone_ms=round(sh_ms, 4),
                      routed_ffn_alone_ms=round(ffn_ms, 4), outputs_identical=bool(torch.equal(out, b["out"])),
                      note="composed: moe_route, moe_dispatch, moe_expert_ffn, moe_shared_ffn and moe_combine; "
                           "two streams: the shared FFN on a second stream from the start, joined before the combine")
        del b

    ep_res = None
    if ep and cfg.packed and not ffn_only and p["E"] % 2 == 0 and p["dtype"] == "bf16":
        log(f"[bench] {name}: expert-parallel receive side, ratios {inputs.EP_RATIOS}")
        ep_res = ep_split(p, t["x"], w_ffn[0], w_ffn[2], steps, warmup)

    res = dict(
        name=name, p=p, ms=ms, wall_s=wall, tokens_per_s=T / (ms / 1e3), alg=alg, ffn_ms=ffn_ms,
        int8_tokens=qres.get("int8"), fp8_tokens=qres.get("fp8"),
        ep_split=ep_res, shared_expert=sh_res,
        counts_max_over_mean=float(counts.max() / counts.mean()), empty_experts=int((counts == 0).sum()),
        layer_hbm_frac=alg["layer_bytes"] / (ms / 1e3) / (HBM_PEAK_GBS * 1e9),
        layer_mfma_frac=alg["layer_flops"] / (ms / 1e3) / (MFMA_BF16_PEAK_TFLOPS * 1e12),
        ffn_gbs=alg["ffn_bytes"] / (ffn_ms / 1e3) / 1e9,
        ffn_tflops=alg["ffn_flops"] / (ffn_ms / 1e3) / 1e12,
        # fraction of the FFN's roofline: the larger of its byte and flop floors over its time
        ffn_roof_frac=max(alg["ffn_bytes"] / (HBM_PEAK_GBS * 1e9), alg["ffn_flops"] / (MFMA_BF16_PEAK_TFLOPS * 1e12))
        / (ffn_ms / 1e3),
        multilayer_ms_per_layer=ml,
    )
    if want_cpu:
        log(f"[bench] {name}: CPU oracle baseline ({cpu_experts or 'all'} whole experts, all tokens routed)")
        res["cpu"] = cpu_baseline(p, t, cpu_experts)
    del t, ws, out, y, w_ffn, w_sh
    torch.cuda.empty_cache()
    return res


def cpu_baseline(p, t, n_experts: int = CPU_EXPERTS):
    """The oracle, as it stands, timed on the host cores over the whole
    workload's routing and a seeded subset of whole experts: gate logits and
    routing of all T tokens, dispatch, the SwiGLU FFN of every row of
    n_experts of the touched experts (a seeded choice; n_experts <= 0: every
    touched expert, the whole layer, the default), the shared expert on
    all T tokens, and the combine of all tokens, everything in fp64. The
    expert-FFN time is scaled by touched / n_experts (every touched expert of
    a uniformly routed workload has about the same rows); the rest is timed
    whole. The sampled experts' weights are copied to host RAM before the
    clock starts (their bf16 -> fp64 conversion is timed)."""
    import numpy as np

    from oracle import moe_oracle as O
    from paper_2603_02376_amd import inputs

    T, E = p["T"], p["E"]
    x = inputs.oracle_view(t["x"])
    wr = inputs.oracle_view(t["w_router"])
    bias = None if p["score"] == "softmax" else inputs.oracle_view(t["bias"])
    kw = dict(k=p["k"], score=p["score"], bias=bias, n_groups=p["n_groups"], topk_groups=p["topk_groups"],
              renorm=p["renorm"], scale=p["scale"])
    # the sampled experts: routed once before the clock starts, their weights copied to host RAM
    touched = np.nonzero(O.dispatch(O.route(O.gate_logits(x, wr), **kw)[0], E)[0])[0]
    rng = np.random.default_rng(0)
    n_pick = touched.size if n_experts <= 0 else min(n_experts, touched.size)
    chosen = np.sort(rng.choice(touched, n_pick, replace=False))
    host_w = {n: {int(e): inputs.oracle_view(t[n][int(e)]) for e in chosen} for n in ("w_gate", "w_up", "w_down")}
    sh = [inputs.oracle_view(t[n]) for n in ("ws_gate", "ws_up", "ws_down")] if p["n_shared"] else None

    t0 = time.perf_counter()
    idx, w = O.route(O.gate_logits(x, wr), **kw)
    counts, offsets, st, _, inv = O.dispatch(idx, E)
    t1 = time.perf_counter()
    y = np.zeros((int(offsets[-1]), p["d"]))   # rows of the experts not run stay 0 (their time is scaled in)
    for e in chosen:
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        y[lo:hi] = O.swiglu_ffn(x[st[lo:hi]], host_w["w_gate"][int(e)], host_w["w_up"][int(e)],
                                host_w["w_down"][int(e)])
    t2 = time.perf_counter()
    shared = O.swiglu_ffn(x, *sh) if sh else None
    O.combine(y, inv, w, shared)
    t3 = time.perf_counter()
    n_touched = int((counts > 0).sum())
    est = (t1 - t0) + (t2 - t1) * n_touched / len(chosen) + (t3 - t2)
    blas, threads = "unknown", None
    try:
        from threadpoolctl import threadpool_info

        info = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        if info:
            blas = f"{info[0].get('internal_api')} {info[0].get('version')} ({info[0].get('architecture')})"
            threads = info[0].get("num_threads")
    except Exception:
        pass
    return dict(value=T / est, unit="tokens/s", cores=threads or len(os.sched_getaffinity(0)),
                host_cpus=len(os.sched_getaffinity(0)), blas=blas, kind="oracle", seconds_timed=t3 - t0,
                seconds_layer_estimate=est,
                sample=(f"the whole {p.get('name')} layer (T={T}): gate, routing, dispatch, the SwiGLU FFN of all "
                        f"{n_touched} touched experts{', the shared expert' if sh else ''} and the combine of all {T} "
                        f"tokens, in fp64" if len(chosen) == n_touched else
                        f"the {p.get('name')} workload (T={T}): gate, routing, dispatch and combine of all {T} tokens"
                        f"{', the shared expert on all of them' if sh else ''}, and the SwiGLU FFN of every row of "
                        f"{len(chosen)} of the {n_touched} touched experts (seeded choice), in fp64; the expert-FFN "
                        f"time scaled by {n_touched}/{len(chosen)} to the whole layer"))


def library_gemm_reference(steps: int, warmup: int) -> dict:
    """Reference only, not part of the measured path: the vendor library
    (torch.matmul, hipBLASLt) on the Mixtral-shaped GEMM1 (d = 4096 into
    2 x 14336 gate and up columns, bf16), for one expert's 1,024 rows, for
    all 8,192 routed rows through one weight matrix, and for the 8 experts'
    1,024-row GEMMs batched (the grouped problem the expert FFN solves)."""
    import torch

    g = torch.Generator(device="cuda")
    g.manual_seed(7)
    d, n, rows, E = 4096, 2 * 14336, 1024, 8
    a = torch.randn((E, rows, d), generator=g, device="cuda").to(torch.bfloat16)
    b = (torch.randn((E, d, n), generator=g, device="cuda") * 0.02).to(torch.bfloat16)  # contiguous, not a view
    out = {}
    cases = {"one_expert": (lambda: torch.matmul(a[0], b[0]), 2.0 * rows * d * n),
             "all_rows_one_weight": (lambda: torch.matmul(a.view(E * rows, d), b[0]), 2.0 * E * rows * d * n),
             "grouped_8_experts": (lambda: torch.matmul(a, b), 2.0 * E * rows * d * n)}
    for key, (fn, flops) in cases.items():
        for _ in range(warmup):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        out[key + "_tflops"] = round(flops / (ms * 1e-3) / 1e12, 1)
    del a, b
    torch.cuda.empty_cache()
    out["note"] = ("torch.matmul (hipBLASLt) on the Mixtral GEMM1 shape (d 4096 -> 2 x 14336, bf16), same run, for "
                   "reference: one expert's 1,024 rows; all 8,192 routed rows through one weight; the 8 experts' "
                   "GEMMs batched")
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="dsv3")
    ap.add_argument("--layout", choices=("packed", "rowmajor"), default="packed",
                    help="routed-expert weight layout (packed: converted once before timing)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true", help="skip the side measurements (other workloads, multi-layer)")
    ap.add_argument("--cpu-experts", type=int, default=CPU_EXPERTS,
                    help="whole experts the CPU-oracle baseline runs, the rest of its expert FFN scaled (0: all)")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="first run 3 plain device copies of this many MiB (reference for HBM byte counters)")
    ap.add_argument("--library-gemm-only", action="store_true",
                    help="only time the vendor-library reference GEMM1 at the Mixtral shape (for profiling it)")
    ap.add_argument("--ffn-only", action="store_true",
                    help="profiling aid: run only the timed expert-FFN loop of the workload and print its timing")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}): the layer is one GPU's share of the "
              "expert-parallel MoE layer and no multi-GPU path is built", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2603_02376_amd import moe

    moe.lib()  # fail loudly if the HIP library is missing
    torch.cuda.set_device(0)
    if args.library_gemm_only:
        print(json.dumps(dict(library_gemm1=library_gemm_reference(args.steps, args.warmup))))
        return
    if args.copy_calibration_mb:
        n = args.copy_calibration_mb << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        c0.record()
        for _ in range(3):
            dst.copy_(src)
        c1.record()
        torch.cuda.synchronize()
        log(f"[bench] copy calibration: 3 x {n} B, {2 * 3 * n / (c0.elapsed_time(c1) / 1e3) / 1e9:.1f} GB/s")
        del src, dst
    main_res = run_workload(args.workload, args.steps, args.warmup, not args.no_cpu_baseline, args.cpu_experts,
                            args.ffn_only, args.layout, multilayer=() if args.no_extra else (1, 4, 16),
                            int8=not args.no_extra, ep=not args.no_extra)
    if args.ffn_only:
        print(json.dumps(dict(workload=args.workload, expert_ffn_ms=main_res["ffn_ms"],
                              expert_ffn_gbs=main_res["ffn_gbs"], expert_ffn_tflops=main_res["ffn_tflops"])))
        return
    extra = {}
    if not args.no_extra:
        for name in ("dsv3_skew", "dsv3_decode", "mixtral"):
            if name == args.workload:
                continue
            r = run_workload(name, args.steps, args.warmup, False, layout=args.layout, int8=name == "dsv3_decode")
            extra[name] = dict(tokens_per_s=round(r["tokens_per_s"], 1), ms_per_step=round(r["ms"], 4),
                               layer_hbm_frac=round(r["layer_hbm_frac"], 4),
                               layer_mfma_frac=round(r["layer_mfma_frac"], 4),
                               expert_ffn_ms=round(r["ffn_ms"], 4), expert_ffn_gbs=round(r["ffn_gbs"], 1),
                               expert_ffn_tflops=round(r["ffn_tflops"], 1),
                               expert_ffn_roofline_frac=round(r["ffn_roof_frac"], 4),
                               touched_experts=r["alg"]["touched_experts"],
                               max_over_mean_load=round(r["counts_max_over_mean"], 3), empty_experts=r["empty_experts"])
            for key in ("int8_tokens", "fp8_tokens"):
                if r[key]:
                    extra[name][key] = r[key]
            if name == "mixtral":
                log("[bench] mixtral: library GEMM reference")
                extra[name]["library_gemm1"] = library_gemm_reference(args.steps, args.warmup)

    r = main_res
    p = r["p"]
    alg = r["alg"]
    hbm_bound = alg["ffn_flops"] / alg["ffn_bytes"] < (MFMA_BF16_PEAK_TFLOPS * 1e12) / (HBM_PEAK_GBS * 1e9)
    if hbm_bound:
        roof = dict(bound="hbm", achieved=round(r["ffn_gbs"], 1), peak=HBM_PEAK_GBS, unit="GB/s",
                    frac=round(r["ffn_gbs"] / HBM_PEAK_GBS, 4))
    else:
        roof = dict(bound="mfma", achieved=round(r["ffn_tflops"], 1), peak=MFMA_BF16_PEAK_TFLOPS, unit="TFLOP/s",
                    frac=round(r["ffn_tflops"] / MFMA_BF16_PEAK_TFLOPS, 4))
    roof["traffic"] = measured_traffic(args.workload, args.layout)
    kern = ("weight-streaming GEMM1+SwiGLU then GEMM2 over packed weights, one launch per call"
            if args.layout == "packed" else "tiled grouped GEMM1+SwiGLU and GEMM2 over row-major weights, "
            "2 launches per call")
    roof.update(kernel=f"moe_expert_ffn: {kern}",
                ms_per_call=round(r["ffn_ms"], 4), algorithmic_bytes=alg["ffn_bytes"],
                algorithmic_flops=alg["ffn_flops"], touched_experts=alg["touched_experts"])
    out = {
        "metric": METRIC,
        "value": round(r["tokens_per_s"], 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(r["ms"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": p["dtype"],
        "data": "synthetic (seeded; random-init weights of the workload's shape)",
        "config": {"workload": (f"{args.workload}: T={p['T']} d={p['d']} E={p['E']} top-{p['k']}"
                                + (f" (top-{p['topk_groups']} of {p['n_groups']} groups)" if p["n_groups"] > 1 else "")
                                + f" I={p['I']}" + (f" + shared I={p['I_shared']}" if p["n_shared"] else "")
                                + f", {args.layout} expert weights"),
                   "global_batch": p["T"], "parallelism": "single GPU (one GPU's share of expert parallelism)"},
        "layer_hbm_frac": round(r["layer_hbm_frac"], 4),
        "layer_mfma_frac": round(r["layer_mfma_frac"], 4),
        "routing": {"max_over_mean_load": round(r["counts_max_over_mean"], 3), "empty_experts": r["empty_experts"]},
        "roofline": roof,
    }
    if "cpu" in r:
        out["cpu_baseline"] = {k: (round(v, 3) if isinstance(v, float) else v) for k, v in r["cpu"].items()}
    for key in ("int8_tokens", "fp8_tokens"):
        if r[key]:
            out[key] = r[key]
    if r["multilayer_ms_per_layer"]:
        out["multilayer"] = {"ms_per_layer": {str(L): round(v, 4) for L, v in r["multilayer_ms_per_layer"].items()},
                             "note": "L layer calls back to back on the same input and weights, each into its own output"}
    if r["shared_expert"]:
        out["shared_expert"] = r["shared_expert"]
    if r["ep_split"]:
        out["ep_split"] = r["ep_split"]
    if extra:
        out["extra"] = extra
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
