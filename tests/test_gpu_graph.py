"""moe_layer captured in a HIP graph (torch.cuda.CUDAGraph) and replayed.

The layer's launches contain no allocation, copy, memset or host
synchronisation, so a caller can capture a whole layer call (both streams of
the two-stream form: the library forks the second stream from the first with
an event and joins it back) and replay it. Each replay reads the current
contents of the captured input, so the test changes the input between
replays, runs eager layer calls on another workspace in between, and requires
every replay to equal, bit for bit, the eager call on the same input.
"""
import pytest
import torch

from paper_2603_02376_amd import inputs, moe
from tests import gpu_util as G

pytestmark = pytest.mark.gpu

_DSV3_LIKE = dict(T=300, d=512, E=32, k=4, n_groups=4, topk_groups=2, I=256, n_shared=1, I_shared=256,
                  score="sigmoid", renorm=True, scale=2.5, dtype="bf16", bias="zipf")

FORMS = {
    # packed weights: the one-launch FFN with the shared expert fused in
    "packed_fused": dict(_DSV3_LIKE, weight_layout="packed"),
    # packed weights, the shared expert as its own FFN on the second stream
    "packed_two_streams": dict(_DSV3_LIKE, I_shared=128, weight_layout="packed"),
    # int8 tokens: quantize kernel, GEMM1 on codes, the shared GEMM1 on its own
    "packed_int8": dict(_DSV3_LIKE, weight_layout="packed", token_quant="int8"),
    # row-major weights: the tiled GEMMs, the shared expert on the second stream
    "rowmajor": dict(_DSV3_LIKE, I_shared=384),
    # groups of ~515 rows: the compute-bound kernel, GEMM2 at K = 8192 with its
    # remainder blocks split over K and summed by a second kernel
    "packed_dense_split": dict(T=1030, d=256, E=4, k=2, n_groups=1, topk_groups=1, I=8192, n_shared=0, I_shared=0,
                               score="softmax", renorm=True, scale=1.0, dtype="bf16", bias="none",
                               weight_layout="packed"),
    # a decode-sized batch
    "packed_decode": dict(T=5, d=512, E=64, k=6, n_groups=8, topk_groups=3, I=128, n_shared=1, I_shared=128,
                          score="sigmoid", renorm=True, scale=2.5, dtype="bf16", bias="zero", weight_layout="packed"),
}
REPLAYS = 4


@pytest.mark.parametrize("form", list(FORMS))
def test_layer_graph_replays_match_eager(form):
    p = FORMS[form]
    G.log("graph", form)
    cfg = G.moe_cfg(p)
    T, d = p["T"], p["d"]
    t = G.device_inputs(p, seed=11)
    xs = [torch.from_numpy(inputs.host_activations(p, seed=200 + i)[0]).to(device="cuda", dtype=cfg.torch_dtype)
          for i in range(REPLAYS)]
    wg, wu, wd = t["w_gate"], t["w_up"], t["w_down"]
    sg, su, sd = t.get("ws_gate"), t.get("ws_up"), t.get("ws_down")
    if cfg.packed:
        wg, wd = moe.pack_weights(cfg, wg, wu, wd)
        wu = None
        if p.get("n_shared", 0):
            sg, sd = moe.pack_shared_weights(cfg, sg, su, sd)
            su = None
    s_aux = torch.cuda.Stream()

    def layer(x, out, ws, s_main):
        moe.moe_layer(cfg, T, x, t["w_router"], t["bias"], wg, wu, wd, sg, su, sd, out, ws,
                      s_main=s_main, s_aux=s_aux)

    # eager references, on a workspace of their own (this also runs every
    # launcher's one-time set-up before the capture)
    ws_eager = moe.alloc_workspace(cfg, T)
    want = []
    for x in xs:
        o = torch.full((T, d), float("nan"), dtype=cfg.torch_dtype, device="cuda")
        layer(x, o, ws_eager, torch.cuda.current_stream())
        want.append(o)
    torch.cuda.synchronize()
    for i, o in enumerate(want):
        assert torch.isfinite(o.float()).all(), f"eager output {i} has unwritten rows"

    ws = moe.alloc_workspace(cfg, T)
    x_in = xs[0].clone()
    out = torch.full((T, d), float("nan"), dtype=cfg.torch_dtype, device="cuda")
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        layer(x_in, out, ws, torch.cuda.current_stream())
    torch.cuda.synchronize()

    scratch = torch.empty((T, d), dtype=cfg.torch_dtype, device="cuda")
    for r in range(2 * REPLAYS):
        i = r % REPLAYS
        x_in.copy_(xs[i])
        out.fill_(float("nan"))
        g.replay()
        # the program's own eager work between replays: a layer call on the
        # other workspace, on the same stream
        layer(xs[(i + 1) % REPLAYS], scratch, ws_eager, torch.cuda.current_stream())
        torch.cuda.synchronize()
        assert torch.equal(out, want[i]), f"replay {r} (input {i}) differs from the eager call"
        assert torch.equal(scratch, want[(i + 1) % REPLAYS]), f"eager call after replay {r} changed"
    G.log("  ", 2 * REPLAYS, "replays identical to the eager calls")
