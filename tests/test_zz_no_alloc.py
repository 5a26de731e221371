"""moe_dispatch_noalloc (the dispatch with the library's own scratch, for
callers that cannot allocate) against moe_dispatch with a caller workspace,
through the C ABI: two calls in a row, the second with fewer tokens, and the
limit checks."""
import numpy as np
import pytest
import torch

from paper_2603_02376_amd import moe
from tests.gpu_util import log

pytestmark = pytest.mark.gpu


def _topk(T, E, k, seed):
    rng = np.random.default_rng(seed)
    return np.argsort(rng.random((T, E)), axis=1)[:, :k].astype(np.int32)


def _outs(T, E, k):
    n = T * k
    return [torch.full((m,), -7, dtype=torch.int32, device="cuda") for m in (E, E + 1, n, n, n)]


@pytest.mark.parametrize("calls", [((4096, 256, 8), (1000, 256, 8)),     # DeepSeek-V3 shape, then fewer tokens
                                   ((65536, 256, 8), (129, 64, 6))])      # the largest size, then another config
def test_noalloc_dispatch_matches_workspace_dispatch(calls):
    for i, (T, E, k) in enumerate(calls):
        log("dispatch_noalloc call", i, "T", T, "E", E, "k", k)
        cfg = moe.MoeConfig(d=64, E=E, k=k, I=64, dtype="bf16")
        idx = torch.from_numpy(_topk(T, E, k, seed=T + i)).cuda()
        ref, got = _outs(T, E, k), _outs(T, E, k)
        moe.moe_dispatch(cfg, T, idx, *ref, moe.alloc_workspace(cfg, T))
        moe.moe_dispatch_noalloc(cfg, T, idx, *got)
        torch.cuda.synchronize()
        for name, a, b in zip(("counts", "offsets", "sorted_token", "sorted_assign", "inv_perm"), ref, got):
            assert torch.equal(a, b), f"call {i}: {name} differs"


def test_noalloc_dispatch_limits():
    # beyond the scratch: rejected before anything is enqueued (outputs untouched)
    cfg = moe.MoeConfig(d=64, E=256, k=8, I=64, dtype="bf16")
    T = 65537
    idx = torch.zeros((T, 8), dtype=torch.int32, device="cuda")
    outs = _outs(T, 256, 8)
    with pytest.raises(moe.MoeError) as e:
        moe.moe_dispatch_noalloc(cfg, T, idx, *outs)
    assert e.value.status == -2 and "scratch limit" in str(e.value)
    torch.cuda.synchronize()
    assert all((o == -7).all() for o in outs)
    # T = 0: a no-op
    moe.moe_dispatch_noalloc(cfg, 0, idx, *outs)
    torch.cuda.synchronize()
    assert all((o == -7).all() for o in outs)
