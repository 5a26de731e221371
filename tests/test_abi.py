"""Host-side checks of the C ABI: the library loads, exports every entry point
declared in include/moe.h, sizes workspaces and rejects bad arguments. No call
here reaches a GPU: every failing case returns during validation, before any
HIP call, and the T = 0 cases return before any launch."""
import ctypes
import os
import re

import pytest

from paper_2603_02376_amd import moe
from paper_2603_02376_amd.inputs import PRESETS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 1 << 20  # an aligned non-NULL address that is never dereferenced


def _header_functions():
    src = open(os.path.join(ROOT, "include", "moe.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(moe_[a-z0-9_]+)\s*\(", src)))


def test_library_exports_every_declared_function():
    L = moe.lib()
    declared = _header_functions()
    assert declared, "no functions parsed from moe.h"
    for name in declared:
        assert hasattr(L, name), f"{name} declared in moe.h but not exported"
    assert set(declared) == set(moe.EXPORTS)


def test_version_and_status_strings():
    assert "gfx950" in moe.version()
    L = moe.lib()
    assert L.moe_status_string(0) == b"ok"
    assert L.moe_status_string(-3) == b"workspace too small"


def _cfg(**kw):
    base = dict(d=128, E=8, k=2, I=256)
    base.update(kw)
    return moe.MoeConfig(**base)


@pytest.mark.parametrize("name", list(PRESETS))
def test_workspace_size_presets(name):
    p = PRESETS[name]
    cfg = moe.MoeConfig(d=p["d"], E=p["E"], k=p["k"], I=p["I"], n_groups=p["n_groups"],
                        topk_groups=p["topk_groups"], n_shared=p["n_shared"], I_shared=p["I_shared"],
                        score=p["score"], scale=p["scale"], dtype=p["dtype"])
    n = moe.workspace_size(cfg, p["T"])
    es = 2 if p["dtype"] == "bf16" else 4
    tk = p["T"] * p["k"]
    # at least h and y_perm, and the shared-expert scratch
    floor = tk * (p["I"] + p["d"]) * es + p["n_shared"] * p["T"] * (p["I_shared"] + p["d"]) * es
    assert floor <= n <= floor + (64 << 20)
    assert n % 256 == 0
    assert moe.workspace_size(cfg, 0) >= 0


@pytest.mark.parametrize("kw,status", [
    (dict(k=9), -1),                                    # k > E
    (dict(E=12, n_groups=5), -1),                       # E % n_groups
    (dict(n_groups=4, topk_groups=5), -1),              # topk_groups > n_groups
    (dict(E=8, k=3, n_groups=4, topk_groups=1), -1),    # k > experts left by the group limit
    (dict(E=512, k=2), -2),                             # E > 256
    (dict(E=32, k=17), -2),                             # k > 16
    (dict(d=96), -2),                                   # d % 64
    (dict(I=100), -2),                                  # I % 64
    (dict(n_shared=2, I_shared=64), -2),                # n_shared > 1
    (dict(n_shared=1, I_shared=0), -1),
    (dict(weight_layout="packed"), -2),                 # packed needs d % 256 == 0
    (dict(d=256, I=192, weight_layout="packed"), -2),   # and I % 128 == 0
    (dict(d=256, I=128, dtype="f32", weight_layout="packed"), -2),
    (dict(d=256, I=128, n_shared=1, I_shared=192, weight_layout="packed"), -2),  # I_shared % 128
])
def test_invalid_configs_rejected(kw, status):
    cfg = _cfg(**kw)
    assert moe.workspace_size(cfg, 16) == 0
    c = cfg.c()
    r = moe.lib().moe_route(ctypes.byref(c), 16, None, None, None, FAKE, FAKE, FAKE, None, 0, None)
    assert r == status
    assert moe.lib().moe_last_error().decode()


def test_packed_layout_rejects_operands_beyond_32bit_offsets():
    cfg = _cfg(d=256, I=128, weight_layout="packed")
    c = cfg.c()
    assert moe.workspace_size(cfg, 1 << 16) > 0
    big = 1 << 24                                       # T*d*2 bytes = 8 GiB
    assert moe.workspace_size(cfg, big) == 0
    r = moe.lib().moe_route(ctypes.byref(c), big, None, None, None, FAKE, FAKE, FAKE, None, 0, None)
    assert r == -2
    assert b"2^31" in moe.lib().moe_last_error()


def test_null_and_negative_arguments():
    c = _cfg().c()
    L = moe.lib()
    assert L.moe_route(None, 4, None, None, None, FAKE, FAKE, FAKE, None, 0, None) == -1
    assert L.moe_route(ctypes.byref(c), -1, None, None, None, FAKE, FAKE, FAKE, None, 0, None) == -1
    assert L.moe_route(ctypes.byref(c), 4, None, None, None, None, FAKE, FAKE, None, 0, None) == -1
    assert b"logits" in L.moe_last_error()
    # misaligned pointer
    assert L.moe_route(ctypes.byref(c), 4, None, None, None, FAKE + 4, FAKE, FAKE, None, 0, None) == -1
    assert b"aligned" in L.moe_last_error()
    # bias with softmax routing
    assert L.moe_route(ctypes.byref(c), 4, None, None, FAKE, FAKE, FAKE, FAKE, None, 0, None) == -1
    # router GEMM without a workspace
    assert L.moe_route(ctypes.byref(c), 4, FAKE, FAKE, None, FAKE, FAKE, FAKE, None, 0, None) == -1
    assert L.moe_route(ctypes.byref(c), 4, FAKE, FAKE, None, FAKE, FAKE, FAKE, FAKE, 16, None) == -3
    # combine / expert_ffn NULLs
    assert L.moe_combine(ctypes.byref(c), 4, None, FAKE, FAKE, None, FAKE, None) == -1
    assert L.moe_expert_ffn(ctypes.byref(c), 4, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE, 1 << 30, None) == -1
    # shared FFN without a shared expert
    assert L.moe_shared_ffn(ctypes.byref(c), 4, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 30, None) == -1


def test_workspace_too_small_and_misaligned():
    cfg = _cfg()
    c = cfg.c()
    L = moe.lib()
    need = moe.workspace_size(cfg, 64)
    args = (ctypes.byref(c), 64, FAKE, FAKE, FAKE, FAKE, None, FAKE)
    assert L.moe_dispatch(*args, FAKE, need - 1, None) == -3
    assert b"workspace too small" in L.moe_last_error()
    assert L.moe_dispatch(*args, FAKE + 16, need, None) == -1
    assert L.moe_dispatch(*args, None, need, None) == -1


def test_pack_weights_validation():
    L = moe.lib()
    c = _cfg(d=256, I=128).c()
    assert L.moe_pack_weights(None, FAKE, FAKE, FAKE, FAKE, FAKE, None) == -1
    assert L.moe_pack_weights(ctypes.byref(c), FAKE, None, FAKE, FAKE, FAKE, None) == -1   # w_up missing
    assert L.moe_pack_weights(ctypes.byref(c), FAKE, FAKE, FAKE, None, None, None) == 0    # nothing to pack
    bad = _cfg(d=128, I=128).c()
    assert L.moe_pack_weights(ctypes.byref(bad), FAKE, FAKE, FAKE, FAKE, FAKE, None) == -2


def test_zero_tokens_is_a_noop():
    cfg = _cfg(n_shared=1, I_shared=64)
    c = cfg.c()
    L = moe.lib()
    need = moe.workspace_size(cfg, 0)
    assert L.moe_route(ctypes.byref(c), 0, None, None, None, FAKE, FAKE, FAKE, None, 0, None) == 0
    assert L.moe_dispatch(ctypes.byref(c), 0, FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE, need, None) == 0
    assert L.moe_combine(ctypes.byref(c), 0, FAKE, FAKE, FAKE, None, FAKE, None) == 0
    assert L.moe_layer(ctypes.byref(c), 0, FAKE, FAKE, None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                       FAKE, need, None, None, None) == 0


def test_last_error_is_per_thread():
    """moe_last_error() holds the message of the calling thread's last failure:
    a failure on another thread leaves this thread's message alone."""
    import threading

    L = moe.lib()
    c = _cfg().c()
    assert L.moe_route(ctypes.byref(c), -1, None, None, None, FAKE, FAKE, FAKE, None, 0, None) == -1
    mine = L.moe_last_error()
    assert b"T < 0" in mine
    seen = {}

    def other():
        seen["before"] = L.moe_last_error()
        seen["status"] = L.moe_route(ctypes.byref(c), 4, None, None, None, None, FAKE, FAKE, None, 0, None)
        seen["after"] = L.moe_last_error()

    th = threading.Thread(target=other)
    th.start()
    th.join()
    assert seen["before"] == b"" and seen["status"] == -1 and b"logits" in seen["after"]
    assert L.moe_last_error() == mine


def test_pack_weights_with_nothing_to_pack_makes_no_hip_call():
    # no output buffer: validated and returns before any HIP call (runs without a GPU)
    c = _cfg(d=256, I=128).c()
    assert moe.lib().moe_pack_weights(ctypes.byref(c), None, None, None, None, None, None) == 0
