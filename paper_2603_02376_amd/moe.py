"""Python binding of libmoe.so: argument marshalling only.

Every function here has the name of the C entry point it calls and does no
arithmetic of the method: it checks tensor devices, dtypes and shapes, turns
tensors into device pointers and torch streams into ``hipStream_t`` handles,
and raises :class:`MoeError` on a non-zero status. PyTorch only provides
device memory and streams. If the library is not built, loading fails loudly;
there is no fallback.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from dataclasses import dataclass

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libmoe.so")

MOE_F32, MOE_BF16 = 0, 1
MOE_SCORE_SOFTMAX, MOE_SCORE_SIGMOID = 0, 1
MOE_LAYOUT_ROWMAJOR, MOE_LAYOUT_PACKED = 0, 1
MOE_QUANT_NONE, MOE_QUANT_INT8, MOE_QUANT_FP8 = 0, 1, 2
_QUANT = {"none": MOE_QUANT_NONE, "int8": MOE_QUANT_INT8, "fp8": MOE_QUANT_FP8}
MOE_EP_SELF, MOE_EP_REMOTE = 0, 1
EP_SCHEDULES = {"sequential": 0, "self_remote": 1, "expert_chunks": 2}
STATUS = {0: "MOE_OK", -1: "MOE_ERR_INVALID_ARG", -2: "MOE_ERR_UNSUPPORTED",
          -3: "MOE_ERR_WORKSPACE", -4: "MOE_ERR_HIP"}


class MoeError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status


class moe_config_t(ctypes.Structure):
    _fields_ = [("d", ctypes.c_int32), ("E", ctypes.c_int32), ("k", ctypes.c_int32),
                ("n_groups", ctypes.c_int32), ("topk_groups", ctypes.c_int32), ("I", ctypes.c_int32),
                ("n_shared", ctypes.c_int32), ("I_shared", ctypes.c_int32), ("score", ctypes.c_int32),
                ("renorm", ctypes.c_int32), ("route_scale", ctypes.c_float), ("dtype", ctypes.c_int32),
                ("weight_layout", ctypes.c_int32), ("token_quant", ctypes.c_int32)]


class moe_ep_options_t(ctypes.Structure):
    _fields_ = [("schedule", ctypes.c_int32), ("chunks", ctypes.c_int32), ("link_workgroups", ctypes.c_int32),
                ("gemm_workgroups", ctypes.c_int32)]


class moe_layer_debug_t(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("logits", "topk_idx", "topk_w", "counts", "offsets",
                                               "sorted_token", "sorted_assign", "inv_perm", "y_perm",
                                               "shared_out")]


_VP, _I32, _SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
_CFG = ctypes.POINTER(moe_config_t)
_SIGS = {
    "moe_workspace_size": (_SZ, [_CFG, _I32]),
    "moe_route": (ctypes.c_int, [_CFG, _I32, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _SZ, _VP]),
    "moe_dispatch": (ctypes.c_int, [_CFG, _I32, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _SZ, _VP]),
    "moe_dispatch_noalloc": (ctypes.c_int, [_CFG, _I32, _VP, _VP, _VP, _VP, _VP, _VP, _VP]),
    "moe_expert_ffn": (ctypes.c_int, [_CFG, _I32, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _SZ, _VP]),
    "moe_shared_ffn": (ctypes.c_int, [_CFG, _I32, _VP, _VP, _VP, _VP, _VP, _VP, _SZ, _VP]),
    "moe_quantize": (ctypes.c_int, [_CFG, _I32, _VP, _VP, _VP, _VP]),
    "moe_expert_ffn_q8": (ctypes.c_int, [_CFG, _I32, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _SZ, _VP]),
    "moe_combine": (ctypes.c_int, [_CFG, _I32, _VP, _VP, _VP, _VP, _VP, _VP]),
    "moe_layer": (ctypes.c_int, [_CFG, _I32, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _SZ,
                                 _VP, _VP, ctypes.POINTER(moe_layer_debug_t)]),
    "moe_pack_weights": (ctypes.c_int, [_CFG, _VP, _VP, _VP, _VP, _VP, _VP]),
    "moe_ep_plan": (ctypes.c_int, [_CFG, _I32, _VP, _VP, _I32, _VP, _VP, _I32, _VP, _I32, _VP, _VP, _VP]),
    "moe_ep_copy_rows": (ctypes.c_int, [_CFG, _I32, _I32, _VP, _I32, _VP, _VP, _VP, _I32, _I32, _VP, _I32, _VP]),
    "moe_expert_ffn_segments": (ctypes.c_int, [_CFG, _I32, _VP, _VP, _VP, _I32, _I32, _VP, _VP, _VP, _I32, _VP,
                                               _SZ, _VP]),
    "moe_ep_expert_ffn": (ctypes.c_int, [_CFG, ctypes.POINTER(moe_ep_options_t), _I32, _VP, _I32, _VP, _I32, _VP,
                                         _VP, _VP, _VP, _VP, _VP, _VP, _VP, _SZ, _VP, _VP]),
    "moe_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "moe_last_error": (ctypes.c_char_p, []),
    "moe_version": (ctypes.c_char_p, []),
}
EXPORTS = tuple(_SIGS)

_lib = None


def lib() -> ctypes.CDLL:
    """Load libmoe.so (once). Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                               "(there is no fallback implementation)")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype, f.argtypes = res, args
        _lib = L
    return _lib


def _check(status: int) -> None:
    if status != 0:
        raise MoeError(status, lib().moe_last_error().decode())


# ---------------------------------------------------------------------------
# configuration
# ---------------------------------------------------------------------------

@dataclass(frozen=True)
class MoeConfig:
    d: int
    E: int
    k: int
    I: int
    n_groups: int = 1
    topk_groups: int = 1
    n_shared: int = 0
    I_shared: int = 0
    score: str = "softmax"     # "softmax" | "sigmoid"
    renorm: bool = True
    scale: float = 1.0
    dtype: str = "bf16"        # "bf16" | "f32"
    weight_layout: str = "rowmajor"  # "rowmajor" | "packed" (expert weights, see moe_pack_weights)
    token_quant: str = "none"        # "none" | "int8" | "fp8" (tokens the routed experts receive)

    @property
    def torch_dtype(self):
        return torch.bfloat16 if self.dtype == "bf16" else torch.float32

    def c(self) -> moe_config_t:
        return moe_config_t(self.d, self.E, self.k, self.n_groups, self.topk_groups, self.I, self.n_shared,
                            self.I_shared, MOE_SCORE_SIGMOID if self.score == "sigmoid" else MOE_SCORE_SOFTMAX,
                            int(bool(self.renorm)), float(self.scale),
                            MOE_BF16 if self.dtype == "bf16" else MOE_F32,
                            MOE_LAYOUT_PACKED if self.weight_layout == "packed" else MOE_LAYOUT_ROWMAJOR,
                            _QUANT[self.token_quant])

    @property
    def packed(self) -> bool:
        return self.weight_layout == "packed"


def workspace_size(cfg: MoeConfig, T: int) -> int:
    c = cfg.c()
    return int(lib().moe_workspace_size(ctypes.byref(c), T))


def alloc_workspace(cfg: MoeConfig, T: int, device="cuda") -> torch.Tensor:
    n = workspace_size(cfg, T)
    if n == 0:
        raise MoeError(-1, lib().moe_last_error().decode() or "invalid config")
    return torch.empty(n, dtype=torch.uint8, device=device)


# ---------------------------------------------------------------------------
# marshalling helpers
# ---------------------------------------------------------------------------

def _ptr(t, name, dtype=None, numel=None):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a device tensor, got {t.device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{name} holds {t.numel()} elements, needs {numel}")
    return t.data_ptr()


def _stream(s):
    if s is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(s, torch.cuda.Stream):
        return s.cuda_stream
    return int(s)


# ---------------------------------------------------------------------------
# entry points (same names as the C ABI)
# ---------------------------------------------------------------------------

def moe_route(cfg: MoeConfig, T, x, w_router, bias, logits, topk_idx, topk_w, ws=None, stream=None):
    """x = None routes from the given logits; otherwise the router GEMM runs
    first and ``ws`` (see :func:`alloc_workspace`) is required."""
    c = cfg.c()
    dt = cfg.torch_dtype
    _check(lib().moe_route(ctypes.byref(c), T, _ptr(x, "x", dt, T * cfg.d),
                           _ptr(w_router, "w_router", dt, cfg.E * cfg.d) if x is not None else None,
                           _ptr(bias, "bias", torch.float32, cfg.E),
                           _ptr(logits, "logits", torch.float32, T * cfg.E),
                           _ptr(topk_idx, "topk_idx", torch.int32, T * cfg.k),
                           _ptr(topk_w, "topk_w", torch.float32, T * cfg.k), _ptr(ws, "ws"),
                           0 if ws is None else ws.numel() * ws.element_size(), _stream(stream)))


def moe_dispatch(cfg: MoeConfig, T, topk_idx, counts, offsets, sorted_token, sorted_assign, inv_perm, ws,
                 stream=None):
    c = cfg.c()
    n = T * cfg.k
    _check(lib().moe_dispatch(ctypes.byref(c), T, _ptr(topk_idx, "topk_idx", torch.int32, n),
                              _ptr(counts, "counts", torch.int32, cfg.E),
                              _ptr(offsets, "offsets", torch.int32, cfg.E + 1),
                              _ptr(sorted_token, "sorted_token", torch.int32, n),
                              _ptr(sorted_assign, "sorted_assign", torch.int32, n),
                              _ptr(inv_perm, "inv_perm", torch.int32, n),
                              _ptr(ws, "ws"), ws.numel() * ws.element_size(), _stream(stream)))


def moe_dispatch_noalloc(cfg: MoeConfig, T, topk_idx, counts, offsets, sorted_token, sorted_assign, inv_perm,
                         stream=None):
    """moe_dispatch with the library's own scratch (no workspace argument)."""
    c = cfg.c()
    n = T * cfg.k
    _check(lib().moe_dispatch_noalloc(ctypes.byref(c), T, _ptr(topk_idx, "topk_idx", torch.int32, n),
                                      _ptr(counts, "counts", torch.int32, cfg.E),
                                      _ptr(offsets, "offsets", torch.int32, cfg.E + 1),
                                      _ptr(sorted_token, "sorted_token", torch.int32, n),
                                      _ptr(sorted_assign, "sorted_assign", torch.int32, n),
                                      _ptr(inv_perm, "inv_perm", torch.int32, n), _stream(stream)))


def moe_expert_ffn(cfg: MoeConfig, T, x, sorted_token, offsets, w_gate, w_up, w_down, y_perm, ws, stream=None):
    c = cfg.c()
    dt = cfg.torch_dtype
    n = T * cfg.k
    wsz = cfg.E * cfg.I * cfg.d
    gsz = 2 * wsz if cfg.packed else wsz
    _check(lib().moe_expert_ffn(ctypes.byref(c), T, _ptr(x, "x", dt, T * cfg.d),
                                _ptr(sorted_token, "sorted_token", torch.int32, n),
                                _ptr(offsets, "offsets", torch.int32, cfg.E + 1),
                                _ptr(w_gate, "w_gate", dt, gsz), _ptr(w_up, "w_up", dt, wsz),
                                _ptr(w_down, "w_down", dt, wsz), _ptr(y_perm, "y_perm", dt, n * cfg.d),
                                _ptr(ws, "ws"), ws.numel() * ws.element_size(), _stream(stream)))


def _codes(codes, n):
    """Codes buffer: 1-byte elements (int8, uint8 or float8_e4m3fn storage)."""
    if codes is not None and codes.element_size() != 1:
        raise TypeError(f"codes must have 1-byte elements, got {codes.dtype}")
    return _ptr(codes, "codes", None, n)


def moe_quantize(cfg: MoeConfig, T, x, codes, scales, stream=None):
    """Per-token quantization (cfg.token_quant "fp8": E4M3 codes, else int8):
    codes [T, d] (1-byte elements), scales fp32 [T]."""
    c = cfg.c()
    _check(lib().moe_quantize(ctypes.byref(c), T, _ptr(x, "x", cfg.torch_dtype, T * cfg.d), _codes(codes, T * cfg.d),
                              _ptr(scales, "scales", torch.float32, T), _stream(stream)))


def moe_expert_ffn_q8(cfg: MoeConfig, T, codes, scales, sorted_token, offsets, w_gate_up, w_down, y_perm, ws,
                      stream=None):
    """Expert FFN on quantized tokens (codes from :func:`moe_quantize` with the
    same cfg; packed weights from :func:`pack_weights`)."""
    c = cfg.c()
    n = T * cfg.k
    wsz = cfg.E * cfg.I * cfg.d
    _check(lib().moe_expert_ffn_q8(ctypes.byref(c), T, _codes(codes, T * cfg.d),
                                   _ptr(scales, "scales", torch.float32, T),
                                   _ptr(sorted_token, "sorted_token", torch.int32, n),
                                   _ptr(offsets, "offsets", torch.int32, cfg.E + 1),
                                   _ptr(w_gate_up, "w_gate_up", torch.bfloat16, 2 * wsz),
                                   _ptr(w_down, "w_down", torch.bfloat16, wsz),
                                   _ptr(y_perm, "y_perm", torch.bfloat16, n * cfg.d),
                                   _ptr(ws, "ws"), ws.numel() * ws.element_size(), _stream(stream)))


def moe_shared_ffn(cfg: MoeConfig, T, x, ws_gate, ws_up, ws_down, out, ws, stream=None):
    c = cfg.c()
    dt = cfg.torch_dtype
    wsz = cfg.I_shared * cfg.d
    gsz = 2 * wsz if cfg.packed else wsz   # packed: gate and up in one buffer, ws_up None
    _check(lib().moe_shared_ffn(ctypes.byref(c), T, _ptr(x, "x", dt, T * cfg.d),
                                _ptr(ws_gate, "ws_gate", dt, gsz), _ptr(ws_up, "ws_up", dt, wsz),
                                _ptr(ws_down, "ws_down", dt, wsz), _ptr(out, "out", dt, T * cfg.d),
                                _ptr(ws, "ws"), ws.numel() * ws.element_size(), _stream(stream)))


def moe_combine(cfg: MoeConfig, T, y_perm, inv_perm, topk_w, shared_out, out, stream=None):
    c = cfg.c()
    dt = cfg.torch_dtype
    n = T * cfg.k
    _check(lib().moe_combine(ctypes.byref(c), T, _ptr(y_perm, "y_perm", dt, n * cfg.d),
                             _ptr(inv_perm, "inv_perm", torch.int32, n),
                             _ptr(topk_w, "topk_w", torch.float32, n),
                             _ptr(shared_out, "shared_out", dt, T * cfg.d),
                             _ptr(out, "out", dt, T * cfg.d), _stream(stream)))


def moe_layer(cfg: MoeConfig, T, x, w_router, bias, w_gate, w_up, w_down, ws_gate, ws_up, ws_down, out, ws,
              s_main=None, s_aux=None, dbg: dict | None = None):
    """The whole layer; ``dbg`` maps intermediate names to device tensors that
    receive them (keys as in ``moe_layer_debug_t``)."""
    c = cfg.c()
    dt = cfg.torch_dtype
    wsz = cfg.E * cfg.I * cfg.d
    gsz = 2 * wsz if cfg.packed else wsz
    swsz = cfg.I_shared * cfg.d
    sgsz = 2 * swsz if cfg.packed else swsz
    dbg_s = None
    if dbg:
        unknown = set(dbg) - {f for f, _ in moe_layer_debug_t._fields_}
        if unknown:
            raise KeyError(f"unknown debug buffers {sorted(unknown)}")
        dbg_s = moe_layer_debug_t(**{k: _ptr(v, k) for k, v in dbg.items()})
    _check(lib().moe_layer(ctypes.byref(c), T, _ptr(x, "x", dt, T * cfg.d),
                           _ptr(w_router, "w_router", dt, cfg.E * cfg.d), _ptr(bias, "bias", torch.float32, cfg.E),
                           _ptr(w_gate, "w_gate", dt, gsz), _ptr(w_up, "w_up", dt, wsz),
                           _ptr(w_down, "w_down", dt, wsz), _ptr(ws_gate, "ws_gate", dt, sgsz),
                           _ptr(ws_up, "ws_up", dt, swsz), _ptr(ws_down, "ws_down", dt, swsz),
                           _ptr(out, "out", dt, T * cfg.d), _ptr(ws, "ws"), ws.numel() * ws.element_size(),
                           _stream(s_main), _stream(s_aux) if s_aux is not None else None,
                           ctypes.byref(dbg_s) if dbg_s is not None else None))


def moe_pack_weights(cfg: MoeConfig, w_gate, w_up, w_down, gate_up_packed, down_packed, stream=None):
    """Pack row-major expert weights for MOE_LAYOUT_PACKED (either output may be None)."""
    c = cfg.c()
    wsz = cfg.E * cfg.I * cfg.d
    _check(lib().moe_pack_weights(ctypes.byref(c), _ptr(w_gate, "w_gate", torch.bfloat16, wsz),
                                  _ptr(w_up, "w_up", torch.bfloat16, wsz),
                                  _ptr(w_down, "w_down", torch.bfloat16, wsz),
                                  _ptr(gate_up_packed, "gate_up_packed", torch.bfloat16, 2 * wsz),
                                  _ptr(down_packed, "down_packed", torch.bfloat16, wsz), _stream(stream)))


def pack_weights(cfg: MoeConfig, w_gate, w_up, w_down):
    """Allocate and fill the packed buffers; returns (gate_up_packed, down_packed)."""
    gu = torch.empty(2 * w_gate.numel(), dtype=torch.bfloat16, device=w_gate.device)
    dn = torch.empty(w_down.numel(), dtype=torch.bfloat16, device=w_down.device)
    moe_pack_weights(cfg, w_gate, w_up, w_down, gu, dn)
    return gu, dn


def pack_shared_weights(cfg: MoeConfig, ws_gate, ws_up, ws_down):
    """Packed buffers of the shared expert ([I_shared][d] and [d][I_shared]
    weights, packed as a single expert); returns (gate_up_packed, down_packed)."""
    one = dataclasses.replace(cfg, E=1, k=1, n_groups=1, topk_groups=1, I=cfg.I_shared, n_shared=0, I_shared=0)
    return pack_weights(one, ws_gate.unsqueeze(0), ws_up.unsqueeze(0), ws_down.unsqueeze(0))


# ---- receive side of expert parallelism (one GPU's share) -------------------

def ep_workspace(cfg: MoeConfig, n_rows: int, device="cuda") -> torch.Tensor:
    """Workspace of the expert-parallel calls for n_rows received rows."""
    return alloc_workspace(cfg, -(-n_rows // cfg.k), device)


def moe_ep_plan(cfg: MoeConfig, e_first, self_offsets, self_sorted_token, self_assignments, peer_offsets,
                peer_sorted_token, peer_assignments, row_token, capacity, offsets, self_end, stream=None):
    """Receive-buffer layout of the local experts (cfg.E of them, from global expert e_first)."""
    c = cfg.c()
    _check(lib().moe_ep_plan(ctypes.byref(c), e_first,
                             _ptr(self_offsets, "self_offsets", torch.int32, e_first + cfg.E + 1),
                             _ptr(self_sorted_token, "self_sorted_token", torch.int32, self_assignments),
                             self_assignments,
                             _ptr(peer_offsets, "peer_offsets", torch.int32, e_first + cfg.E + 1),
                             _ptr(peer_sorted_token, "peer_sorted_token", torch.int32, peer_assignments),
                             peer_assignments, _ptr(row_token, "row_token", torch.int32, capacity), capacity,
                             _ptr(offsets, "offsets", torch.int32, cfg.E + 1),
                             _ptr(self_end, "self_end", torch.int32, cfg.E), _stream(stream)))


def moe_ep_copy_rows(cfg: MoeConfig, source, n_rows, x_src, src_tokens, row_token, offsets, self_end, e_begin, e_end,
                     recv, max_workgroups=0, stream=None):
    """Fill the self (source 0) or remote (1) rows of experts [e_begin, e_end)."""
    c = cfg.c()
    dt = cfg.torch_dtype
    _check(lib().moe_ep_copy_rows(ctypes.byref(c), int(source), n_rows, _ptr(x_src, "x_src", dt, src_tokens * cfg.d),
                                  src_tokens, _ptr(row_token, "row_token", torch.int32, n_rows),
                                  _ptr(offsets, "offsets", torch.int32, cfg.E + 1),
                                  _ptr(self_end, "self_end", torch.int32, cfg.E), e_begin, e_end,
                                  _ptr(recv, "recv", dt, n_rows * cfg.d), int(max_workgroups), _stream(stream)))


def moe_expert_ffn_segments(cfg: MoeConfig, n_rows, x, seg_begin, seg_end, e_begin, e_end, w_gate_up, w_down, y, ws,
                            max_workgroups=0, stream=None):
    """FFN of experts [e_begin, e_end) over rows [seg_begin[e], seg_end[e]) of x
    (seg_end None: [seg_begin[e], seg_begin[e+1]))."""
    c = cfg.c()
    wsz = cfg.E * cfg.I * cfg.d
    _check(lib().moe_expert_ffn_segments(ctypes.byref(c), n_rows, _ptr(x, "x", torch.bfloat16, n_rows * cfg.d),
                                         _ptr(seg_begin, "seg_begin", torch.int32, cfg.E + (seg_end is None)),
                                         _ptr(seg_end, "seg_end", torch.int32, cfg.E), e_begin, e_end,
                                         _ptr(w_gate_up, "w_gate_up", torch.bfloat16, 2 * wsz),
                                         _ptr(w_down, "w_down", torch.bfloat16, wsz),
                                         _ptr(y, "y", torch.bfloat16, n_rows * cfg.d), int(max_workgroups),
                                         _ptr(ws, "ws"), ws.numel() * ws.element_size(), _stream(stream)))


def moe_ep_expert_ffn(cfg: MoeConfig, schedule: str, n_rows, x_self, self_tokens, x_peer, peer_tokens, row_token,
                      offsets, self_end, w_gate_up, w_down, recv, y, ws, chunks=1, link_workgroups=0,
                      gemm_workgroups=0, s_compute=None, s_link=None):
    """The receive side in one call (schedule: "sequential", "self_remote" or "expert_chunks")."""
    c = cfg.c()
    o = moe_ep_options_t(EP_SCHEDULES[schedule], int(chunks), int(link_workgroups), int(gemm_workgroups))
    wsz = cfg.E * cfg.I * cfg.d
    _check(lib().moe_ep_expert_ffn(ctypes.byref(c), ctypes.byref(o), n_rows,
                                   _ptr(x_self, "x_self", torch.bfloat16, self_tokens * cfg.d), self_tokens,
                                   _ptr(x_peer, "x_peer", torch.bfloat16, peer_tokens * cfg.d), peer_tokens,
                                   _ptr(row_token, "row_token", torch.int32, n_rows),
                                   _ptr(offsets, "offsets", torch.int32, cfg.E + 1),
                                   _ptr(self_end, "self_end", torch.int32, cfg.E),
                                   _ptr(w_gate_up, "w_gate_up", torch.bfloat16, 2 * wsz),
                                   _ptr(w_down, "w_down", torch.bfloat16, wsz),
                                   _ptr(recv, "recv", torch.bfloat16, n_rows * cfg.d),
                                   _ptr(y, "y", torch.bfloat16, n_rows * cfg.d),
                                   _ptr(ws, "ws"), ws.numel() * ws.element_size(), _stream(s_compute),
                                   _stream(s_link) if s_link is not None else None))


def version() -> str:
    return lib().moe_version().decode()
