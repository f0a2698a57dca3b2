"""MoE verification pass of EcoSpec (arXiv 2607.12696) on MI355X / gfx950.

Thin ctypes binding of ``libecospec_moe.so`` (declared in
``include/ecospec_moe.h``).  The functions carry the C names and only
marshal arguments: PyTorch supplies device memory and the current HIP
stream, and every step of the pass runs in the library's HIP kernels.  If
the library has not been built, importing the functions that need it raises
``ImportError``; there is no fallback.

    moe_route_topk(logits, k, score)            -> (topk_idx, topk_w)
    moe_route_topk_hidden(x, w_router, k, score) -> (topk_idx, topk_w)
    moe_route_topk_grouped(logits, bias, k, n_group, topk_group, scale) -> (topk_idx, topk_w)
    moe_expert_union(topk_idx, E)               -> Routing
    moe_verify_workspace_size(weights, T, k)    -> bytes
    moe_pack_weights(fmt, w, s)                 -> (w_packed, s_packed)   once per model load
    moe_pack_gate_up / moe_pack_down            -> the paired layouts pack_layer uses by default
    moe_verify_layer(x, weights, routing)       -> y   (weights packed)
    moe_select_tree(parent, P, pred, E, budget) -> (selected, marginal_cost)
    moe_route_union(logits, k, score)           -> Routing   (route + union in one call)
    moe_verify_step(x, logits, weights, k, score) = moe_route_union + moe_verify_layer
"""
from __future__ import annotations

import ctypes as C
import os
import threading
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libecospec_moe.so")

MOE_OK, MOE_ERR_INVALID_ARG, MOE_ERR_UNSUPPORTED, MOE_ERR_WORKSPACE, MOE_ERR_HIP = range(5)
MOE_SCORE_SOFTMAX, MOE_SCORE_SIGMOID = 0, 1
MOE_W_BF16, MOE_W_FP8_E4M3_B128, MOE_W_MXFP4 = 0, 1, 2
MOE_SEL_COST_RATIO, MOE_SEL_CONFIDENCE, MOE_SEL_GLOBAL_COST, MOE_SEL_COST_DIFF = 0, 1, 2, 3
MOE_ACT_SWIGLU, MOE_ACT_SWIGLU_OAI = 0, 1
MOE_ACTQ_BF16, MOE_ACTQ_MXFP8 = 0, 1

EXPORTED = ("moe_route_topk", "moe_route_union", "moe_route_topk_grouped", "moe_router_workspace_size", "moe_route_topk_hidden", "moe_expert_union", "moe_verify_workspace_size", "moe_verify_layer",
            "moe_verify_layer_timed", "moe_packed_size", "moe_pack_weights", "moe_pack_gate_up", "moe_pack_down",
            "moe_select_tree", "moe_status_string", "moe_last_error", "moe_verify_layer_noalloc")


class MoeError(RuntimeError):
    def __init__(self, fn: str, status: int, detail: str = ""):
        self.status = status
        super().__init__(f"{fn}: status {status} ({_status_string(status)}){': ' + detail if detail else ''}")


class moe_weights_t(C.Structure):
    _fields_ = [("fmt", C.c_int), ("d", C.c_int), ("d_ff", C.c_int), ("E", C.c_int)] + [
        (n, C.c_void_p) for n in ("w_gate", "w_up", "w_down", "s_gate", "s_up", "s_down", "sh_gate", "sh_up",
                                  "sh_down", "sh_s_gate", "sh_s_up", "sh_s_down")] + [
        ("act", C.c_int), ("alpha", C.c_float), ("limit", C.c_float),
        ("b_gate", C.c_void_p), ("b_up", C.c_void_p), ("b_down", C.c_void_p), ("act_fmt", C.c_int),
        ("down_paired", C.c_int)]


class moe_routing_t(C.Structure):
    _fields_ = [("T", C.c_int), ("k", C.c_int), ("E", C.c_int)] + [
        (n, C.c_void_p) for n in ("topk_idx", "topk_w", "counts", "union_ids", "n_unique", "offsets", "perm")]


_lock = threading.Lock()
_lib = None


def lib() -> C.CDLL:
    """The loaded library; raises ImportError if it has not been built."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2607_12696_amd.build`")
            L = C.CDLL(LIB_PATH)
            p, i = C.c_void_p, C.c_int
            L.moe_route_topk.argtypes = [p, i, i, i, i, p, p, p]
            L.moe_route_union.argtypes = [p, i, i, i, i, p, p, p, p, p, p, p, p]
            L.moe_route_topk_grouped.argtypes = [p, p, i, i, i, i, i, C.c_float, p, p, p]
            L.moe_router_workspace_size.argtypes = [i, i, i, C.POINTER(C.c_size_t)]
            L.moe_route_topk_hidden.argtypes = [p, p, i, i, i, i, i, p, p, p, p, C.c_size_t, p]
            L.moe_expert_union.argtypes = [p, i, i, i, p, p, p, p, p, p]
            L.moe_verify_workspace_size.argtypes = [C.POINTER(moe_weights_t), i, i, C.POINTER(C.c_size_t)]
            L.moe_verify_layer.argtypes = [p, C.POINTER(moe_weights_t), C.POINTER(moe_routing_t), p, p, C.c_size_t, p]
            L.moe_verify_layer_noalloc.argtypes = [p, C.POINTER(moe_weights_t), C.POINTER(moe_routing_t), p, p]
            L.moe_verify_layer_timed.argtypes = [p, C.POINTER(moe_weights_t), C.POINTER(moe_routing_t), p, p,
                                                 C.c_size_t, p, C.POINTER(C.c_void_p)]
            L.moe_packed_size.argtypes = [i, i, i, i, C.POINTER(C.c_size_t), C.POINTER(C.c_size_t)]
            L.moe_pack_weights.argtypes = [i, i, i, i, p, p, p, p, p]
            L.moe_pack_gate_up.argtypes = [i, i, i, i, p, p, p, p, p, p, p, p]
            L.moe_pack_down.argtypes = [i, i, i, i, p, p, p, p, p]
            L.moe_select_tree.argtypes = [i, p, p, i, i, p, i, p, i, C.c_double, C.c_double, i, p, p, p]
            L.moe_status_string.argtypes = [i]
            L.moe_status_string.restype = C.c_char_p
            L.moe_last_error.restype = C.c_char_p
            for f in ("moe_route_topk", "moe_route_union", "moe_route_topk_grouped", "moe_router_workspace_size", "moe_route_topk_hidden", "moe_expert_union", "moe_verify_workspace_size", "moe_verify_layer",
                      "moe_verify_layer_noalloc", "moe_verify_layer_timed", "moe_packed_size", "moe_pack_weights", "moe_pack_gate_up",
                      "moe_pack_down", "moe_select_tree"):
                getattr(L, f).restype = i
            _lib = L
    return _lib


def _status_string(s: int) -> str:
    try:
        return lib().moe_status_string(s).decode()
    except ImportError:
        return "library not loaded"


def _check(fn: str, status: int):
    if status != MOE_OK:
        detail = lib().moe_last_error().decode() if status == MOE_ERR_HIP else ""
        raise MoeError(fn, status, detail)


def _torch():
    import torch
    return torch


def _stream(t) -> int:
    torch = _torch()
    return torch.cuda.current_stream(t.device).cuda_stream


def _dev_ptr(t, what: str) -> int:
    if t is None:
        return 0
    if not t.is_cuda:
        raise ValueError(f"{what} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    return t.data_ptr()


# --------------------------------------------------------------------------- routing

def moe_route_topk(logits, k: int, score: int, topk_idx=None, topk_w=None):
    """Router top-k of fp32 logits [T, E] on the device -> (int32 [T, k], fp32 [T, k])."""
    torch = _torch()
    T, E = logits.shape
    if logits.dtype != torch.float32:
        raise ValueError("logits must be float32")
    if topk_idx is None:
        topk_idx = torch.empty(T, k, dtype=torch.int32, device=logits.device)
    if topk_w is None:
        topk_w = torch.empty(T, k, dtype=torch.float32, device=logits.device)
    _check("moe_route_topk", lib().moe_route_topk(_dev_ptr(logits, "logits"), T, E, k, score,
                                                    _dev_ptr(topk_idx, "topk_idx"), _dev_ptr(topk_w, "topk_w"),
                                                    _stream(logits)))
    return topk_idx, topk_w


def moe_route_topk_grouped(logits, bias, k: int, n_group: int, topk_group: int, scale: float, topk_idx=None,
                           topk_w=None):
    """Group-limited sigmoid routing (correction bias [E] or None, routed scaling `scale`) of fp32
    logits [T, E] on the device -> (int32 [T, k], fp32 [T, k])."""
    torch = _torch()
    T, E = logits.shape
    if logits.dtype != torch.float32 or (bias is not None and (bias.dtype != torch.float32 or bias.numel() != E)):
        raise ValueError("logits [T, E] and bias [E] must be float32")
    if topk_idx is None:
        topk_idx = torch.empty(T, k, dtype=torch.int32, device=logits.device)
    if topk_w is None:
        topk_w = torch.empty(T, k, dtype=torch.float32, device=logits.device)
    _check("moe_route_topk_grouped", lib().moe_route_topk_grouped(
        _dev_ptr(logits, "logits"), _dev_ptr(bias, "bias"), T, E, k, n_group, topk_group, scale,
        _dev_ptr(topk_idx, "topk_idx"), _dev_ptr(topk_w, "topk_w"), _stream(logits)))
    return topk_idx, topk_w


def moe_router_workspace_size(T: int, d: int, E: int) -> int:
    n = C.c_size_t(0)
    _check("moe_router_workspace_size", lib().moe_router_workspace_size(T, d, E, C.byref(n)))
    return n.value


def moe_route_topk_hidden(x, w_router, k: int, score: int, logits=None, workspace=None, topk_idx=None, topk_w=None):
    """Router logits x . W_r^T (bf16 x [T, d], bf16 W_r [E, d]) and their top-k on the device
    -> (int32 [T, k], fp32 [T, k]); the fp32 logits land in `logits` [T, E] when it is given."""
    torch = _torch()
    T, d = x.shape
    E, d2 = w_router.shape
    if d2 != d:
        raise ValueError("x and w_router disagree on d")
    if x.dtype != torch.bfloat16 or w_router.dtype != torch.bfloat16:
        raise ValueError("x and w_router must be bfloat16")
    if logits is not None and (logits.dtype != torch.float32 or tuple(logits.shape) != (T, E)):
        raise ValueError("logits must be float32 [T, E]")
    if topk_idx is None:
        topk_idx = torch.empty(T, k, dtype=torch.int32, device=x.device)
    if topk_w is None:
        topk_w = torch.empty(T, k, dtype=torch.float32, device=x.device)
    if workspace is None:
        workspace = torch.empty(moe_router_workspace_size(T, d, E), dtype=torch.uint8, device=x.device)
    _check("moe_route_topk_hidden", lib().moe_route_topk_hidden(
        _dev_ptr(x, "x"), _dev_ptr(w_router, "w_router"), T, d, E, k, score, _dev_ptr(topk_idx, "topk_idx"),
        _dev_ptr(topk_w, "topk_w"), _dev_ptr(logits, "logits"), _dev_ptr(workspace, "workspace"),
        workspace.numel() * workspace.element_size(), _stream(x)))
    return topk_idx, topk_w


@dataclass
class Routing:
    """Device routing of T tokens: the outputs of moe_route_topk and moe_expert_union.  moe_verify_layer
    reads topk_idx / topk_w and writes the union and grouping arrays itself."""
    T: int
    k: int
    E: int
    topk_idx: object
    topk_w: object
    counts: object
    union_ids: object
    n_unique: object
    offsets: object
    perm: object

    def c_struct(self) -> moe_routing_t:
        r = moe_routing_t()
        r.T, r.k, r.E = self.T, self.k, self.E
        for n in ("topk_idx", "topk_w", "counts", "union_ids", "n_unique", "offsets", "perm"):
            setattr(r, n, _dev_ptr(getattr(self, n), n))
        return r


def moe_expert_union(topk_idx, E: int, topk_w=None, out: Routing | None = None) -> Routing:
    """Expert union, counts, offsets and stable grouping of topk_idx [T, k] on the device."""
    torch = _torch()
    T, k = topk_idx.shape
    dev = topk_idx.device
    if out is None:
        i32 = dict(dtype=torch.int32, device=dev)
        out = Routing(T, k, E, topk_idx, topk_w, torch.empty(E, **i32), torch.empty(E, **i32),
                      torch.empty(1, **i32), torch.empty(E + 1, **i32), torch.empty(T * k, **i32))
    _check("moe_expert_union", lib().moe_expert_union(
        _dev_ptr(topk_idx, "topk_idx"), T, k, E, _dev_ptr(out.counts, "counts"), _dev_ptr(out.union_ids, "union_ids"),
        _dev_ptr(out.n_unique, "n_unique"), _dev_ptr(out.offsets, "offsets"), _dev_ptr(out.perm, "perm"),
        _stream(topk_idx)))
    return out


def routing_for(topk_idx, topk_w, E: int) -> Routing:
    """A Routing around a top-k (moe_route_topk's output) with empty union and grouping arrays, which
    moe_verify_layer fills."""
    torch = _torch()
    T, k = topk_idx.shape
    i32 = dict(dtype=torch.int32, device=topk_idx.device)
    return Routing(T, k, E, topk_idx, topk_w, torch.empty(E, **i32), torch.empty(E, **i32), torch.empty(1, **i32),
                   torch.empty(E + 1, **i32), torch.empty(T * k, **i32))


def moe_route_union(logits, k: int, score: int, out: Routing | None = None) -> Routing:
    """moe_route_topk + moe_expert_union of fp32 logits [T, E] in one call."""
    torch = _torch()
    T, E = logits.shape
    if logits.dtype != torch.float32:
        raise ValueError("logits must be float32")
    dev = logits.device
    if out is None:
        i32 = dict(dtype=torch.int32, device=dev)
        out = Routing(T, k, E, torch.empty(T, k, **i32), torch.empty(T, k, dtype=torch.float32, device=dev),
                      torch.empty(E, **i32), torch.empty(E, **i32), torch.empty(1, **i32), torch.empty(E + 1, **i32),
                      torch.empty(T * k, **i32))
    _check("moe_route_union", lib().moe_route_union(
        _dev_ptr(logits, "logits"), T, E, k, score, _dev_ptr(out.topk_idx, "topk_idx"), _dev_ptr(out.topk_w, "topk_w"),
        _dev_ptr(out.counts, "counts"), _dev_ptr(out.union_ids, "union_ids"), _dev_ptr(out.n_unique, "n_unique"),
        _dev_ptr(out.offsets, "offsets"), _dev_ptr(out.perm, "perm"), _stream(logits)))
    return out


# --------------------------------------------------------------------------- weight packing

def moe_packed_size(fmt: int, E: int, N: int, K: int) -> tuple[int, int]:
    wb, sb = C.c_size_t(), C.c_size_t()
    _check("moe_packed_size", lib().moe_packed_size(fmt, E, N, K, C.byref(wb), C.byref(sb)))
    return wb.value, sb.value


def moe_pack_weights(fmt: int, w, s=None):
    """Pack stacked device weights w [E, N, K(/2)] (+ scales) into the streaming layout.

    Returns (w_packed, s_packed) as flat uint8 device tensors (s_packed None for bf16).
    """
    torch = _torch()
    E, N = w.shape[0], w.shape[1]
    K = w.shape[2] * (2 if fmt == MOE_W_MXFP4 else 1)
    wb, sb = moe_packed_size(fmt, E, N, K)
    wp = torch.empty(wb, dtype=torch.uint8, device=w.device)
    sp = torch.empty(sb, dtype=torch.uint8, device=w.device) if sb else None
    _check("moe_pack_weights", lib().moe_pack_weights(fmt, E, N, K, _dev_ptr(w, "w"), _dev_ptr(s, "s"),
                                                        _dev_ptr(wp, "w_packed"), _dev_ptr(sp, "s_packed"),
                                                        _stream(w)))
    return wp, sp


def moe_pack_gate_up(fmt: int, w_gate, w_up, s_gate=None, s_up=None):
    """Pack stacked device W_gate and W_up [E, N, K(/2)] (+ scales) as one pair.

    Returns (w_packed, s_gate_packed, s_up_packed); the scales are None for bf16.
    """
    torch = _torch()
    E, N = w_gate.shape[0], w_gate.shape[1]
    K = w_gate.shape[2] * (2 if fmt == MOE_W_MXFP4 else 1)
    wb, sb = moe_packed_size(fmt, E, N, K)
    wp = torch.empty(2 * wb, dtype=torch.uint8, device=w_gate.device)
    sgp = torch.empty(sb, dtype=torch.uint8, device=w_gate.device) if sb else None
    sup = torch.empty(sb, dtype=torch.uint8, device=w_gate.device) if sb else None
    _check("moe_pack_gate_up", lib().moe_pack_gate_up(
        fmt, E, N, K, _dev_ptr(w_gate, "w_gate"), _dev_ptr(s_gate, "s_gate"), _dev_ptr(w_up, "w_up"),
        _dev_ptr(s_up, "s_up"), _dev_ptr(wp, "w_packed"), _dev_ptr(sgp, "s_gate_packed"), _dev_ptr(sup, "s_up_packed"),
        _stream(w_gate)))
    return wp, sgp, sup


def moe_pack_down(fmt: int, w, s=None):
    """Pack stacked device W_down [E, N, K(/2)] (+ scales) with each wavefront's two row tiles
    interleaved.  Returns (w_packed, s_packed) like moe_pack_weights."""
    torch = _torch()
    E, N = w.shape[0], w.shape[1]
    K = w.shape[2] * (2 if fmt == MOE_W_MXFP4 else 1)
    wb, sb = moe_packed_size(fmt, E, N, K)
    wp = torch.empty(wb, dtype=torch.uint8, device=w.device)
    sp = torch.empty(sb, dtype=torch.uint8, device=w.device) if sb else None
    _check("moe_pack_down", lib().moe_pack_down(fmt, E, N, K, _dev_ptr(w, "w"), _dev_ptr(s, "s"),
                                                  _dev_ptr(wp, "w_packed"), _dev_ptr(sp, "s_packed"), _stream(w)))
    return wp, sp


def pack_layer(layer: dict, pair: bool = True, down_pair: bool = True) -> dict:
    """A layer dict (interchange layout, device tensors) with every matrix packed; with `pair`,
    W_gate and W_up as one pair (moe_pack_gate_up; the dict then has no "up" / "sh_up" entry);
    with `down_pair`, W_down by moe_pack_down (the dict then has down_paired = 1)."""
    out = {k: layer[k] for k in ("fmt", "d", "d_ff", "act", "alpha", "limit", "b_gate", "b_up", "b_down", "act_fmt")
           if k in layer}
    if down_pair:
        out["down_paired"] = 1
    out["E"] = int(layer.get("E", layer["gate"].shape[0]))
    fmt = int(layer["fmt"])
    for prefix in ("", "sh_"):
        names = ("gate", "up", "down")
        if pair and layer.get(prefix + "gate") is not None and layer.get(prefix + "up") is not None:
            wp, sgp, sup = moe_pack_gate_up(fmt, layer[prefix + "gate"], layer[prefix + "up"],
                                            layer.get(prefix + "s_gate"), layer.get(prefix + "s_up"))
            out[prefix + "gate"] = wp
            if sgp is not None:
                out[prefix + "s_gate"], out[prefix + "s_up"] = sgp, sup
            names = ("down",)
        for name in names:
            if layer.get(prefix + name) is None:
                continue
            pack = moe_pack_down if name == "down" and down_pair else moe_pack_weights
            wp, sp = pack(fmt, layer[prefix + name], layer.get(prefix + "s_" + name))
            out[prefix + name] = wp
            if sp is not None:
                out[prefix + "s_" + name] = sp
    return out


# --------------------------------------------------------------------------- verify layer

def weights_struct(w: dict) -> moe_weights_t:
    """moe_weights_t for a layer dict (keys fmt, d, d_ff, E, gate, up, down, optional s_*, sh_*,
    fp32 biases b_gate / b_up [E, d_ff] and b_down [E, d], act / alpha / limit, and act_fmt)."""
    s = moe_weights_t()
    torch = _torch()
    s.act = int(w.get("act", MOE_ACT_SWIGLU))
    s.act_fmt = int(w.get("act_fmt", MOE_ACTQ_BF16))
    s.down_paired = int(w.get("down_paired", 0))
    s.alpha, s.limit = float(w.get("alpha", 1.702)), float(w.get("limit", 7.0))
    for name in ("b_gate", "b_up", "b_down"):
        b = w.get(name)
        if b is not None and b.dtype != torch.float32:
            raise ValueError(f"{name} must be float32")
        setattr(s, name, _dev_ptr(b, name))
    s.fmt, s.d, s.d_ff = int(w["fmt"]), int(w["d"]), int(w["d_ff"])
    s.E = int(w["E"]) if "E" in w else int(w["gate"].shape[0])
    for name in ("gate", "up", "down"):
        setattr(s, "w_" + name, _dev_ptr(w.get(name), name))
        setattr(s, "s_" + name, _dev_ptr(w.get("s_" + name), "s_" + name))
        setattr(s, "sh_" + name, _dev_ptr(w.get("sh_" + name), "sh_" + name))
        setattr(s, "sh_s_" + name, _dev_ptr(w.get("sh_s_" + name), "sh_s_" + name))
    return s


def moe_verify_workspace_size(weights: dict, T: int, k: int) -> int:
    n = C.c_size_t()
    ws = weights_struct(weights)
    _check("moe_verify_workspace_size", lib().moe_verify_workspace_size(C.byref(ws), T, k, C.byref(n)))
    return n.value


def moe_verify_layer(x, weights: dict, routing: Routing, y=None, workspace=None):
    """y [T, d] bf16 = the MoE layer over the routed tokens x [T, d] bf16."""
    torch = _torch()
    T, d = x.shape
    if x.dtype != torch.bfloat16:
        raise ValueError("x must be bfloat16")
    if y is None:
        y = torch.empty_like(x)
    if workspace is None:
        workspace = torch.empty(moe_verify_workspace_size(weights, T, routing.k), dtype=torch.uint8, device=x.device)
    ws = weights_struct(weights)
    rs = routing.c_struct()
    _check("moe_verify_layer", lib().moe_verify_layer(
        _dev_ptr(x, "x"), C.byref(ws), C.byref(rs), _dev_ptr(y, "y"), _dev_ptr(workspace, "workspace"),
        workspace.numel() * workspace.element_size(), _stream(x)))
    return y


def moe_verify_layer_noalloc(x, weights: dict, routing: Routing, y=None):
    """moe_verify_layer on the library's fixed per-GPU scratch (no workspace argument, nothing allocated
    by the library)."""
    torch = _torch()
    if x.dtype != torch.bfloat16:
        raise ValueError("x must be bfloat16")
    if y is None:
        y = torch.empty_like(x)
    ws = weights_struct(weights)
    rs = routing.c_struct()
    status = lib().moe_verify_layer_noalloc(_dev_ptr(x, "x"), C.byref(ws), C.byref(rs), _dev_ptr(y, "y"), _stream(x))
    if status == MOE_ERR_WORKSPACE:
        raise MoeError("moe_verify_layer_noalloc", status, lib().moe_last_error().decode())
    _check("moe_verify_layer_noalloc", status)
    return y


def moe_verify_layer_timed(x, weights: dict, routing: Routing, y, workspace, events):
    """moe_verify_layer that also records 5 torch.cuda.Event marks on the current stream:
    before the gate/up expert kernel, after it, before the down expert kernel, after it,
    after the combine kernel."""
    if len(events) != 5:
        raise ValueError("moe_verify_layer_timed takes 5 events")
    arr = (C.c_void_p * 5)(*[e.cuda_event if e is not None else None for e in events])
    ws = weights_struct(weights)
    rs = routing.c_struct()
    _check("moe_verify_layer_timed", lib().moe_verify_layer_timed(
        _dev_ptr(x, "x"), C.byref(ws), C.byref(rs), _dev_ptr(y, "y"), _dev_ptr(workspace, "workspace"),
        workspace.numel() * workspace.element_size(), _stream(x), arr))
    return y


def moe_verify_step(x, logits, weights: dict, k: int, score: int, workspace=None, y=None):
    """Route (top-k), then verify one layer, which builds the union and grouping itself: the whole hot
    path on the device.  Returns y and the routing, its union arrays filled by the verification."""
    idx, w = moe_route_topk(logits, k, score)
    r = routing_for(idx, w, logits.shape[1])
    return moe_verify_layer(x, weights, r, y=y, workspace=workspace), r


# --------------------------------------------------------------------------- selector (host)

def moe_select_tree(parent, P, pred, E: int, budget: int, eps: float = 0.1, lam: float = 0.0,
                    mode: int = MOE_SEL_COST_RATIO, B0=None):
    """Cost-aware draft selection (Algorithm 1) on the host -> (selected, marginal_cost) int32 arrays."""
    par = np.ascontiguousarray(parent, np.int32)
    Pa = np.ascontiguousarray(P, np.float64)
    pr = np.ascontiguousarray(pred, np.int32)
    n, L, K = pr.shape
    sel = np.zeros(max(budget, 1), np.int32)
    cost = np.zeros(max(budget, 1), np.int32)
    nsel = np.zeros(1, np.int32)
    b0 = None if B0 is None else np.ascontiguousarray(B0, np.uint64)
    _check("moe_select_tree", lib().moe_select_tree(
        n, par.ctypes.data, Pa.ctypes.data, L, K, pr.ctypes.data, E, None if b0 is None else b0.ctypes.data,
        budget, eps, lam, mode, sel.ctypes.data, cost.ctypes.data, nsel.ctypes.data))
    m = int(nsel[0])
    return sel[:m].copy(), cost[:m].copy()
