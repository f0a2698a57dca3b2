"""CPU oracle for the MoE verification pass -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the product
library: the arithmetic lives in ``oracle.c`` (plain fp64 C, built here with
gcc) and in ``select.py`` (Algorithm 1 in plain Python); this file only
marshals numpy arrays into it.

Public functions
----------------
route(logits, k, score)          -> idx int32 [T,k], w float64 [T,k]
router_logits(x, w_router)       -> float64 [T,E] = x . W_r^T of bf16 inputs
route_grouped(logits, bias, k, n_group, topk_group, scale) -> idx, w (group-limited sigmoid routing)
union(idx, E)                    -> dict(counts, union_ids, n_unique, offsets, perm)
verify_tokens(layer, x, idx, w, tokens, threads) -> y float64 [len(tokens), d]
decode_table(kind)               -> float64 array of every code's value
weight_at(fmt, w, s, n, c)       -> one decoded weight element
expert_bytes(fmt, d, d_ff)       -> (weight bytes, scale bytes)
mx_quantize(v)                   -> (quantised values, block exponents) of the MX activation mode
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None


def build(force: bool = True) -> str:
    """Compile oracle.c into liboracle.so with gcc (-O2, OpenMP, fp64 math)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.run(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99", "-Wall",
                        "-o", tmp, _SRC, "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


class _Layer(C.Structure):
    _fields_ = [("fmt", C.c_int), ("d", C.c_int), ("d_ff", C.c_int), ("n_experts", C.c_int),
                ("gate", C.POINTER(C.c_void_p)), ("up", C.POINTER(C.c_void_p)),
                ("down", C.POINTER(C.c_void_p)), ("s_gate", C.POINTER(C.c_void_p)),
                ("s_up", C.POINTER(C.c_void_p)), ("s_down", C.POINTER(C.c_void_p)),
                ("sh_gate", C.c_void_p), ("sh_up", C.c_void_p), ("sh_down", C.c_void_p),
                ("sh_s_gate", C.c_void_p), ("sh_s_up", C.c_void_p), ("sh_s_down", C.c_void_p),
                ("act", C.c_int), ("alpha", C.c_double), ("limit", C.c_double),
                ("b_gate", C.POINTER(C.c_void_p)), ("b_up", C.POINTER(C.c_void_p)),
                ("b_down", C.POINTER(C.c_void_p)), ("act_fmt", C.c_int)]


def lib():
    global _lib
    with _lock:
        if _lib is None:
            build(force=False)
            L = C.CDLL(_LIB)
            p = C.c_void_p
            L.orc_route.argtypes = [p, C.c_int, C.c_int, C.c_int, C.c_int, p, p]
            L.orc_route_grouped.argtypes = [p, p, C.c_int, C.c_int, C.c_int, C.c_int, C.c_int, C.c_double, p, p]
            L.orc_router_logits.argtypes = [p, p, C.c_int, C.c_int, C.c_int, p]
            L.orc_union.argtypes = [p, C.c_int, C.c_int, C.c_int, p, p, p, p, p]
            L.orc_verify_tokens.argtypes = [C.POINTER(_Layer), p, C.c_int, C.c_int, p, p, C.c_int, p, p,
                                            C.c_int]
            L.orc_decode_table.argtypes = [C.c_int, p]
            L.orc_weight_at.argtypes = [C.c_int, p, p, C.c_int, C.c_int, C.c_int, C.c_int]
            L.orc_weight_at.restype = C.c_double
            L.orc_expert_bytes.argtypes = [C.c_int, C.c_long, C.c_long, C.POINTER(C.c_long),
                                           C.POINTER(C.c_long)]
            L.orc_mx_quant.argtypes = [p, C.c_int, p]
            _lib = L
    return _lib


def _np(a, dtype):
    """Contiguous numpy view of a numpy array or CPU torch tensor, reinterpreted as dtype."""
    if hasattr(a, "detach"):
        a = a.detach().cpu().contiguous()
        if str(a.dtype) in ("torch.bfloat16", "torch.float8_e4m3fn"):
            import torch
            a = a.view(torch.uint16 if a.dtype == torch.bfloat16 else torch.uint8)
        a = a.numpy()
    a = np.ascontiguousarray(a)
    if a.dtype != np.dtype(dtype):
        if a.dtype.itemsize == np.dtype(dtype).itemsize and a.dtype.kind in "ui" and np.dtype(dtype).kind in "ui":
            a = a.view(dtype)
        else:
            a = a.astype(dtype)
    return a


def _ptr(a) -> int:
    return a.ctypes.data


def route(logits, k: int, score: int):
    lg = _np(logits, np.float32)
    T, E = lg.shape
    idx = np.zeros((T, k), np.int32)
    w = np.zeros((T, k), np.float64)
    rc = lib().orc_route(_ptr(lg), T, E, k, score, _ptr(idx), _ptr(w))
    if rc:
        raise ValueError(f"orc_route rc={rc}")
    return idx, w


def route_grouped(logits, bias, k: int, n_group: int, topk_group: int, scale: float):
    lg = _np(logits, np.float32)
    T, E = lg.shape
    b = None if bias is None else _np(bias, np.float32)
    idx = np.zeros((T, k), np.int32)
    w = np.zeros((T, k), np.float64)
    rc = lib().orc_route_grouped(_ptr(lg), None if b is None else _ptr(b), T, E, k, n_group, topk_group,
                                 float(scale), _ptr(idx), _ptr(w))
    if rc:
        raise ValueError(f"orc_route_grouped rc={rc}")
    return idx, w


def router_logits(x, w_router):
    """fp64 x . W_r^T of bf16 x [T, d] and W_r [E, d] (torch bf16 tensors or uint16 bit arrays)."""
    xb = _np(x, np.uint16)
    wb = _np(w_router, np.uint16)
    T, d = xb.shape
    E = wb.shape[0]
    out = np.zeros((T, E), np.float64)
    rc = lib().orc_router_logits(_ptr(xb), _ptr(wb), T, d, E, _ptr(out))
    if rc:
        raise ValueError(f"orc_router_logits rc={rc}")
    return out


def union(idx, E: int) -> dict:
    ix = _np(idx, np.int32)
    T, k = ix.shape
    out = dict(counts=np.zeros(E, np.int32), union_ids=np.zeros(E, np.int32),
               n_unique=np.zeros(1, np.int32), offsets=np.zeros(E + 1, np.int32),
               perm=np.zeros(T * k, np.int32))
    rc = lib().orc_union(_ptr(ix), T, k, E, _ptr(out["counts"]), _ptr(out["union_ids"]),
                         _ptr(out["n_unique"]), _ptr(out["offsets"]), _ptr(out["perm"]))
    if rc:
        raise ValueError(f"orc_union rc={rc}")
    out["n_unique"] = int(out["n_unique"][0])
    return out


def _expert_ptrs(mats, n):
    arr = (C.c_void_p * n)()
    keep = []
    for e in range(n):
        m = mats(e)
        if m is not None:
            keep.append(m)
            arr[e] = _ptr(m)
    return arr, keep


def verify_tokens(layer: dict, x, idx, w, tokens=None, threads: int = 1):
    """fp64 y rows for the given tokens (default: all).

    ``layer`` holds fmt, d, d_ff and either stacked arrays gate/up/down
    [E, N, K(/2)] (+ s_gate/s_up/s_down) or dicts {expert id: array} for just
    the experts that are needed, plus optional sh_* arrays of the shared expert,
    optional fp32 biases b_gate/b_up [E, d_ff] and b_down [E, d] (same forms) and
    the activation: act 0 (SwiGLU, default) or 1 (GPT-OSS clamped SwiGLU with
    alpha and limit), and act_fmt 1 for MX FP8 quantised projection inputs
    (``mx_quantize``).
    """
    fmt, d, d_ff = int(layer["fmt"]), int(layer["d"]), int(layer["d_ff"])
    wdt = {0: np.uint16, 1: np.uint8, 2: np.uint8}[fmt]
    sdt = {0: None, 1: np.float32, 2: np.uint8}[fmt]
    xa = _np(x, np.uint16)
    ix = _np(idx, np.int32)
    wa = _np(w, np.float64)
    T, k = ix.shape
    toks = np.arange(T, dtype=np.int32) if tokens is None else np.asarray(tokens, np.int32)
    n_exp = int(ix.max()) + 1 if ix.size else 1
    keep = []

    def getter(name, dt):
        src = layer.get(name)
        if src is None:
            return None
        if isinstance(src, dict):
            def f(e):
                return _np(src[e], dt) if e in src else None
        else:
            def f(e):
                return _np(src[e], dt) if e < len(src) else None
        return f

    lay = _Layer()
    lay.fmt, lay.d, lay.d_ff, lay.n_experts = fmt, d, d_ff, n_exp
    lay.act = int(layer.get("act", 0))
    lay.act_fmt = int(layer.get("act_fmt", 0))
    lay.alpha = float(layer.get("alpha", 1.702))
    lay.limit = float(layer.get("limit", 7.0))
    for name in ("b_gate", "b_up", "b_down"):
        g = getter(name, np.float32)
        if g is not None:
            arr, kp = _expert_ptrs(g, n_exp)
            keep += [arr, kp]
            setattr(lay, name, C.cast(arr, C.POINTER(C.c_void_p)))
    for name in ("gate", "up", "down"):
        arr, kp = _expert_ptrs(getter(name, wdt), n_exp)
        keep += [arr, kp]
        setattr(lay, name, C.cast(arr, C.POINTER(C.c_void_p)))
        g = getter("s_" + name, sdt) if sdt is not None else None
        if g is not None:
            arr, kp = _expert_ptrs(g, n_exp)
            keep += [arr, kp]
            setattr(lay, "s_" + name, C.cast(arr, C.POINTER(C.c_void_p)))
        if layer.get("sh_" + name) is not None:
            m = _np(layer["sh_" + name], wdt).reshape(-1)
            keep.append(m)
            setattr(lay, "sh_" + name, _ptr(m))
            if sdt is not None:
                s = _np(layer["sh_s_" + name], sdt).reshape(-1)
                keep.append(s)
                setattr(lay, "sh_s_" + name, _ptr(s))
    y = np.zeros((len(toks), d), np.float64)
    rc = lib().orc_verify_tokens(C.byref(lay), _ptr(xa), T, k, _ptr(ix), _ptr(wa), len(toks), _ptr(toks),
                                 _ptr(y), int(threads))
    if rc:
        raise ValueError(f"orc_verify_tokens rc={rc}")
    return y


def mx_quantize(v) -> tuple[np.ndarray, np.ndarray]:
    """OCP MX FP8 quantisation of one activation row (the optional act_fmt 1 mode):
    returns the quantised fp64 values and the exponent E of every block of 32."""
    a = np.array(v, dtype=np.float64).reshape(-1)
    K = a.size
    exps = np.zeros((K + 31) // 32, np.int32)
    rc = lib().orc_mx_quant(_ptr(a), K, _ptr(exps))
    if rc:
        raise ValueError(f"orc_mx_quant rc={rc}")
    return a, exps


def decode_table(kind: int) -> np.ndarray:
    n = {0: 256, 1: 16, 2: 256, 3: 65536}[kind]
    out = np.zeros(n, np.float64)
    lib().orc_decode_table(kind, _ptr(out))
    return out


def weight_at(fmt: int, w, s, n: int, c: int) -> float:
    """Decoded element (n, c) of one matrix w [N, K] (bf16 bits, e4m3 codes or packed e2m1)."""
    wdt = {0: np.uint16, 1: np.uint8, 2: np.uint8}[fmt]
    wa = _np(w, wdt)
    N = wa.shape[0]
    K = wa.shape[1] * (2 if fmt == 2 else 1)
    sa = None if s is None else _np(s, np.float32 if fmt == 1 else np.uint8)
    return lib().orc_weight_at(fmt, _ptr(wa), None if sa is None else _ptr(sa), N, K, n, c)


def expert_bytes(fmt: int, d: int, d_ff: int) -> tuple[int, int]:
    wb, sb = C.c_long(), C.c_long()
    lib().orc_expert_bytes(fmt, d, d_ff, C.byref(wb), C.byref(sb))
    return wb.value, sb.value
