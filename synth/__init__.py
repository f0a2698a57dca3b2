"""Seeded synthetic inputs for the MoE verification pass.

This module only *draws* inputs: activations, router logits, expert weights
in the three storage formats, and draft trees with per-node expert sets.  It
contains none of the verification arithmetic (no top-k, no union, no decode,
no FFN, no selection score), so both the CPU oracle and the HIP path can be
fed from it without sharing any of the method's code.

All draws go through ``torch.Generator`` objects seeded from (seed, tag), on
the device the caller names.  A given (seed, tag, device type) always yields
the same bytes; tests draw once and hand the same bytes to both sides.

Shapes follow the models of the paper's Table 13 (appendix "Model Details"):
DeepSeek-V3.1 (256 routed + 1 shared experts, top-8), Qwen3-235B-A22B (128,
top-8) and GPT-OSS-120B (128, top-4).  Real weights, router traces and the
benchmark datasets are not available; these generators stand in for them.
"""
from __future__ import annotations

import hashlib
import math
from dataclasses import dataclass

import numpy as np
import torch

__all__ = [
    "Shape", "SHAPES", "expert_bytes", "generator", "activations",
    "logits_scattered", "routes_clustered", "routes_exact_u", "routes_to_logits",
    "logits_tie_grid", "weights_bf16", "weights_fp8_b128", "weights_mxfp4",
    "layer_weights", "draft_tree", "tree_expert_sets", "FMT_BF16", "FMT_FP8",
    "FMT_MXFP4",
]

FMT_BF16 = 0    # bf16 [E][N][K]
FMT_FP8 = 1     # e4m3fn [E][N][K] + fp32 scales [E][N/128][K/128]
FMT_MXFP4 = 2   # e2m1 packed [E][N][K/2] (low nibble = even K) + e8m0 [E][N][K/32]


@dataclass(frozen=True)
class Shape:
    """One MoE layer shape: hidden d, expert width d_ff, E routed experts, top-k."""
    name: str
    d: int
    d_ff: int
    E: int
    k: int
    fmt: int
    score: int          # 0 = softmax over the selected logits, 1 = sigmoid renormalised
    shared: bool        # one always-on shared expert (DeepSeek-V3.1)


SHAPES = {
    "toy": Shape("toy", 256, 128, 16, 2, FMT_BF16, 0, False),
    "qwen": Shape("qwen", 4096, 1536, 128, 8, FMT_BF16, 0, False),
    "ds": Shape("ds", 7168, 2048, 256, 8, FMT_FP8, 1, True),
    "gpt": Shape("gpt", 2880, 2880, 128, 4, FMT_MXFP4, 0, False),
}


def expert_bytes(d: int, d_ff: int, fmt: int) -> tuple[int, int]:
    """(weight bytes, scale bytes) of one SwiGLU expert (gate, up, down) in a storage format."""
    n = 3 * d * d_ff
    if fmt == FMT_BF16:
        return 2 * n, 0
    if fmt == FMT_FP8:
        return n, 4 * 3 * (d // 128) * (d_ff // 128)
    if fmt == FMT_MXFP4:
        return n // 2, n // 32
    raise ValueError(fmt)


def _seed_of(seed: int, tag: str) -> int:
    h = hashlib.blake2b(f"{seed}/{tag}".encode(), digest_size=8).digest()
    return int.from_bytes(h, "little") & ((1 << 63) - 1)


def generator(seed: int, tag: str, device="cpu") -> torch.Generator:
    g = torch.Generator(device=torch.device(device))
    g.manual_seed(_seed_of(seed, tag))
    return g


def _rng(seed: int, tag: str) -> np.random.Generator:
    return np.random.default_rng(_seed_of(seed, tag))


# --------------------------------------------------------------------------- activations / logits

def activations(T: int, d: int, seed: int = 0, device="cpu", tag="x") -> torch.Tensor:
    """x ~ N(0,1), rounded to bf16, shape [T, d]."""
    g = generator(seed, tag, device)
    return torch.randn(T, d, generator=g, device=device, dtype=torch.float32).to(torch.bfloat16)


def logits_scattered(T: int, E: int, seed: int = 0, device="cpu", tag="logits") -> torch.Tensor:
    """Independent N(0,1) fp32 router logits [T, E] (diffuse routing)."""
    g = generator(seed, tag, device)
    return torch.randn(T, E, generator=g, device=device, dtype=torch.float32)


def router_bias(E: int, seed: int = 0, device="cpu", tag="rbias", amp: float = 0.1) -> torch.Tensor:
    """fp32 per-expert routing correction bias [E] ~ U(-amp, amp)."""
    g = generator(seed, tag, device)
    return (torch.rand(E, generator=g, device=device) * 2 - 1) * amp


def logits_tie_grid(T: int, E: int, seed: int = 0, device="cpu", tag="ties") -> torch.Tensor:
    """Logits on a 0.5 grid in [-2, 2], so that many entries tie exactly (incl. -0.0)."""
    g = generator(seed, tag, device)
    v = torch.randint(-4, 5, (T, E), generator=g, device=device).to(torch.float32) * 0.5
    coin = torch.randint(0, 2, (T, E), generator=g, device=device).bool()
    neg_zero = torch.full_like(v, -0.0)
    return torch.where((v == 0) & coin, neg_zero, v)


def routes_clustered(T: int, E: int, k: int, p: float, seed: int = 0, tag="clustered") -> np.ndarray:
    """Expert lists [T, k] for tokens laid out as a binary heap tree (parent(t) = (t-1)//2).

    Each of a token's k slots takes a not-yet-used expert of its parent with
    probability p, otherwise a uniform expert not already in its list.  This
    mimics the locality of draft-tree routing (children reuse parent experts).
    """
    rng = _rng(seed, tag)
    out = np.zeros((T, k), dtype=np.int64)
    for t in range(T):
        chosen: list[int] = []
        parent = list(out[(t - 1) // 2]) if t > 0 else []
        for _ in range(k):
            unused = [e for e in parent if e not in chosen]
            if unused and rng.random() < p:
                chosen.append(int(unused[rng.integers(len(unused))]))
            else:
                free = np.setdiff1d(np.arange(E), np.array(chosen, dtype=np.int64))
                chosen.append(int(free[rng.integers(len(free))]))
        out[t] = chosen
    return out


def routes_exact_u(T: int, E: int, k: int, U: int, seed: int = 0, tag="exactu") -> np.ndarray:
    """Expert lists [T, k] whose union has exactly U experts (needs k <= U <= T*k, U <= E).

    A seeded permutation of the E experts gives a list L of U experts; slot j
    of token t takes L[(t*k + j) mod U].  Consecutive slots are distinct when
    U >= k, and every one of the U experts is used when T*k >= U.
    """
    if not (k <= U <= min(E, T * k)):
        raise ValueError(f"need k <= U <= min(E, T*k); got T={T} k={k} U={U} E={E}")
    rng = _rng(seed, tag)
    L = rng.permutation(E)[:U]
    slots = (np.arange(T)[:, None] * k + np.arange(k)[None, :]) % U
    return L[slots].astype(np.int64)


def routes_to_logits(routes: np.ndarray, E: int, seed: int = 0, device="cpu", tag="rlogits") -> torch.Tensor:
    """fp32 logits [T, E] whose descending order starts with each row of ``routes``.

    The expert in position r gets 9 - 0.25 r + N(0, 0.01); the others get
    N(0, 1) clipped to [-4, 4].  The 0.25 spacing dominates the noise, so the
    top-k list (in order) is exactly the given one.
    """
    T, k = routes.shape
    rng = _rng(seed, tag)
    lg = np.clip(rng.standard_normal((T, E)), -4.0, 4.0)
    rank = np.arange(k)[None, :]
    noise = np.clip(rng.standard_normal((T, k)) * 0.01, -0.05, 0.05)
    np.put_along_axis(lg, routes, 9.0 - 0.25 * rank + noise, axis=1)
    return torch.from_numpy(lg.astype(np.float32)).to(device)


# --------------------------------------------------------------------------- weights

def weights_bf16(n_exp: int, N: int, K: int, seed: int = 0, tag="w", device="cpu", std: float = 0.02) -> torch.Tensor:
    """bf16 weights [n_exp, N, K] ~ N(0, std), stored out x in (K contiguous)."""
    g = generator(seed, tag, device)
    out = torch.empty(n_exp, N, K, dtype=torch.bfloat16, device=device)
    for e in range(n_exp):
        out[e] = (torch.randn(N, K, generator=g, device=device) * std).to(torch.bfloat16)
    return out


def router_weight(E: int, d: int, seed: int = 0, device="cpu", tag="router", std: float = 0.02) -> torch.Tensor:
    """bf16 router matrix W_r [E, d] ~ N(0, std), d contiguous."""
    g = generator(seed, tag, device)
    return (torch.randn(E, d, generator=g, device=device) * std).to(torch.bfloat16)


def expert_biases(n_exp: int, N: int, seed: int = 0, tag="b", device="cpu", std: float = 0.5) -> torch.Tensor:
    """fp32 per-expert biases [n_exp, N] ~ N(0, std)."""
    g = generator(seed, tag, device)
    return torch.randn(n_exp, N, generator=g, device=device) * std


def weights_fp8_b128(n_exp: int, N: int, K: int, seed: int = 0, tag="w", device="cpu",
                     std: float = 0.02) -> tuple[torch.Tensor, torch.Tensor]:
    """FP8 e4m3fn codes [n_exp, N, K] (uint8) and fp32 block scales [n_exp, N/128, K/128].

    Each 128x128 block draws N(0, std * 2^u) with u uniform in {-2..2}; its
    scale is amax/448 and the codes are the RNE e4m3fn rounding of w / scale.
    The decoded weight of element (n, c) is e4m3fn(q[n, c]) * s[n//128, c//128].
    """
    if N % 128 or K % 128:
        raise ValueError("FP8 block-scaled weights need N and K multiples of 128")
    g = generator(seed, tag, device)
    nb, kb = N // 128, K // 128
    q = torch.empty(n_exp, N, K, dtype=torch.uint8, device=device)
    s = torch.empty(n_exp, nb, kb, dtype=torch.float32, device=device)
    for e in range(n_exp):
        u = torch.randint(-2, 3, (nb, kb), generator=g, device=device).to(torch.float32)
        sig = std * torch.exp2(u)
        w = torch.randn(nb, 128, kb, 128, generator=g, device=device) * sig[:, None, :, None]
        amax = w.abs().amax(dim=(1, 3)).clamp_min(1e-12)
        sc = (amax / 448.0).to(torch.float32)
        r = (w / sc[:, None, :, None]).clamp(-448.0, 448.0)
        q[e] = r.to(torch.float8_e4m3fn).view(torch.uint8).reshape(N, K)
        s[e] = sc
    return q, s


def weights_mxfp4(n_exp: int, N: int, K: int, seed: int = 0, tag="w", device="cpu",
                  scale_codes=(119, 120, 121)) -> tuple[torch.Tensor, torch.Tensor]:
    """MXFP4 weights: packed e2m1 codes [n_exp, N, K/2] and e8m0 scale codes [n_exp, N, K/32].

    Both nibbles of every byte are uniform over the 16 e2m1 codes (low nibble
    holds the even K index).  Scale codes are uniform over ``scale_codes``.
    """
    if K % 32:
        raise ValueError("MXFP4 weights need K a multiple of 32")
    g = generator(seed, tag, device)
    q = torch.randint(0, 256, (n_exp, N, K // 2), generator=g, device=device, dtype=torch.int32).to(torch.uint8)
    lo, hi = min(scale_codes), max(scale_codes)
    sc = torch.randint(lo, hi + 1, (n_exp, N, K // 32), generator=g, device=device, dtype=torch.int32).to(torch.uint8)
    return q, sc


def layer_weights(shape: Shape, n_exp: int | None = None, seed: int = 0, device="cpu", layer: int = 0) -> dict:
    """All weights of one layer: routed experts [n_exp] and (if the shape has one) the shared expert.

    Returns a dict with keys gate, up, down (+ s_gate, s_up, s_down for the
    scaled formats) and sh_* for the shared expert (leading dim 1).
    """
    n_exp = shape.E if n_exp is None else n_exp
    d, f = shape.d, shape.d_ff
    out: dict = {"fmt": shape.fmt, "d": d, "d_ff": f, "E": n_exp}

    def one(prefix, count, tagp):
        for name, (N, K) in (("gate", (f, d)), ("up", (f, d)), ("down", (d, f))):
            tag = f"L{layer}/{tagp}/{name}"
            if shape.fmt == FMT_BF16:
                out[prefix + name] = weights_bf16(count, N, K, seed, tag, device)
            elif shape.fmt == FMT_FP8:
                out[prefix + name], out[prefix + "s_" + name] = weights_fp8_b128(count, N, K, seed, tag, device)
            else:
                out[prefix + name], out[prefix + "s_" + name] = weights_mxfp4(count, N, K, seed, tag, device)

    one("", n_exp, "routed")
    if shape.shared:
        one("sh_", 1, "shared")
    return out


# --------------------------------------------------------------------------- draft trees

def draft_tree(n: int, branching: int, seed: int = 0, tag="tree", a: float = 2.0, b: float = 2.0):
    """Heap-ordered draft tree: parent(i) = (i-1)//branching, parent(0) = -1.

    Each non-root node draws a conditional acceptance score c_i ~ Beta(a, b);
    the cumulative path probability is P_i = P_parent * c_i with P_0 = 1.
    Returns (parent int32 [n], P float64 [n]).
    """
    rng = _rng(seed, tag)
    parent = np.array([-1] + [(i - 1) // branching for i in range(1, n)], dtype=np.int32)
    c = rng.beta(a, b, size=n)
    P = np.ones(n, dtype=np.float64)
    for i in range(1, n):
        P[i] = P[parent[i]] * c[i]
    return parent, P


def tree_expert_sets(parent: np.ndarray, L: int, E: int, K: int, p_inherit: float, seed: int = 0,
                     tag="tree_sets") -> np.ndarray:
    """Per-node, per-layer expert lists pred [n, L, K] (int32, distinct within a list).

    The root draws K distinct experts per layer uniformly.  A child's slot
    takes a not-yet-used expert of its parent's list (same layer) with
    probability p_inherit, else a uniform expert not already in its list.
    """
    rng = _rng(seed, tag)
    n = len(parent)
    pred = np.zeros((n, L, K), dtype=np.int32)
    for i in range(n):
        for l in range(L):
            chosen: list[int] = []
            par = list(pred[parent[i], l]) if parent[i] >= 0 else []
            for _ in range(K):
                unused = [e for e in par if e not in chosen]
                if unused and rng.random() < p_inherit:
                    chosen.append(int(unused[rng.integers(len(unused))]))
                else:
                    free = np.setdiff1d(np.arange(E), np.array(chosen, dtype=np.int64))
                    chosen.append(int(free[rng.integers(len(free))]))
            pred[i, l] = chosen
    return pred
