#!/usr/bin/env python3
"""Benchmark of the MoE verification pass on one MI355X.

Workload: one DeepSeek-V3.1-shaped MoE layer (d=7168, d_ff=2048, 256 routed
experts + 1 shared, top-8 sigmoid routing, FP8 e4m3 weights with 128x128
fp32 block scales), T=64 draft tokens whose routing touches exactly U routed
experts (headline U=32).  A step is the whole hot path on the device:
router top-k -> expert union/grouping -> grouped SwiGLU experts -> combine.

Inputs are seeded synthetic draws (no model weights or datasets exist here)
and are resident in HBM before timing starts.  Every timed step routes to a
different expert set and uses one of several shared-expert copies, so each
step streams cold weights (the 256 MB Infinity Cache holds far less than the
~1.45 GB a U=32 step reads).

Prints ONE JSON line on stdout; progress goes to stderr.

    python bench.py [--gpus 1] [--steps 50] [--warmup 100] [--no-sweep] [--no-cpu] [--no-stack]
    python bench.py --profile [--shape ds|gpt]       # short run for rocprofv3 (+ a copy kernel for counter calibration)
    python bench.py --summarize-kstats DIR OUT [--shape ds|gpt]  # rocprofv3 --kernel-trace --stats output -> profiles/ summary
    python bench.py --summarize-pmc FETCH WRITE OUT [--shape ds|gpt]  # rocprofv3 --pmc output -> profiles/ summary
    python bench.py --summarize-sq SQ_A SQ_B OUT [--shape ds|gpt]     # two SQ counter passes -> profiles/ summary
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MoE verify-layer µs and HBM GB/s vs unique experts (V3.1 shape, FP8)"
PEAK_HBM_GBS = 8000.0
PROFILES = os.path.join(ROOT, "profiles")
KSTATS_SUMMARY = os.path.join(PROFILES, "verify_ds_fp8_T64_U32.kernel_stats.txt")
KSTATS_FILES = {"ds": "profiles/verify_ds_fp8_T64_U32.kernel_stats.txt",
                "gpt": "profiles/verify_gpt_mxfp4_T64_U32.kernel_stats.txt"}
PMC_SUMMARY = {"ds": os.path.join(PROFILES, "expert_ffn_ds_fp8_T64_U32.pmc.txt"),
               "gpt": os.path.join(PROFILES, "expert_ffn_gpt_mxfp4_T64_U32.pmc.txt")}
# The expert kernels' sources: the kernel file and the headers it includes.
FFN_SOURCES = [os.path.join(ROOT, "paper_2607_12696_amd", "csrc", f)
               for f in ("expert_ffn.hip", "device.hpp", "launch.hpp", "split.hpp")]
GATEUP_FP8 = "expert_ffn_kernel<1, false"   # demangled-name prefix of the FP8 gate/up kernel
SWEEP_WARMUP = 20                           # untimed steps before each sweep point (the GPU stays busy between points)
COPY_BYTES = 1 << 30                         # calibration copy: reads and writes 1 GiB

# The paper's own end-to-end speedups over autoregressive decoding (maxima over its benchmarks), quoted as
# context: another machine, a whole model and a different runtime, not this layer's target.
PAPER_CONTEXT = {
    "max_speedup_vs_autoregressive": {"Qwen3-235B-A22B": 1.62, "GPT-OSS-120B": 1.50, "DeepSeek-V3.1": 1.47},
    "hardware": "8x NVIDIA H200", "runtime": "HuggingFace Transformers research prototype",
    "workload": "batch 1, greedy decoding, 4 verified tokens per step; end-to-end speedup, not a per-layer number",
    "unique_experts_per_layer_at_4_verified_tokens": {"Qwen3-235B-A22B": [23.7, 20.5], "GPT-OSS-120B": [11.6, 10.6],
                                                      "DeepSeek-V3.1": [31.4, 31.2]},
    "unique_experts_note": "[baseline drafter, cost-aware selection]",
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def source_sha() -> str:
    h = hashlib.sha256()
    for f in FFN_SOURCES:
        h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


def pct(v, q):
    s = sorted(v)
    return s[min(len(s) - 1, max(0, int(round(q * (len(s) - 1)))))]


def dist(v_ms):
    """median / p10 / p90 of per-step times given in ms, in us."""
    return {"median": pct(v_ms, 0.5) * 1e3, "p10": pct(v_ms, 0.1) * 1e3, "p90": pct(v_ms, 0.9) * 1e3}


def linfit(xs, ys):
    n = len(xs)
    mx, my = sum(xs) / n, sum(ys) / n
    sxx = sum((x - mx) ** 2 for x in xs)
    sxy = sum((x - mx) * (y - my) for x, y in zip(xs, ys))
    b = sxy / sxx if sxx else 0.0
    a = my - b * mx
    ss_res = sum((y - (a + b * x)) ** 2 for x, y in zip(xs, ys))
    ss_tot = sum((y - my) ** 2 for y in ys)
    return a, b, (1 - ss_res / ss_tot) if ss_tot else 1.0


# --------------------------------------------------------------------------- byte accounting

def expert_bytes(sh):
    """Weight + scale bytes of one expert (gate, up, down) in the layer's storage format."""
    import synth
    return sum(synth.expert_bytes(sh.d, sh.d_ff, sh.fmt))


def matrix_bytes(sh, N, K):
    """Bytes of one N x K matrix of one expert, scales included (as the kernels stream them)."""
    if sh.fmt == 0:
        return 2 * N * K
    if sh.fmt == 1:
        return N * K + 4 * (N // 128) * (K // 128)
    return N * K // 2 + N * K // 32


def step_alg_bytes(sh, T, U):
    """Algorithmic HBM bytes of one step: every activated expert once, plus the activations, logits
    and routing arrays once each."""
    n_exp = U + (1 if sh.shared else 0)
    routing = 4 * (2 * T * sh.k + T * sh.k + 2 * sh.E + 1 + (sh.E + 1))
    return n_exp * expert_bytes(sh) + 2 * T * sh.d * 2 + 4 * T * sh.E + routing


def kernel_alg_bytes(sh, T, U, down):
    """Algorithmic bytes of one expert launch: its matrices (+ scales) of every activated expert once;
    gate/up also reads x and writes the bf16 SwiGLU rows, down reads those rows and writes fp32 O."""
    n_exp = U + (1 if sh.shared else 0)
    rows = T * sh.k + (T if sh.shared else 0)
    if not down:
        return n_exp * 2 * matrix_bytes(sh, sh.d_ff, sh.d) + 2 * T * sh.d + 2 * rows * sh.d_ff
    return n_exp * matrix_bytes(sh, sh.d, sh.d_ff) + 2 * rows * sh.d_ff + 4 * rows * sh.d


def read_summary(path):
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    return kv if kv.get("kernel_source_sha") == source_sha() else None


def rocprof_gateup_us():
    """Average duration of the FP8 gate/up kernel in the committed rocprofv3 summary of the headline
    steps, or None if it is missing or was taken on another kernel source."""
    kv = read_summary(KSTATS_SUMMARY)
    if not kv:
        return None
    for line in open(KSTATS_SUMMARY):
        if line.startswith(GATEUP_FP8.split("<")[0] + "<1, false") or GATEUP_FP8 in line:
            try:
                return float(line.split("|")[2])
            except (IndexError, ValueError):
                return None
    return None


# --------------------------------------------------------------------------- workloads

class Layer:
    """A layer's weights on the device (interchange layout for the oracle, packed for the kernels).
    DeepSeek-shaped layers also get extra copies of the shared expert, rotated over the steps, so
    that the always-on expert is read cold too."""

    def __init__(self, name, seed=0, n_shared_copies=1):
        import torch
        import synth
        import paper_2607_12696_amd as moe
        self.torch, self.moe, self.synth = torch, moe, synth
        self.dev = torch.device("cuda:0")
        self.sh = sh = synth.SHAPES[name]
        t0 = time.time()
        self.raw = synth.layer_weights(sh, seed=seed, device=self.dev)
        shared = [{k: self.raw[k] for k in self.raw if k.startswith("sh_")}] if sh.shared else [{}]
        for c in range(1, n_shared_copies if sh.shared else 1):
            cp = {}
            for nm, (N, K) in (("gate", (sh.d_ff, sh.d)), ("up", (sh.d_ff, sh.d)), ("down", (sh.d, sh.d_ff))):
                cp["sh_" + nm], cp["sh_s_" + nm] = synth.weights_fp8_b128(1, N, K, seed, f"bench/shared{c}/{nm}",
                                                                          self.dev)
            shared.append(cp)
        routed = moe.pack_layer({k: v for k, v in self.raw.items() if not k.startswith("sh_")})
        self.rawdicts, self.wdicts = [], []
        for cp in shared:
            raw = {k: v for k, v in self.raw.items() if not k.startswith("sh_")}
            raw.update(cp)
            self.rawdicts.append(raw)
            wd = dict(routed)
            if cp:
                wd["sh_gate"], wd["sh_s_gate"], wd["sh_s_up"] = moe.moe_pack_gate_up(
                    sh.fmt, cp["sh_gate"], cp["sh_up"], cp["sh_s_gate"], cp["sh_s_up"])
                wd["sh_down"], wd["sh_s_down"] = moe.moe_pack_down(sh.fmt, cp["sh_down"], cp["sh_s_down"])
            self.wdicts.append(wd)
        torch.cuda.synchronize()
        log(f"{name}: weights generated and packed in {time.time() - t0:.1f}s "
            f"({(sh.E + len(shared) - (0 if sh.shared else 1)) * expert_bytes(sh) / 1e9:.1f} GB)")


class Runner:
    """Preallocated buffers for steps of T tokens on a Layer: nothing is allocated in a timed region."""

    def __init__(self, layer, T, act_fmt=0):
        torch, moe, sh = layer.torch, layer.moe, layer.sh
        self.layer, self.T, self.torch, self.moe, self.sh = layer, T, torch, moe, sh
        dev = layer.dev
        self.wds = [dict(w, act_fmt=act_fmt) for w in layer.wdicts]
        self.x = layer.synth.activations(T, sh.d, seed=1, device=dev)
        self.y = torch.empty_like(self.x)
        i32 = dict(dtype=torch.int32, device=dev)
        self.r = moe.Routing(T, sh.k, sh.E, torch.empty(T, sh.k, **i32),
                             torch.empty(T, sh.k, dtype=torch.float32, device=dev), torch.empty(sh.E, **i32),
                             torch.empty(sh.E, **i32), torch.empty(1, **i32), torch.empty(sh.E + 1, **i32),
                             torch.empty(T * sh.k, **i32))
        self.ws = torch.empty(moe.moe_verify_workspace_size(self.wds[0], T, sh.k), dtype=torch.uint8, device=dev)

    def step(self, lg, i, events=None):
        """One pass of the hot path: the router top-k, then the verification, which builds the expert
        union and grouping itself (in the gate/up kernel; T > 64: a union kernel and the token-group plan
        first).  events = optional 6 marks: before the top-k, then the 5 marks of the timed verify entry
        point (before and after the gate/up expert kernel, before and after the down expert kernel, after
        combine)."""
        moe, sh = self.moe, self.sh
        wd = self.wds[i % len(self.wds)]
        if events is not None:
            events[0].record()
        moe.moe_route_topk(lg, sh.k, sh.score, topk_idx=self.r.topk_idx, topk_w=self.r.topk_w)
        if events is None:
            moe.moe_verify_layer(self.x, wd, self.r, y=self.y, workspace=self.ws)
        else:
            moe.moe_verify_layer_timed(self.x, wd, self.r, self.y, self.ws, events[1:])

    def pool(self, kind, n, U=None, seed=0):
        synth, sh, T, dev = self.layer.synth, self.sh, self.T, self.layer.dev
        out = []
        for i in range(n):
            s = seed + 1000 * T + 17 * i
            if kind == "scattered":
                out.append(synth.logits_scattered(T, sh.E, seed=s, device=dev))
            elif kind == "clustered":
                p = 0.7 if sh.shared else 0.8
                out.append(synth.routes_to_logits(synth.routes_clustered(T, sh.E, sh.k, p, seed=s), sh.E, seed=s,
                                                  device=dev))
            else:
                out.append(synth.routes_to_logits(synth.routes_exact_u(T, sh.E, sh.k, U, seed=s), sh.E, seed=s,
                                                  device=dev))
        return out

    def unique(self, pool):
        out = []
        for i, lg in enumerate(pool):
            self.step(lg, i)
            out.append(int(self.r.n_unique.item()))
        return out

    def time_plain(self, pool, steps, warmup):
        """Mean ms per step over `steps` back-to-back steps (two events around all of them)."""
        torch = self.torch
        for i in range(warmup):
            self.step(pool[i % len(pool)], i)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for i in range(steps):
            self.step(pool[(warmup + i) % len(pool)], warmup + i)
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / steps

    def time_marks(self, pool, steps, warmup):
        """Per-step spans (ms) from HIP events recorded on the launch stream around each kernel."""
        torch = self.torch
        for i in range(warmup):
            self.step(pool[i % len(pool)], i)
        torch.cuda.synchronize()
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(steps)]
        for row in evs:  # torch creates the HIP event on first record; the library records raw handles
            for e in row:
                e.record()
        torch.cuda.synchronize()
        for i in range(steps):
            self.step(pool[(warmup + i) % len(pool)], warmup + i, evs[i])
        torch.cuda.synchronize()
        spans = {"step": (0, 5), "route": (0, 1), "verify": (1, 5), "gateup": (1, 2), "gateup_fixup": (2, 3),
                 "down": (3, 4), "combine": (4, 5)}
        return {k: [e[a].elapsed_time(e[b]) for e in evs] for k, (a, b) in spans.items()}


def point(runner, pool, steps, warmup, U=None):
    """One measured point: the mean time of `steps` unmarked steps (two events around all of them) with its
    algorithmic GB/s, then the same steps run again through the timed entry point for per-kernel medians.
    Every mark adds a few us of launch gap, so the marked step (`marked_step_us`) is longer than `step_us`."""
    sh, T = runner.sh, runner.T
    if U is None:
        U = float(np.median(runner.unique(pool)))
    us = runner.time_plain(pool, steps, warmup) * 1e3
    per = runner.time_marks(pool, steps, 0)
    B = step_alg_bytes(sh, T, U)
    return {"T": T, "U": U, "step_us": us, "GB_s": B / (us * 1e-6) / 1e9,
            "frac_of_8TBs": B / (us * 1e-6) / 1e9 / PEAK_HBM_GBS, "alg_bytes": B,
            "marked_step_us": dist(per["step"]),
            "kernels_us": {k: pct(v, 0.5) * 1e3 for k, v in per.items() if k != "step"}}


# --------------------------------------------------------------------------- sweeps

def u_sweeps(layer, Ts_Us, steps, warmup, n_pool=8):
    """Exact-U routing (a different expert set every step): latency vs unique experts at several T."""
    out = []
    for T, Us in Ts_Us:
        rn = Runner(layer, T)
        pts = []
        for U in Us:
            pool = rn.pool("exact", n_pool, U=U, seed=100 * U)
            p = point(rn, pool, steps, warmup, U=U)
            pts.append(p)
            log(f"  {layer.sh.name} T={T:3d} U={U:4d}: step {p['step_us']:8.1f} us  {p['GB_s']:7.0f} GB/s")
        fit = None
        if len(pts) >= 3:
            a, b, r2 = linfit([p["U"] for p in pts], [p["step_us"] for p in pts])
            fit = {"us_intercept": a, "us_per_expert": b, "r2": r2,
                   "GB_s_marginal": expert_bytes(layer.sh) / (b * 1e-6) / 1e9 if b > 0 else None}
        out.append({"T": T, "points": pts, "linear_fit_us_vs_U": fit})
        del rn
    return out


def routing_grid(layer, Ts, kinds, steps, warmup, n_pool=8, act_fmt=0):
    """Clustered draft-tree-like and scattered (i.i.d.) routing at several T (U is whatever the
    routing touches; its median over the pool is reported)."""
    out = []
    for T in Ts:
        rn = Runner(layer, T, act_fmt=act_fmt)
        for kind in kinds:
            pool = rn.pool(kind, n_pool, seed=7)
            p = point(rn, pool, steps, warmup)
            p["routing"] = kind
            out.append(p)
            log(f"  {layer.sh.name}{' MX act' if act_fmt else ''} T={T:3d} {kind:9s} U~{p['U']:5.1f}: "
                f"step {p['step_us']:8.1f} us  {p['GB_s']:7.0f} GB/s")
        del rn
    return out


def token_sweep(layer, Ms=(1, 4, 16, 32, 64), U=32, steps=20, warmup=None, n_pool=8, act_fmt=0):
    """Tokens per expert: exact-U routing with T = M * U / k gives each of the U experts exactly M tokens
    (and the shared expert T).  Per-kernel medians show where the matrix-core work of a step starts
    to cost on top of the weight stream."""
    sh = layer.sh
    n_exp = U + (1 if sh.shared else 0)
    warmup = SWEEP_WARMUP if warmup is None else warmup
    out = []
    for M in Ms:
        T = M * U // sh.k
        if T < 1 or T * sh.k != M * U:
            continue
        rn = Runner(layer, T, act_fmt=act_fmt)
        pool = rn.pool("exact", n_pool, U=U, seed=700 * M)
        step_us = rn.time_plain(pool, steps, warmup) * 1e3  # unmarked steps
        per = rn.time_marks(pool, steps, 0)
        med = {k: 1e3 * pct(v, 0.5) for k, v in per.items()}
        gu, dn = kernel_alg_bytes(sh, T, U, False), kernel_alg_bytes(sh, T, U, True)
        pt = {"M": M, "T": T, "step_us": step_us, "gateup_us": med["gateup"], "fixup_us": med["gateup_fixup"],
              "down_us": med["down"], "combine_us": med["combine"],
              "gateup_GB_s": gu / (med["gateup"] * 1e-6) / 1e9, "down_GB_s": dn / (med["down"] * 1e-6) / 1e9,
              "step_GB_s": n_exp * expert_bytes(sh) / (step_us * 1e-6) / 1e9}
        out.append(pt)
        log(f"  {sh.name}{' MX act' if act_fmt else ''} M={M:3d} (T={T:4d}): step {pt['step_us']:7.1f} us, "
            f"gate/up {pt['gateup_us']:6.1f} us ({pt['gateup_GB_s']:5.0f} GB/s), "
            f"down {pt['down_us']:6.1f} us ({pt['down_GB_s']:5.0f} GB/s)")
        del rn
    return {"shape": sh.name, "fmt": sh.fmt, "act_fmt": act_fmt, "U": U, "points": out}


def graph_us(torch, fn, reps=20, replays=10):
    """fn captured `reps` times in one HIP graph, replayed: host launch cost does not enter."""
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        fn()
    torch.cuda.current_stream().wait_stream(s)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(reps):
            fn()
    g.replay()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(replays):
        g.replay()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) * 1e3 / (reps * replays)


def router_timing(layer, T=64):
    """Router from hidden states (x . W_r^T in split-K on the matrix cores, then the top-k that sums the
    K slices) against top-k from given logits, and DeepSeek-V3 group-limited routing against plain
    sigmoid top-8 on the same logits."""
    torch, moe, synth, sh, dev = layer.torch, layer.moe, layer.synth, layer.sh, layer.dev
    x = synth.activations(T, sh.d, seed=2, device=dev)
    w_r = synth.router_weight(sh.E, sh.d, seed=3, device=dev)
    ws = torch.empty(moe.moe_router_workspace_size(T, sh.d, sh.E), dtype=torch.uint8, device=dev)
    idx = torch.empty(T, sh.k, dtype=torch.int32, device=dev)
    tw = torch.empty(T, sh.k, dtype=torch.float32, device=dev)
    lg = torch.empty(T, sh.E, dtype=torch.float32, device=dev)
    idx2, tw2 = torch.empty_like(idx), torch.empty_like(tw)
    moe.moe_route_topk_hidden(x, w_r, sh.k, sh.score, logits=lg, workspace=ws, topk_idx=idx, topk_w=tw)
    moe.moe_route_topk(lg, sh.k, sh.score, topk_idx=idx2, topk_w=tw2)
    torch.cuda.synchronize()
    consistent = bool(torch.equal(idx, idx2) and torch.equal(tw, tw2))
    hid = graph_us(torch, lambda: moe.moe_route_topk_hidden(x, w_r, sh.k, sh.score, workspace=ws, topk_idx=idx,
                                                            topk_w=tw))
    lgt = graph_us(torch, lambda: moe.moe_route_topk(lg, sh.k, sh.score, topk_idx=idx2, topk_w=tw2))
    bias = synth.router_bias(sh.E, seed=3, device=dev)
    grp = graph_us(torch, lambda: moe.moe_route_topk_grouped(lg, bias, sh.k, 8, 4, 2.5, topk_idx=idx, topk_w=tw))
    return {"T": T, "d": sh.d, "E": sh.E, "router_from_hidden_us": hid, "route_from_logits_us": lgt,
            "grouped_route_us": grp, "router_gemm_bytes": 2 * sh.E * sh.d + 2 * T * sh.d,
            "routing_matches_logits_entry": consistent}


def gpt_variants(layer, T=64, steps=30, warmup=None, n_pool=8):
    """GPT-OSS-shaped layer, clustered routing: plain SwiGLU against the GPT-OSS expert (biases, clamped
    SwiGLU) and against MX FP8 activations."""
    torch, moe, synth, sh, dev = layer.torch, layer.moe, layer.synth, layer.sh, layer.dev
    ext = dict(act=moe.MOE_ACT_SWIGLU_OAI, alpha=1.702, limit=7.0,
               b_gate=synth.expert_biases(sh.E, sh.d_ff, 0, "bg", dev), b_up=synth.expert_biases(sh.E, sh.d_ff, 0, "bu", dev),
               b_down=synth.expert_biases(sh.E, sh.d, 0, "bd", dev))
    out = {}
    for name, act_fmt, extra in (("plain_swiglu", 0, {}), ("gpt_oss_expert", 0, ext), ("mx_fp8_activations", 1, {})):
        rn = Runner(layer, T, act_fmt=act_fmt)
        rn.wds = [dict(w, **extra) for w in rn.wds]
        pool = rn.pool("clustered", n_pool, seed=50)
        p = point(rn, pool, steps, SWEEP_WARMUP if warmup is None else warmup)
        out[name] = {"U": p["U"], "step_us": p["step_us"], "GB_s": p["GB_s"]}
        log(f"  gpt T={T} clustered {name}: step {p['step_us']:.1f} us")
        del rn
    return out


# --------------------------------------------------------------------------- CPU baseline (oracle)

def cpu_baseline(layer, rn, lg, U, n_tokens):
    """The oracle on the host cores for n_tokens of the headline step; returns the baseline dict and the
    sampled rows' max error of the GPU output against it."""
    import oracle
    torch, sh = layer.torch, layer.sh
    rn.step(lg, 0)
    torch.cuda.synchronize()
    y_gpu = rn.y.float().cpu().numpy()
    idx_o, w_o = oracle.route(lg.cpu().numpy(), sh.k, sh.score)
    rows = list(range(n_tokens))
    used = sorted(set(idx_o[rows].reshape(-1).tolist()))
    wd = layer.rawdicts[0]
    hl = {"fmt": sh.fmt, "d": sh.d, "d_ff": sh.d_ff}
    for n in ("gate", "up", "down", "s_gate", "s_up", "s_down"):
        hl[n] = {e: wd[n][e].cpu() for e in used}
    for n in ("sh_gate", "sh_up", "sh_down", "sh_s_gate", "sh_s_up", "sh_s_down"):
        hl[n] = wd[n].cpu()
    x_h = rn.x.cpu()
    threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or min(16, os.cpu_count() or 1)
    t0 = time.time()
    y_ref = oracle.verify_tokens(hl, x_h, idx_o, w_o, tokens=rows, threads=threads)
    dt = time.time() - t0
    full = dt * rn.T / n_tokens   # the oracle's cost is proportional to the token count
    err = float(np.abs(y_gpu[rows] - y_ref).max() / np.abs(y_ref).max())
    cpu_model = ""
    try:
        with open("/proc/cpuinfo") as f:
            cpu_model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), "")
    except OSError:
        pass
    base = {"value": step_alg_bytes(sh, rn.T, U) / full / 1e9, "unit": "GB/s", "cores": threads, "kind": "oracle",
            "nproc": os.cpu_count(), "cpu_model": cpu_model, "omp_num_threads": os.environ.get("OMP_NUM_THREADS"),
            "sample": f"fp64 C oracle on {n_tokens} of the {rn.T} tokens of the same step (U={U}), "
                      f"{n_tokens * (sh.k + 1)} expert FFNs in {dt:.2f}s; scaled x{rn.T / n_tokens:g} to the "
                      f"whole step ({full:.1f}s)"}
    return base, err


# --------------------------------------------------------------------------- 8-layer verification step

class Stack:
    """Eight DeepSeek-V3.1-shaped FP8 MoE layers verifying T=16 tokens of synthetic 64-node draft trees
    (branching 4, per-node scores ~ Beta(2,2), children inherit a parent expert per slot with probability
    0.7), the tokens chosen by confidence (highest path score first), by the cost-aware selector
    (Algorithm 1, Eq. 9) and by the global-cost ablation (Eq. 10), over several seeded trees.  Each
    layer's routing comes from synthetic router logits whose top-8 are the nodes' expert sets, and each
    layer gets its own synthetic N(0,1) hidden states (there is no model around the MoE layers to carry
    them: no norm or residual, without which stacked random layers overflow bf16)."""

    L, N_NODES, BRANCH, BUDGET, P_INHERIT = 8, 64, 4, 16, 0.7
    SELECTORS = ("confidence", "cost_aware", "global_cost")

    def __init__(self, seed=0):
        import torch
        import synth
        import paper_2607_12696_amd as moe
        self.torch, self.moe, self.synth = torch, moe, synth
        self.dev = torch.device("cuda:0")
        sh = self.sh = synth.SHAPES["ds"]
        self.seed = seed
        t0 = time.time()
        self.layers = []
        for l in range(self.L):
            raw = synth.layer_weights(sh, seed=seed + 17, device=self.dev, layer=l)
            self.layers.append(moe.pack_layer(raw))
            del raw
        torch.cuda.synchronize()
        log(f"stack: {self.L} layers packed in {time.time() - t0:.1f}s")
        T = self.BUDGET
        i32 = dict(dtype=torch.int32, device=self.dev)
        self.xs = [synth.activations(T, sh.d, seed=seed + 5 + l, device=self.dev) for l in range(self.L)]
        self.ys = [torch.empty_like(x) for x in self.xs]
        self.ws = torch.empty(moe.moe_verify_workspace_size(self.layers[0], T, sh.k), dtype=torch.uint8,
                              device=self.dev)
        self.routs = [moe.Routing(T, sh.k, sh.E, torch.empty(T, sh.k, **i32),
                                  torch.empty(T, sh.k, dtype=torch.float32, device=self.dev),
                                  torch.empty(sh.E, **i32), torch.empty(sh.E, **i32), torch.empty(1, **i32),
                                  torch.empty(sh.E + 1, **i32), torch.empty(T * sh.k, **i32)) for _ in range(self.L)]

    def tree(self, t):
        """Selections and per-layer logits of seeded tree t."""
        moe, synth, sh = self.moe, self.synth, self.sh
        parent, P = synth.draft_tree(self.N_NODES, self.BRANCH, seed=self.seed + t)
        pred = synth.tree_expert_sets(parent, self.L, sh.E, sh.k, self.P_INHERIT, seed=self.seed + t)
        modes = {"confidence": moe.MOE_SEL_CONFIDENCE, "cost_aware": moe.MOE_SEL_COST_RATIO,
                 "global_cost": moe.MOE_SEL_GLOBAL_COST}
        out = {}
        for name in self.SELECTORS:
            nodes = moe.moe_select_tree(parent, P, pred, sh.E, self.BUDGET, mode=modes[name])[0]
            logits = [synth.routes_to_logits(pred[nodes, l, :], sh.E, seed=self.seed + 100 * l + 1, device=self.dev)
                      for l in range(self.L)]
            out[name] = (nodes, logits, float(P[nodes].sum()))
        return out

    def run(self, logits):
        """The 8-layer pass for one selection; returns the layer outputs."""
        moe, sh = self.moe, self.sh
        for l in range(self.L):
            r = self.routs[l]
            moe.moe_route_topk(logits[l], sh.k, sh.score, topk_idx=r.topk_idx, topk_w=r.topk_w)
            moe.moe_verify_layer(self.xs[l], self.layers[l], self.routs[l], y=self.ys[l], workspace=self.ws)
        return self.ys

    def time_us(self, logits, steps, warmup):
        torch = self.torch
        for _ in range(warmup):
            self.run(logits)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(steps):
            self.run(logits)
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e3 / steps

    def graph_check(self, logits, steps):
        """The same pass captured once as a HIP graph and replayed; every replay is checked bit for bit
        against the eager result, with eager work between the replays."""
        torch = self.torch
        torch.cuda.synchronize()
        ref = torch.stack(self.run(logits)).clone()
        g = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            self.run(logits)
        torch.cuda.current_stream().wait_stream(s)
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            self.run(logits)
        ok = True
        for _ in range(3):
            g.replay()
            torch.cuda.synchronize()
            ok &= bool(torch.equal(torch.stack(self.ys), ref))
            self.run(logits)
            torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(steps):
            g.replay()
        b.record()
        torch.cuda.synchronize()
        ok &= bool(torch.equal(torch.stack(self.ys), ref))
        finite = bool(torch.isfinite(ref.float()).all())
        del g
        return a.elapsed_time(b) * 1e3 / steps, ok, finite

    def measure(self, trees, steps, warmup):
        out = {"layers": self.L, "T": self.BUDGET, "tree_nodes": self.N_NODES, "branching": self.BRANCH,
               "p_inherit": self.P_INHERIT, "trees": []}
        for t in range(trees):
            sel = self.tree(t)
            row = {"tree_seed": self.seed + t}
            for name, (nodes, logits, psum) in sel.items():
                us = self.time_us(logits, steps, warmup)
                uniq = [int(r.n_unique.item()) for r in self.routs]
                row[name] = {"unique_expert_layers": sum(uniq), "unique_experts_per_layer": uniq, "stack_us": us,
                             "sum_path_prob": psum, "nodes": [int(v) for v in nodes]}
                if t == 0:
                    g_us, ok, finite = self.graph_check(logits, steps)
                    row[name].update({"graph_us": g_us, "graph_replays_match_eager": ok, "outputs_finite": finite})
            out["trees"].append(row)
            log(f"stack tree {t}: " + ", ".join(f"{n} {row[n]['unique_expert_layers']} expert-layers "
                                                f"{row[n]['stack_us']:.0f} us" for n in self.SELECTORS))
        summ = {}
        for name in self.SELECTORS:
            u = np.array([r[name]["unique_expert_layers"] for r in out["trees"]], float)
            s = np.array([r[name]["stack_us"] for r in out["trees"]], float)
            summ[name] = {"unique_expert_layers_mean": u.mean(), "unique_expert_layers_std": u.std(ddof=1),
                          "stack_us_mean": s.mean(), "stack_us_std": s.std(ddof=1)}
        conf = np.array([r["confidence"]["stack_us"] for r in out["trees"]])
        for name in ("cost_aware", "global_cost"):
            other = np.array([r[name]["stack_us"] for r in out["trees"]])
            ue = np.array([r["confidence"]["unique_expert_layers"] - r[name]["unique_expert_layers"]
                           for r in out["trees"]])
            summ[name]["speedup_vs_confidence_mean"] = float(np.mean(conf / other))
            summ[name]["expert_layers_saved_vs_confidence_mean"] = float(ue.mean())
            summ[name]["trees_fewer_experts_than_confidence"] = int((ue > 0).sum())
        out["summary"] = summ
        return out


# --------------------------------------------------------------------------- profiler summaries

def summarize_kstats(kt_dir, out_path, shape="ds", last=50, T=64, U=32):
    """The library's kernels of a `rocprofv3 --kernel-trace --stats` run of `bench.py --profile`: duration
    statistics over the last `last` dispatches of each kernel (the timed steps, after the warm-up)."""
    paths = glob.glob(os.path.join(kt_dir, "**", "*kernel_trace.csv"), recursive=True)
    if not paths:
        raise SystemExit(f"no kernel_trace.csv under {kt_dir}")
    runs = {}
    for r in csv.DictReader(open(paths[0])):
        n = r["Kernel_Name"]
        if "ecospec" in n and "pack" not in n:
            runs.setdefault(n, []).append((int(r["Start_Timestamp"]), int(r["End_Timestamp"])))
    rows = []
    for n, v in runs.items():
        v.sort()
        d = [(e - b) / 1e3 for b, e in v[-last:]]
        rows.append((n, len(v), len(d), sum(d) / len(d), min(d), max(d)))
    rows.sort(key=lambda r: -r[3] * r[2])
    name = {"ds": f"DeepSeek-V3.1-shaped FP8 layer, T={T} draft tokens routed to U={U} of 256 experts + 1 shared",
            "gpt": f"GPT-OSS-120B-shaped MXFP4 layer, T={T} draft tokens routed to U={U} of 128 experts"}[shape]
    tu = "" if (T, U) == (64, 32) else f" --T {T} --U {U}"
    out_name = KSTATS_FILES[shape] if (T, U) == (64, 32) else out_path
    with open(out_path, "w") as f:
        f.write(f"# rocprofv3 kernel-trace statistics of the verification pass: {name}\n")
        f.write(f"# (bench.py --profile: 100 warm-up steps, then 50; statistics over the last {last} dispatches of\n")
        f.write("# each kernel, i.e. the 50 steps after the warm-up).\n# commands (repository root, TMPDIR=/tmp):\n")
        f.write("#   rocprofv3 --kernel-trace --stats -d KT_DIR --output-format csv -- python3 bench.py --profile "
                f"--shape {shape}{tu}\n")
        f.write(f"#   python3 bench.py --summarize-kstats KT_DIR {out_name} --shape {shape}{tu}\n")
        f.write("# rows: this library's kernels of the steps (weight packing and input generation omitted)\n")
        f.write(f"kernel_source_sha: {source_sha()}\n")
        f.write("# kernel | dispatches (summarised) | average us | min us | max us\n")
        for n, tot, k, avg, mn, mx in rows:
            f.write(f"{n} | {tot} ({k}) | {avg:.1f} | {mn:.1f} | {mx:.1f}\n")
    print(open(out_path).read())


def summarize_pmc(fetch_dir, write_dir, out_path, shape):
    """FETCH_SIZE / WRITE_SIZE (KiB per dispatch) of each expert kernel of a `bench.py --profile` run,
    each scaled by what the same counter reads for the 1 GiB calibration copy, against the kernel's
    algorithmic bytes."""
    import synth
    sh = synth.SHAPES[shape]
    T, U = 64, 32

    def load(d, counter):
        rows = []
        for p in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            with open(p) as f:
                rows += [r for r in csv.DictReader(f) if r.get("Counter_Name") == counter]
        return rows

    def mean_for(rows, pred):
        v = [float(r["Counter_Value"]) for r in rows if pred(r["Kernel_Name"])]
        return (sum(v) / len(v), len(v)) if v else (float("nan"), 0)

    fr, wr = load(fetch_dir, "FETCH_SIZE"), load(write_dir, "WRITE_SIZE")
    f_cp, _ = mean_for(fr, lambda n: "bitwise_not" in n)
    w_cp, _ = mean_for(wr, lambda n: "bitwise_not" in n)
    cal_f, cal_w = COPY_BYTES / (f_cp * 1024.0), COPY_BYTES / (w_cp * 1024.0)
    with open(out_path, "w") as f:
        name = {"ds": "DeepSeek-V3.1-shaped FP8", "gpt": "GPT-OSS-120B-shaped MXFP4"}[shape]
        f.write(f"# rocprofv3 counter summary: expert kernels, {name} layer, T=64, exact-U routing, U=32\n")
        f.write("# commands (repository root, TMPDIR=/tmp):\n")
        f.write(f"#   rocprofv3 --pmc FETCH_SIZE -d FETCH_DIR --output-format csv -- python3 bench.py --profile --shape {shape}\n")
        f.write(f"#   rocprofv3 --pmc WRITE_SIZE -d WRITE_DIR --output-format csv -- python3 bench.py --profile --shape {shape}\n")
        f.write(f"#   python3 bench.py --summarize-pmc FETCH_DIR WRITE_DIR {os.path.relpath(PMC_SUMMARY[shape], ROOT)} --shape {shape}\n")
        f.write("# counters are KiB per dispatch; each is scaled by COPY_BYTES / (its reading for the calibration\n")
        f.write("# kernel, torch.bitwise_not over 1 GiB of int32, which reads and writes 1 GiB each)\n")
        f.write(f"kernel_source_sha: {source_sha()}\n")
        f.write(f"calibration_fetch: {cal_f:.4f}\ncalibration_write: {cal_w:.4f}\n")
        for down in (False, True):
            tag = f"expert_ffn_kernelILi{sh.fmt}ELb{int(down)}E"
            plain = f"expert_ffn_kernel<{sh.fmt}, {'true' if down else 'false'}"
            pred = lambda n, tag=tag, plain=plain: tag in n or plain in n
            fk, nf = mean_for(fr, pred)
            wk, nw = mean_for(wr, pred)
            hbm = fk * 1024.0 * cal_f + wk * 1024.0 * cal_w
            alg = kernel_alg_bytes(sh, T, U, down)
            k = "down" if down else "gateup"
            f.write(f"{k}_dispatches: fetch {nf}, write {nw}\n")
            f.write(f"{k}_fetch_kib_per_dispatch: {fk:.1f}\n{k}_write_kib_per_dispatch: {wk:.1f}\n")
            f.write(f"{k}_hbm_bytes_per_launch: {hbm:.0f}\n{k}_alg_bytes_per_launch: {alg}\n")
            f.write(f"{k}_hbm_over_alg: {hbm / alg:.4f}\n")
    print(open(out_path).read())


SQ_PASSES = {
    "A": "SQ_WAVE_CYCLES SQ_BUSY_CYCLES SQ_WAIT_ANY SQ_WAIT_INST_ANY SQ_ACTIVE_INST_ANY SQ_ACTIVE_INST_VALU "
         "SQ_VALU_MFMA_BUSY_CYCLES SQ_ACTIVE_INST_LDS",
    "B": "SQ_INSTS_VALU SQ_INSTS_MFMA SQ_INSTS_SALU SQ_INSTS_LDS SQ_INSTS_VMEM_RD SQ_WAIT_INST_LDS SQ_INSTS_VALU_CVT "
         "SQ_ACTIVE_INST_VMEM",
}
SQ_SUMMARY = {"ds": "profiles/expert_ffn_ds_fp8_T64_U32.sq.txt", "gpt": "profiles/expert_ffn_gpt_mxfp4_T64_U32.sq.txt"}


def summarize_sq(dir_a, dir_b, out_path, shape, last=50):
    """Shader-sequencer counters of the two expert kernels of a `bench.py --profile` run (two counter passes),
    per dispatch over the last `last` dispatches, with the derived fractions of wavefront time: issuing any
    instruction, issuing VALU, waiting for an instruction's inputs (SQ_WAIT_INST_ANY), waiting for anything.
    Cycle counters count quad-cycles per wavefront; instruction counts are per wavefront and step (a step is
    one 128-wide block, two for MXFP4, of one item on each of the workgroup's wavefronts)."""
    import synth
    sh = synth.SHAPES[shape]
    T, U, waves_per_wg = 64, 32, 8
    rows = {}
    for d in (dir_a, dir_b):
        for p in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            with open(p) as f:
                for r in csv.DictReader(f):
                    n = r["Kernel_Name"]
                    if "expert_ffn_kernel" not in n:
                        continue
                    down = ", true" in n or "ELb1E" in n
                    per = rows.setdefault((down, r["Counter_Name"]), {})
                    disp = int(r.get("Dispatch_Id", 0) or 0)
                    per[disp] = per.get(disp, 0.0) + float(r["Counter_Value"])
    n_exp = U + (1 if sh.shared else 0)
    with open(out_path, "w") as f:
        name = {"ds": "DeepSeek-V3.1-shaped FP8", "gpt": "GPT-OSS-120B-shaped MXFP4"}[shape]
        f.write(f"# rocprofv3 shader-sequencer counters: expert kernels, {name} layer, T=64, exact-U routing, U=32\n")
        f.write("# commands (repository root, TMPDIR=/tmp):\n")
        for tag, cs in SQ_PASSES.items():
            f.write(f"#   rocprofv3 --pmc {cs} -d SQ_{tag} --output-format csv -- python3 bench.py --profile --shape {shape}\n")
        f.write(f"#   python3 bench.py --summarize-sq SQ_A SQ_B {SQ_SUMMARY[shape]} --shape {shape}\n")
        f.write(f"# per dispatch, mean over the last {last} dispatches of each kernel\n")
        f.write(f"kernel_source_sha: {source_sha()}\n")
        for down in (False, True):
            k = "down" if down else "gateup"
            blocks = -(-(sh.d_ff if down else sh.d) // 128)
            steps = -(-blocks // (2 if sh.fmt == 2 else 1))
            bands = -(-(sh.d if down else sh.d_ff) // (256 if down else 128))
            wave_steps = n_exp * bands * steps * waves_per_wg
            c = {}
            for (dn, name_), per in rows.items():
                if dn == down:
                    ds_ = sorted(per)[-last:]
                    c[name_] = sum(per[i] for i in ds_) / max(1, len(ds_))
            for name_ in sorted(c):
                f.write(f"{k}_{name_}: {c[name_]:.0f}\n")
            wc = c.get("SQ_WAVE_CYCLES")
            if wc:
                for cn in ("SQ_ACTIVE_INST_ANY", "SQ_ACTIVE_INST_VALU", "SQ_WAIT_INST_ANY", "SQ_WAIT_ANY",
                           "SQ_ACTIVE_INST_LDS", "SQ_ACTIVE_INST_VMEM"):
                    if cn in c:
                        f.write(f"{k}_frac_of_wave_time_{cn[3:].lower()}: {c[cn] / wc:.3f}\n")
            f.write(f"{k}_wave_steps: {wave_steps}\n")
            for cn in ("SQ_INSTS_VALU", "SQ_INSTS_VALU_CVT", "SQ_INSTS_MFMA", "SQ_INSTS_SALU", "SQ_INSTS_LDS",
                       "SQ_INSTS_VMEM_RD"):
                if cn in c:
                    f.write(f"{k}_{cn[9:].lower() or 'valu'}_per_wave_step: {c[cn] / wave_steps:.1f}\n")
    print(open(out_path).read())


def pmc_traffic(shape, kernel="gateup"):
    kv = read_summary(PMC_SUMMARY[shape])
    if not kv:
        return None
    try:
        return float(kv[f"{kernel}_hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


# --------------------------------------------------------------------------- main

def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    # The GPU runs the first ~50 steps after an idle spell ~5% slower (its clocks ramp up; after 2 s idle the
    # first 50 steps are again slow), so 100 untimed steps precede every timed region of the headline.
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--T", type=int, default=64)
    ap.add_argument("--U", type=int, default=32)
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--cpu-tokens", type=int, default=48)
    ap.add_argument("--no-stack", action="store_true", help="skip the 8-layer draft-tree verification step")
    ap.add_argument("--stack-only", action="store_true", help="only the 8-layer draft-tree verification step")
    ap.add_argument("--trees", type=int, default=12, help="seeded draft trees of the 8-layer step")
    ap.add_argument("--profile", action="store_true", help="short run for rocprofv3 plus a calibration copy")
    ap.add_argument("--shape", default="ds", choices=["ds", "gpt"], help="layer of --profile / --summarize-pmc")
    ap.add_argument("--summarize-kstats", nargs=2, metavar=("KT_DIR", "OUT"))
    ap.add_argument("--summarize-pmc", nargs=3, metavar=("FETCH_DIR", "WRITE_DIR", "OUT"))
    ap.add_argument("--summarize-sq", nargs=3, metavar=("SQ_A", "SQ_B", "OUT"))
    args = ap.parse_args()

    if args.summarize_kstats:
        summarize_kstats(*args.summarize_kstats, args.shape, T=args.T, U=args.U)
        return 0
    if args.summarize_pmc:
        summarize_pmc(*args.summarize_pmc, args.shape)
        return 0
    if args.summarize_sq:
        summarize_sq(*args.summarize_sq, args.shape)
        return 0
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path (run with --gpus 1)", file=sys.stderr)
        return 2

    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    import paper_2607_12696_amd as moe
    moe.lib()  # fail loudly if the HIP library is missing

    if args.stack_only:
        st = Stack()
        print(json.dumps(st.measure(args.trees, max(10, args.steps // 2), 3)))
        return 0

    if args.profile:
        # The headline's own steps (or the GPT-OSS layer's at T=64, U=32): W warm-ups, then K steps.
        layer = Layer(args.shape, n_shared_copies=4)
        rn = Runner(layer, args.T)
        pool = rn.pool("exact", 16, U=args.U, seed=100 * args.U)
        for i in range(args.warmup + args.steps):
            rn.step(pool[i % len(pool)], i)
        # Calibration copy for the HBM counters: one elementwise kernel that reads and writes COPY_BYTES
        # each, with a name nothing else in the run uses.
        src = torch.ones(COPY_BYTES // 4, dtype=torch.int32, device=layer.dev)
        dst = torch.empty_like(src)
        torch.bitwise_not(src, out=dst)
        torch.cuda.synchronize()
        log("profile run done")
        return 0

    ds = Layer("ds", n_shared_copies=4)
    sh = ds.sh
    rn = Runner(ds, args.T)
    pool = rn.pool("exact", 16, U=args.U, seed=100 * args.U)
    # Headline: K plain steps between two events, then the same steps with per-kernel marks.
    ms = rn.time_plain(pool, args.steps, args.warmup)
    per = rn.time_marks(pool, args.steps, args.warmup)
    B = step_alg_bytes(sh, args.T, args.U)
    gu_ms = sum(per["gateup"]) / len(per["gateup"])
    gu_bytes = kernel_alg_bytes(sh, args.T, args.U, False)
    gu_gbs = gu_bytes / (gu_ms * 1e-3) / 1e9
    gu_rp = rocprof_gateup_us()
    log(f"U={args.U}: step {ms * 1e3:.1f} us, {B / (ms * 1e-3) / 1e9:.0f} GB/s; gate/up {gu_ms * 1e3:.1f} us "
        f"({gu_gbs:.0f} GB/s), down {1e3 * sum(per['down']) / len(per['down']):.1f} us")
    headline = point(rn, pool, args.steps, args.warmup, U=args.U)
    # The same steps after two seconds of idle GPU, without warm-up (the ramp the warm-up excludes).
    time.sleep(2.0)
    cold_ms = rn.time_plain(pool, args.steps, 0)

    cpu, err = (None, None)
    if not args.no_cpu:
        log("timing the oracle on the host ...")
        cpu, err = cpu_baseline(ds, rn, pool[0], args.U, args.cpu_tokens)
    del rn

    sweeps = {}
    if not args.no_sweep:
        # The oracle timing left the GPU idle for seconds: bring its clocks back up first.
        rn = Runner(ds, args.T)
        rn.time_plain(pool, args.warmup, 0)
        del rn
        k = sh.k
        Us_all = [8, 16, 24, 32, 48, 64, 96, 128, 192, 256]
        sweeps["ds_u_sweeps"] = u_sweeps(ds, [(T, [u for u in Us_all if k <= u <= T * k]) for T in (64, 32, 16, 8)],
                                         steps=20, warmup=SWEEP_WARMUP)
        sweeps["ds_routing"] = routing_grid(ds, (4, 8, 16, 32, 64, 128, 256), ("clustered", "scattered"), steps=20,
                                            warmup=SWEEP_WARMUP)
        sweeps["ds_router"] = router_timing(ds)
        sweeps["ds_tokens_per_expert_U32"] = token_sweep(ds)
    del ds
    torch.cuda.empty_cache()
    if not args.no_sweep:
        qw = Layer("qwen")
        sweeps["qwen_routing"] = routing_grid(qw, (1, 4, 8, 16, 32, 64), ("clustered", "scattered"), steps=20,
                                              warmup=SWEEP_WARMUP)
        sweeps["qwen_u_sweep_T64"] = u_sweeps(qw, [(64, [8, 32, 64, 128])], steps=20, warmup=SWEEP_WARMUP)
        sweeps["qwen_tokens_per_expert_U32"] = token_sweep(qw)
        del qw
        torch.cuda.empty_cache()
        gp = Layer("gpt")
        sweeps["gpt_routing"] = routing_grid(gp, (4, 8, 32, 64), ("clustered", "scattered"), steps=20, warmup=SWEEP_WARMUP)
        sweeps["gpt_routing_mx_act"] = routing_grid(gp, (4, 8, 32, 64), ("clustered", "scattered"), steps=20,
                                                    warmup=SWEEP_WARMUP, act_fmt=1)
        sweeps["gpt_u_sweep_T64"] = u_sweeps(gp, [(64, [8, 32, 64, 128])], steps=20, warmup=SWEEP_WARMUP)
        sweeps["gpt_tokens_per_expert_U32"] = token_sweep(gp)
        sweeps["gpt_tokens_per_expert_U32_mx_act"] = token_sweep(gp, act_fmt=1)
        sweeps["gpt_variants_T64"] = gpt_variants(gp)
        del gp
        torch.cuda.empty_cache()

    stack = None
    if not args.no_stack:
        st = Stack()
        stack = st.measure(args.trees, max(10, args.steps // 5), 10)
        del st
        torch.cuda.empty_cache()

    traffic = pmc_traffic("ds")
    out = {
        "metric": METRIC, "value": B / (ms * 1e-3) / 1e9, "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"DeepSeek-V3.1-shaped MoE verify layer, FP8 e4m3 128x128-scaled weights, "
                               f"T={args.T} draft tokens routed to U={args.U} of 256 experts + 1 shared",
                   "d": sh.d, "d_ff": sh.d_ff, "E": sh.E, "k": sh.k, "T": args.T, "U": args.U,
                   "routing": "exact-U, sigmoid top-8, a different expert set every step",
                   "alg_bytes_per_step": B},
        "roofline": {"bound": "hbm", "achieved": gu_gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": gu_gbs / PEAK_HBM_GBS, "traffic": traffic,
                     "kernel": "expert_ffn_kernel<1, false, 3, false> (FP8 gate/up + SwiGLU)",
                     "alg_bytes_per_launch": gu_bytes, "avg_launch_us": gu_ms * 1e3,
                     "frac_source": "avg_launch_us: HIP events on the launch stream around the kernel in this run",
                     "rocprof_avg_launch_us": gu_rp,
                     "frac_from_rocprof": None if gu_rp is None else gu_bytes / (gu_rp * 1e-6) / 1e9 / PEAK_HBM_GBS,
                     "traffic_over_alg": None if traffic is None else traffic / gu_bytes},
        "cpu_baseline": cpu,
        "parity_sampled_rows_max_rel_err": err,
        "headline_point": headline,
        "kernels_us": {k: 1e3 * sum(v) / len(v) for k, v in per.items()},
        "ms_per_step_first_steps_after_2s_idle": cold_ms,
        "paper_context": PAPER_CONTEXT,
        "stack_8_layers_T16": stack,
    }
    out.update(sweeps)
    print(json.dumps(out))
    return 0


if __name__ == "__main__":
    sys.exit(main())
