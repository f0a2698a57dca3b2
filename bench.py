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

    python bench.py [--gpus 1] [--steps 50] [--warmup 5] [--no-sweep] [--no-cpu]
    python bench.py --profile            # short run for rocprofv3 (plus a copy kernel for counter calibration)
    python bench.py --summarize-pmc DIR  # turn rocprofv3 --pmc output into the summary read below
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MoE verify-layer µs and HBM GB/s vs unique experts (V3.1 shape, FP8)"
PEAK_HBM_GBS = 8000.0
PMC_SUMMARY = os.path.join(ROOT, "profiles", "expert_ffn_gateup_ds_fp8_T64_U32.pmc.txt")
FFN_SOURCE = os.path.join(ROOT, "paper_2607_12696_amd", "csrc", "expert_ffn.hip")
GATEUP_KERNEL = "expert_ffn_kernel<1, false"   # demangled-name prefix of the FP8 gate/up kernel
COPY_BYTES = 1 << 30                            # calibration copy: reads and writes 1 GiB


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def source_sha() -> str:
    return hashlib.sha256(open(FFN_SOURCE, "rb").read()).hexdigest()[:16]


# --------------------------------------------------------------------------- byte accounting

def expert_bytes(d, d_ff):
    """FP8 expert: gate+up+down codes and their fp32 128x128 block scales."""
    return 3 * d * d_ff + 3 * (d // 128) * (d_ff // 128) * 4


def step_alg_bytes(sh, T, U):
    """Algorithmic HBM bytes of one step: every activated expert once, plus the
    activations, logits and routing arrays once each."""
    n_exp = U + (1 if sh.shared else 0)
    routing = 4 * (2 * T * sh.k + T * sh.k + 2 * sh.E + 1 + (sh.E + 1))
    return n_exp * expert_bytes(sh.d, sh.d_ff) + 2 * T * sh.d * 2 + 4 * T * sh.E + routing


def gateup_alg_bytes(sh, T, U):
    """Algorithmic bytes of one gate/up launch: W_gate and W_up (+scales) of every
    activated expert, x read once, the bf16 SwiGLU rows written once."""
    n_exp = U + (1 if sh.shared else 0)
    rows = T * sh.k + (T if sh.shared else 0)
    return n_exp * (2 * sh.d * sh.d_ff + 2 * (sh.d // 128) * (sh.d_ff // 128) * 4) + 2 * T * sh.d + 2 * rows * sh.d_ff


def read_pmc_summary():
    """HBM traffic of the gate/up launch from the committed counter summary, or
    None if it is missing or was taken on a different kernel source."""
    if not os.path.exists(PMC_SUMMARY):
        return None
    kv = {}
    for line in open(PMC_SUMMARY):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("kernel_source_sha") != source_sha():
        return None
    try:
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


# --------------------------------------------------------------------------- workload

class Workload:
    def __init__(self, T, Us, n_pool, n_shared_copies, seed=0):
        import torch
        import synth
        import paper_2607_12696_amd as moe
        self.torch, self.moe, self.synth = torch, moe, synth
        self.dev = torch.device("cuda:0")
        self.sh = synth.SHAPES["ds"]
        sh = self.sh
        self.T = T
        t0 = time.time()
        self.layer = synth.layer_weights(sh, seed=seed, device=self.dev)
        self.shared = [{k: self.layer[k] for k in self.layer if k.startswith("sh_")}]
        for c in range(1, n_shared_copies):
            cp = {}
            for name, (N, K) in (("gate", (sh.d_ff, sh.d)), ("up", (sh.d_ff, sh.d)), ("down", (sh.d, sh.d_ff))):
                cp["sh_" + name], cp["sh_s_" + name] = synth.weights_fp8_b128(1, N, K, seed, f"bench/shared{c}/{name}",
                                                                              self.dev)
            self.shared.append(cp)
        torch.cuda.synchronize()
        log(f"weights generated in {time.time() - t0:.1f}s "
            f"({(sh.E + n_shared_copies) * expert_bytes(sh.d, sh.d_ff) / 1e9:.1f} GB)")
        self.x = synth.activations(T, sh.d, seed=seed, device=self.dev)
        self.pool = {}
        for U in Us:
            self.pool[U] = [synth.routes_to_logits(synth.routes_exact_u(T, sh.E, sh.k, U, seed=1000 * U + i), sh.E,
                                                   seed=i, device=self.dev) for i in range(n_pool)]
        # Preallocated outputs: nothing is allocated inside the timed region.
        i32 = dict(dtype=torch.int32, device=self.dev)
        self.idx = torch.empty(T, sh.k, **i32)
        self.w = torch.empty(T, sh.k, dtype=torch.float32, device=self.dev)
        self.routing = moe.Routing(T, sh.k, sh.E, self.idx, self.w, torch.empty(sh.E, **i32),
                                   torch.empty(sh.E, **i32), torch.empty(1, **i32), torch.empty(sh.E + 1, **i32),
                                   torch.empty(T * sh.k, **i32))
        self.y = torch.empty_like(self.x)
        # Interchange-layout dicts (for the oracle) and their packed device copies (for the kernels).
        self.rawdicts, self.wdicts = [], []
        routed_packed = moe.pack_layer({k: v for k, v in self.layer.items() if not k.startswith("sh_")})
        for cp in self.shared:
            raw = {k: v for k, v in self.layer.items() if not k.startswith("sh_")}
            raw.update(cp)
            self.rawdicts.append(raw)
            wd = dict(routed_packed)
            wd["sh_gate"], wd["sh_s_gate"], wd["sh_s_up"] = moe.moe_pack_gate_up(
                sh.fmt, cp["sh_gate"], cp["sh_up"], cp["sh_s_gate"], cp["sh_s_up"])
            pack_down = moe.moe_pack_down if wd.get("down_paired") else moe.moe_pack_weights
            wd["sh_down"], wd["sh_s_down"] = pack_down(sh.fmt, cp["sh_down"], cp["sh_s_down"])
            self.wdicts.append(wd)
        torch.cuda.synchronize()
        nbytes = moe.moe_verify_workspace_size(self.wdicts[0], T, sh.k)
        self.ws = torch.empty(nbytes, dtype=torch.uint8, device=self.dev)

    def step(self, U, i, events=None):
        """One pass of the hot path; events = optional 6 marks: before route, then the 5
        marks of the timed verify entry point (before and after the gate/up expert kernel,
        before and after the down expert kernel, after combine)."""
        moe, sh = self.moe, self.sh
        lg = self.pool[U][i % len(self.pool[U])]
        wd = self.wdicts[i % len(self.wdicts)]
        if events is not None:
            events[0].record()
        moe.moe_route_union(lg, sh.k, sh.score, out=self.routing)
        if events is None:
            moe.moe_verify_layer(self.x, wd, self.routing, y=self.y, workspace=self.ws)
        else:
            moe.moe_verify_layer_timed(self.x, wd, self.routing, self.y, self.ws, events[1:])

    def time_steps(self, U, steps, warmup, marks):
        torch = self.torch
        for i in range(warmup):
            self.step(U, i)
        torch.cuda.synchronize()
        if not marks:
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for i in range(steps):
                self.step(U, warmup + i)
            b.record()
            torch.cuda.synchronize()
            return a.elapsed_time(b) / steps, None
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(steps)]
        for row in evs:  # torch creates the HIP event on first record; the library records raw handles
            for e in row:
                e.record()
        torch.cuda.synchronize()
        for i in range(steps):
            self.step(U, warmup + i, evs[i])
        torch.cuda.synchronize()
        spans = {"step": (0, 5), "route_union": (0, 1), "verify": (1, 5), "gateup": (1, 2), "gateup_fixup": (2, 3),
                 "down": (3, 4), "combine": (4, 5)}
        per = {k: [e[a].elapsed_time(e[b]) for e in evs] for k, (a, b) in spans.items()}
        return None, per


class TSweep:
    """Steps at T tokens with i.i.d. router logits, on a Workload's resident weights."""

    def __init__(self, wl, T, n_pool=8):
        import torch
        import synth
        moe, sh = wl.moe, wl.sh
        self.wl, self.T, self.torch = wl, T, torch
        self.logits = [synth.logits_scattered(T, sh.E, seed=7000 + 31 * T + i).to(wl.dev) for i in range(n_pool)]
        i32 = dict(dtype=torch.int32, device=wl.dev)
        self.r = moe.Routing(T, sh.k, sh.E, torch.empty(T, sh.k, **i32),
                             torch.empty(T, sh.k, dtype=torch.float32, device=wl.dev), torch.empty(sh.E, **i32),
                             torch.empty(sh.E, **i32), torch.empty(1, **i32), torch.empty(sh.E + 1, **i32),
                             torch.empty(T * sh.k, **i32))
        self.x = synth.activations(T, sh.d, seed=9, device=wl.dev)
        self.y = torch.empty_like(self.x)
        self.ws = torch.empty(moe.moe_verify_workspace_size(wl.wdicts[0], T, sh.k), dtype=torch.uint8,
                              device=wl.dev)

    def step(self, i):
        wl, sh = self.wl, self.wl.sh
        wl.moe.moe_route_union(self.logits[i % len(self.logits)], sh.k, sh.score, out=self.r)
        wl.moe.moe_verify_layer(self.x, wl.wdicts[i % len(wl.wdicts)], self.r, y=self.y, workspace=self.ws)

    def time(self, steps, warmup):
        torch = self.torch
        uniq = []
        for i in range(warmup):
            self.step(i)
        for i in range(len(self.logits)):
            self.step(i)
            uniq.append(int(self.r.n_unique.item()))
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for i in range(steps):
            self.step(i)
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e3 / steps, float(np.median(uniq))

    def alg_bytes(self, U):
        sh = self.wl.sh
        return step_alg_bytes(sh, self.T, U)


def router_timing(wl, reps=20, replays=10):
    """Router from hidden states (x . W_r^T in split-K on the matrix cores, then the top-k that
    sums the K slices) against top-k from given logits, at the workload's T.  Each is captured
    `reps` times into one HIP graph and replayed, so host launch cost does not enter."""
    import torch
    import synth
    moe, sh = wl.moe, wl.sh
    T = wl.T
    w_r = synth.router_weight(sh.E, sh.d, seed=3, device=wl.dev)
    ws = torch.empty(moe.moe_router_workspace_size(T, sh.d, sh.E), dtype=torch.uint8, device=wl.dev)
    idx = torch.empty(T, sh.k, dtype=torch.int32, device=wl.dev)
    tw = torch.empty(T, sh.k, dtype=torch.float32, device=wl.dev)
    lg = torch.empty(T, sh.E, dtype=torch.float32, device=wl.dev)
    idx2, tw2 = torch.empty_like(idx), torch.empty_like(tw)
    moe.moe_route_topk_hidden(wl.x, w_r, sh.k, sh.score, logits=lg, workspace=ws, topk_idx=idx, topk_w=tw)
    moe.moe_route_topk(lg, sh.k, sh.score, topk_idx=idx2, topk_w=tw2)
    torch.cuda.synchronize()
    consistent = bool(torch.equal(idx, idx2) and torch.equal(tw, tw2))

    def graph_us(fn):
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

    hid = graph_us(lambda: moe.moe_route_topk_hidden(wl.x, w_r, sh.k, sh.score, workspace=ws, topk_idx=idx,
                                                     topk_w=tw))
    lgt = graph_us(lambda: moe.moe_route_topk(lg, sh.k, sh.score, topk_idx=idx2, topk_w=tw2))
    return {"T": T, "d": sh.d, "E": sh.E, "router_from_hidden_us": hid, "route_from_logits_us": lgt,
            "router_gemm_bytes": 2 * sh.E * sh.d + 2 * T * sh.d, "routing_matches_logits_entry": consistent}


def variant_timing(T=64, steps=30, warmup=3, n_pool=8):
    """The real-model variants: a GPT-OSS-120B-shaped MXFP4 layer (d 2880, d_ff 2880, 128 experts,
    top-4 softmax) with clustered routing (children keep a parent expert with p = 0.8), plain
    SwiGLU against the GPT-OSS expert (biases, clamped SwiGLU); and DeepSeek-V3's group-limited
    routing (8 groups of 32, 4 kept, correction bias, scale 2.5) against plain sigmoid top-8 on
    the same logits, each captured 20 times in a HIP graph and replayed."""
    import torch
    import synth
    import paper_2607_12696_amd as moe
    dev = torch.device("cuda:0")
    sh = synth.SHAPES["gpt"]
    raw = synth.layer_weights(sh, seed=0, device=dev)
    plain = moe.pack_layer(raw)
    del raw
    oai = dict(plain, act=moe.MOE_ACT_SWIGLU_OAI, alpha=1.702, limit=7.0,
               b_gate=synth.expert_biases(sh.E, sh.d_ff, 0, "bg", dev), b_up=synth.expert_biases(sh.E, sh.d_ff, 0, "bu", dev),
               b_down=synth.expert_biases(sh.E, sh.d, 0, "bd", dev))
    x = synth.activations(T, sh.d, seed=1, device=dev)
    pool = [synth.routes_to_logits(synth.routes_clustered(T, sh.E, sh.k, 0.8, seed=50 + i), sh.E, seed=i,
                                   device=dev) for i in range(n_pool)]
    # The MX-activation layout needs the most workspace of the three variants.
    ws = torch.empty(moe.moe_verify_workspace_size(dict(plain, act_fmt=moe.MOE_ACTQ_MXFP8), T, sh.k),
                     dtype=torch.uint8, device=dev)
    y = torch.empty_like(x)
    uniq = []
    for lg in pool:
        _, r = moe.moe_verify_step(x, lg, plain, sh.k, sh.score, workspace=ws, y=y)
        uniq.append(int(r.n_unique.item()))
    U = float(np.median(uniq))

    def steps_us(wd):
        for i in range(warmup):
            moe.moe_verify_step(x, pool[i % n_pool], wd, sh.k, sh.score, workspace=ws, y=y)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for i in range(steps):
            moe.moe_verify_step(x, pool[i % n_pool], wd, sh.k, sh.score, workspace=ws, y=y)
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e3 / steps

    t_plain, t_oai, t_mx = steps_us(plain), steps_us(oai), steps_us(dict(plain, act_fmt=moe.MOE_ACTQ_MXFP8))
    per_expert = sum(synth.expert_bytes(sh.d, sh.d_ff, sh.fmt))  # weights + e8m0 scales, unpadded
    B = U * per_expert + 4 * T * sh.d + 4 * T * sh.E
    out = {"gpt_oss_T64_clustered": {"unique_experts_median": U, "plain_swiglu_us": t_plain,
                                     "gpt_oss_expert_us": t_oai, "GB_s_gpt_oss_expert": B / (t_oai * 1e-6) / 1e9,
                                     "mx_fp8_activations_us": t_mx, "alg_bytes": B}}
    del plain, oai, ws
    torch.cuda.empty_cache()

    E, k = 256, 8
    lg = synth.logits_scattered(T, E, seed=3, device=dev)
    bias = synth.router_bias(E, seed=3, device=dev)
    idx = torch.empty(T, k, dtype=torch.int32, device=dev)
    tw = torch.empty(T, k, dtype=torch.float32, device=dev)

    def graph_us(fn, reps=20, replays=10):
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

    out["ds_routing_T64"] = {
        "grouped_us": graph_us(lambda: moe.moe_route_topk_grouped(lg, bias, k, 8, 4, 2.5, topk_idx=idx, topk_w=tw)),
        "plain_sigmoid_us": graph_us(lambda: moe.moe_route_topk(lg, k, moe.MOE_SCORE_SIGMOID, topk_idx=idx,
                                                                topk_w=tw))}
    return out


def shape_sweep(name, Us, T=64, steps=20, warmup=3, n_pool=8, act_fmt=0):
    """Step latency and algorithmic GB/s vs U for another model shape (exact-U routing, a different
    expert set every step, so weights are read cold: the sets rotate over all experts of the layer).
    act_fmt 1: MX FP8 activations on the scaled FP4 x FP8 matrix-core instruction (MXFP4 only)."""
    import torch
    import synth
    import paper_2607_12696_amd as moe
    dev = torch.device("cuda:0")
    sh = synth.SHAPES[name]
    raw = synth.layer_weights(sh, seed=0, device=dev)
    wd = dict(moe.pack_layer(raw), act_fmt=act_fmt)
    del raw
    x = synth.activations(T, sh.d, seed=1, device=dev)
    y = torch.empty_like(x)
    ws = torch.empty(moe.moe_verify_workspace_size(wd, T, sh.k), dtype=torch.uint8, device=dev)
    per_expert = sum(synth.expert_bytes(sh.d, sh.d_ff, sh.fmt))
    out = []
    for U in Us:
        pool = [synth.routes_to_logits(synth.routes_exact_u(T, sh.E, sh.k, U, seed=500 * U + i), sh.E, seed=i,
                                       device=dev) for i in range(n_pool)]
        for i in range(warmup):
            moe.moe_verify_step(x, pool[i % n_pool], wd, sh.k, sh.score, workspace=ws, y=y)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for i in range(steps):
            moe.moe_verify_step(x, pool[i % n_pool], wd, sh.k, sh.score, workspace=ws, y=y)
        b.record()
        torch.cuda.synchronize()
        us = a.elapsed_time(b) * 1e3 / steps
        B = (U + (1 if sh.shared else 0)) * per_expert + 4 * T * sh.d + 4 * T * sh.E
        out.append({"U": U, "step_us": us, "GB_s": B / (us * 1e-6) / 1e9, "frac_of_8TBs": B / (us * 1e-6) / 8e12})
        log(f"  {name}{' MX act' if act_fmt else ''} U={U:4d}: step {us:8.1f} us  {out[-1]['GB_s']:7.0f} GB/s")
    del wd, ws
    torch.cuda.empty_cache()
    return {"shape": name, "d": sh.d, "d_ff": sh.d_ff, "E": sh.E, "k": sh.k, "fmt": sh.fmt, "act_fmt": act_fmt,
            "T": T, "points": out}


def token_sweep(name, Ms=(1, 4, 16, 32, 64), U=32, steps=20, warmup=3, n_pool=8, act_fmt=0):
    """Tokens per expert: exact-U routing with T = M * U / k gives every one of the U experts exactly
    M tokens (and the shared expert T).  Per-kernel medians (HIP events around each expert launch)
    show where the matrix-core work of a step starts to cost on top of the weight stream: the
    contraction grows with the 16-token blocks of an item, the weight bytes do not."""
    import torch
    import synth
    import paper_2607_12696_amd as moe
    dev = torch.device("cuda:0")
    sh = synth.SHAPES[name]
    raw = synth.layer_weights(sh, seed=0, device=dev)
    wd = dict(moe.pack_layer(raw), act_fmt=act_fmt)
    del raw
    w_b, s_b = synth.expert_bytes(sh.d, sh.d_ff, sh.fmt)
    n_exp = U + (1 if sh.shared else 0)
    spans = {"step": (0, 5), "gateup": (1, 2), "fixup": (2, 3), "down": (3, 4), "combine": (4, 5)}
    out = []
    for M in Ms:
        T = M * U // sh.k
        if T < 1 or T * sh.k != M * U:
            continue
        x = synth.activations(T, sh.d, seed=1, device=dev)
        y = torch.empty_like(x)
        ws = torch.empty(moe.moe_verify_workspace_size(wd, T, sh.k), dtype=torch.uint8, device=dev)
        pool = [synth.routes_to_logits(synth.routes_exact_u(T, sh.E, sh.k, U, seed=700 * M + i), sh.E, seed=i,
                                       device=dev) for i in range(n_pool)]
        i32 = dict(dtype=torch.int32, device=dev)
        r = moe.Routing(T, sh.k, sh.E, torch.empty(T, sh.k, **i32), torch.empty(T, sh.k, dtype=torch.float32,
                                                                                    device=dev),
                        torch.empty(sh.E, **i32), torch.empty(sh.E, **i32), torch.empty(1, **i32),
                        torch.empty(sh.E + 1, **i32), torch.empty(T * sh.k, **i32))
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(steps)]
        for row in evs:
            for e in row:
                e.record()
        for i in range(warmup):
            moe.moe_route_union(pool[i % n_pool], sh.k, sh.score, out=r)
            moe.moe_verify_layer(x, wd, r, y=y, workspace=ws)
        torch.cuda.synchronize()
        for i in range(steps):
            evs[i][0].record()
            moe.moe_route_union(pool[i % n_pool], sh.k, sh.score, out=r)
            moe.moe_verify_layer_timed(x, wd, r, y, ws, evs[i][1:])
        torch.cuda.synchronize()
        med = {k: 1e3 * pct([e[a].elapsed_time(e[b]) for e in evs], 0.5) for k, (a, b) in spans.items()}
        gu_bytes = n_exp * (2 * w_b + 2 * s_b) / 3
        dn_bytes = n_exp * (w_b + s_b) / 3
        pt = {"M": M, "T": T, "step_us": med["step"], "gateup_us": med["gateup"], "fixup_us": med["fixup"],
              "down_us": med["down"], "combine_us": med["combine"],
              "gateup_GB_s": gu_bytes / (med["gateup"] * 1e-6) / 1e9,
              "down_GB_s": dn_bytes / (med["down"] * 1e-6) / 1e9,
              "step_GB_s": n_exp * (w_b + s_b) / (med["step"] * 1e-6) / 1e9}
        out.append(pt)
        log(f"  {name}{' MX act' if act_fmt else ''} M={M:3d} (T={T:4d}): step {pt['step_us']:7.1f} us, gate/up {pt['gateup_us']:6.1f} us "
            f"({pt['gateup_GB_s']:5.0f} GB/s), down {pt['down_us']:6.1f} us ({pt['down_GB_s']:5.0f} GB/s)")
        del x, y, ws, pool, r
    del wd
    torch.cuda.empty_cache()
    return {"shape": name, "fmt": sh.fmt, "act_fmt": act_fmt, "U": U, "points": out}


def pct(v, q):
    s = sorted(v)
    return s[min(len(s) - 1, max(0, int(round(q * (len(s) - 1)))))]


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


# --------------------------------------------------------------------------- CPU baseline (oracle)

def cpu_baseline(wl, U, n_tokens):
    """The oracle on the host cores for n_tokens of the headline step; returns the
    baseline dict and the sampled rows' max error of the GPU output against it."""
    import numpy as np
    import oracle
    torch, sh = wl.torch, wl.sh
    lg = wl.pool[U][0]
    wl.step(U, 0)
    torch.cuda.synchronize()
    y_gpu = wl.y.float().cpu().numpy()
    lg_h = lg.cpu().numpy()
    idx_o, w_o = oracle.route(lg_h, sh.k, sh.score)
    rows = list(range(n_tokens))
    used = sorted(set(idx_o[rows].reshape(-1).tolist()))
    wd = wl.rawdicts[0]
    hl = {"fmt": sh.fmt, "d": sh.d, "d_ff": sh.d_ff}
    for n in ("gate", "up", "down", "s_gate", "s_up", "s_down"):
        hl[n] = {e: wd[n][e].cpu() for e in used}
    for n in ("sh_gate", "sh_up", "sh_down", "sh_s_gate", "sh_s_up", "sh_s_down"):
        hl[n] = wd[n].cpu()
    x_h = wl.x.cpu()
    threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or min(16, os.cpu_count() or 1)
    t0 = time.time()
    y_ref = oracle.verify_tokens(hl, x_h, idx_o, w_o, tokens=rows, threads=threads)
    dt = time.time() - t0
    full = dt * wl.T / n_tokens   # the oracle's cost is proportional to the token count
    err = float(np.abs(y_gpu[rows] - y_ref).max() / np.abs(y_ref).max())
    cpu_model = ""
    try:
        with open("/proc/cpuinfo") as f:
            cpu_model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), "")
    except OSError:
        pass
    base = {"value": step_alg_bytes(sh, wl.T, U) / full / 1e9, "unit": "GB/s", "cores": threads, "kind": "oracle",
            "nproc": os.cpu_count(), "cpu_model": cpu_model, "omp_num_threads": os.environ.get("OMP_NUM_THREADS"),
            "sample": f"fp64 C oracle on {n_tokens} of the {wl.T} tokens of the same step (U={U}), "
                      f"{n_tokens * (sh.k + 1)} expert FFNs in {dt:.2f}s; scaled x{wl.T / n_tokens:g} to the "
                      f"whole step ({full:.1f}s)"}
    return base, err


# --------------------------------------------------------------------------- 8-layer verification step

class Stack:
    """Eight DeepSeek-V3.1-shaped FP8 MoE layers verifying T=16 tokens of a synthetic
    64-node draft tree (branching 4, per-node scores ~ Beta(2,2), children inherit a
    parent expert per slot with probability 0.7), the tokens chosen once by
    confidence (highest path score first) and once by the cost-aware selector
    (Algorithm 1).  Each layer's routing comes from synthetic router logits whose
    top-8 are the nodes' expert sets, and each layer gets its own synthetic N(0,1)
    hidden states (there is no model around the MoE layers to carry them: no norm
    or residual, without which stacked random layers overflow bf16)."""

    L, N_NODES, BRANCH, BUDGET, P_INHERIT = 8, 64, 4, 16, 0.7

    def __init__(self, seed=0):
        import torch
        import synth
        import paper_2607_12696_amd as moe
        self.torch, self.moe = torch, moe
        self.dev = torch.device("cuda:0")
        sh = self.sh = synth.SHAPES["ds"]
        t0 = time.time()
        self.layers = []
        for l in range(self.L):
            raw = synth.layer_weights(sh, seed=seed + 17, device=self.dev, layer=l)
            self.layers.append(moe.pack_layer(raw))
            del raw
        torch.cuda.synchronize()
        log(f"stack: {self.L} layers packed in {time.time() - t0:.1f}s")
        self.parent, self.P = synth.draft_tree(self.N_NODES, self.BRANCH, seed=seed)
        self.pred = synth.tree_expert_sets(self.parent, self.L, sh.E, sh.k, self.P_INHERIT, seed=seed)
        self.sel = {
            "confidence": moe.moe_select_tree(self.parent, self.P, self.pred, sh.E, self.BUDGET,
                                              mode=moe.MOE_SEL_CONFIDENCE)[0],
            "cost_aware": moe.moe_select_tree(self.parent, self.P, self.pred, sh.E, self.BUDGET,
                                              mode=moe.MOE_SEL_COST_RATIO)[0],
            "global_cost": moe.moe_select_tree(self.parent, self.P, self.pred, sh.E, self.BUDGET,
                                               mode=moe.MOE_SEL_GLOBAL_COST)[0],
        }
        T = self.BUDGET
        i32 = dict(dtype=torch.int32, device=self.dev)
        self.xs = [synth.activations(T, sh.d, seed=seed + 5 + l, device=self.dev) for l in range(self.L)]
        self.ys = [torch.empty_like(x) for x in self.xs]
        self.ws = torch.empty(moe.moe_verify_workspace_size(self.layers[0], T, sh.k), dtype=torch.uint8,
                              device=self.dev)
        self.plans = {}
        for name, nodes in self.sel.items():
            logits, routs = [], []
            for l in range(self.L):
                routes = self.pred[nodes, l, :]
                logits.append(synth.routes_to_logits(routes, sh.E, seed=seed + 100 * l + 1, device=self.dev))
                routs.append(moe.Routing(T, sh.k, sh.E, torch.empty(T, sh.k, **i32),
                                         torch.empty(T, sh.k, dtype=torch.float32, device=self.dev),
                                         torch.empty(sh.E, **i32), torch.empty(sh.E, **i32), torch.empty(1, **i32),
                                         torch.empty(sh.E + 1, **i32), torch.empty(T * sh.k, **i32)))
            self.plans[name] = (logits, routs)

    def run(self, name):
        """The 8-layer pass for one selection; returns the stacked layer outputs [L, T, d]."""
        moe, sh = self.moe, self.sh
        logits, routs = self.plans[name]
        for l in range(self.L):
            moe.moe_route_union(logits[l], sh.k, sh.score, out=routs[l])
            moe.moe_verify_layer(self.xs[l], self.layers[l], routs[l], y=self.ys[l], workspace=self.ws)
        return self.ys

    def measure(self, steps, warmup):
        torch = self.torch
        out = {"layers": self.L, "T": self.BUDGET, "tree_nodes": self.N_NODES, "branching": self.BRANCH,
               "p_inherit": self.P_INHERIT}
        for name in self.sel:
            for _ in range(warmup):
                self.run(name)
            torch.cuda.synchronize()
            ref = torch.stack(self.run(name))
            uniq = [int(r.n_unique.item()) for r in self.plans[name][1]]
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for _ in range(steps):
                self.run(name)
            b.record()
            torch.cuda.synchronize()
            eager_us = a.elapsed_time(b) * 1e3 / steps
            # The same pass captured once as a graph and replayed; every replay is
            # checked bit for bit against the eager result, with eager work between.
            g = torch.cuda.CUDAGraph()
            s = torch.cuda.Stream()
            s.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(s):
                self.run(name)
            torch.cuda.current_stream().wait_stream(s)
            torch.cuda.synchronize()
            with torch.cuda.graph(g):
                self.run(name)
            gout = self.ys
            graph_ok, diffs = True, []
            for _ in range(3):
                g.replay()
                torch.cuda.synchronize()
                graph_ok &= bool(torch.equal(torch.stack(gout), ref))
                diffs.append(float((torch.stack(gout).float() - ref.float()).abs().max()))
                self.run(name)
                torch.cuda.synchronize()
            a.record()
            for _ in range(steps):
                g.replay()
            b.record()
            torch.cuda.synchronize()
            graph_us = a.elapsed_time(b) * 1e3 / steps
            graph_ok &= bool(torch.equal(torch.stack(gout), ref))
            finite = bool(torch.isfinite(ref.float()).all())
            del g
            out[name] = {"nodes": [int(v) for v in self.sel[name]], "unique_experts_per_layer": uniq,
                         "unique_experts_total": sum(uniq), "eager_us": eager_us, "graph_us": graph_us,
                         "graph_replays_match_eager": graph_ok, "outputs_finite": finite,
                         "weight_bytes": sum(u + 1 for u in uniq) * expert_bytes(self.sh.d, self.sh.d_ff)}
            log(f"stack {name}: unique/layer {uniq} (sum {sum(uniq)}), eager {eager_us:.0f} us, "
                f"graph {graph_us:.0f} us, replays match: {graph_ok}")
        out["speedup_cost_aware_vs_confidence"] = out["confidence"]["eager_us"] / out["cost_aware"]["eager_us"]
        out["unique_experts_saved_vs_confidence"] = (out["confidence"]["unique_experts_total"]
                                                     - out["cost_aware"]["unique_experts_total"])
        return out


# --------------------------------------------------------------------------- PMC summary

def summarize_pmc(fetch_dir, write_dir, out_path):
    """Average FETCH_SIZE / WRITE_SIZE (KiB per dispatch) of the gate/up kernel, each
    scaled by what the same counter reads for the 1 GiB calibration copy."""
    def load(d, counter):
        rows = []
        for p in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            with open(p) as f:
                rows += [r for r in csv.DictReader(f) if r.get("Counter_Name") == counter]
        return rows

    def mean_for(rows, pred):
        v = [float(r["Counter_Value"]) for r in rows if pred(r["Kernel_Name"])]
        return (sum(v) / len(v), len(v)) if v else (float("nan"), 0)

    is_gu = lambda n: (GATEUP_KERNEL.replace(" ", "") in n.replace(" ", "")
                       or "_ZN7ecospec17expert_ffn_kernelILi1ELb0E" in n)
    is_copy = lambda n: "bitwise_not" in n
    fr, wr = load(fetch_dir, "FETCH_SIZE"), load(write_dir, "WRITE_SIZE")
    f_gu, nf = mean_for(fr, is_gu)
    w_gu, nw = mean_for(wr, is_gu)
    f_cp, _ = mean_for(fr, is_copy)
    w_cp, _ = mean_for(wr, is_copy)
    cal_f = COPY_BYTES / (f_cp * 1024.0)
    cal_w = COPY_BYTES / (w_cp * 1024.0)
    hbm = f_gu * 1024.0 * cal_f + w_gu * 1024.0 * cal_w
    with open(out_path, "w") as f:
        f.write("# rocprofv3 counter summary: FP8 gate/up kernel, DeepSeek-V3.1 layer, T=64, U=32\n")
        f.write("# commands (repository root, TMPDIR=/tmp):\n")
        f.write("#   rocprofv3 --pmc FETCH_SIZE -d FETCH_DIR --output-format csv -- python3 bench.py --profile\n")
        f.write("#   rocprofv3 --pmc WRITE_SIZE -d WRITE_DIR --output-format csv -- python3 bench.py --profile\n")
        f.write("#   python3 bench.py --summarize-pmc FETCH_DIR WRITE_DIR\n")
        f.write("# counters are KiB per dispatch; each is scaled by COPY_BYTES / (its reading for the calibration\n")
        f.write("# kernel, torch.bitwise_not over 1 GiB of int32, which reads and writes 1 GiB each)\n")
        f.write(f"kernel_source_sha: {source_sha()}\n")
        f.write(f"gateup_dispatches: fetch {nf}, write {nw}\n")
        f.write(f"fetch_kib_per_dispatch: {f_gu:.1f}\n")
        f.write(f"write_kib_per_dispatch: {w_gu:.1f}\n")
        f.write(f"copy_fetch_kib: {f_cp:.1f}\ncopy_write_kib: {w_cp:.1f}\n")
        f.write(f"calibration_fetch: {cal_f:.4f}\ncalibration_write: {cal_w:.4f}\n")
        f.write(f"hbm_bytes_per_launch: {hbm:.0f}\n")
    print(open(out_path).read())


# --------------------------------------------------------------------------- main

def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--T", type=int, default=64)
    ap.add_argument("--U", type=int, default=32)
    ap.add_argument("--sweep", default="8,16,24,32,48,64,96,128,192,256")
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--cpu-tokens", type=int, default=48)
    ap.add_argument("--no-stack", action="store_true", help="skip the 8-layer draft-tree verification step")
    ap.add_argument("--stack-only", action="store_true", help="only the 8-layer draft-tree verification step")
    ap.add_argument("--tokens-only", action="store_true", help="only the tokens-per-expert sweep of the three shapes")
    ap.add_argument("--mx-only", action="store_true", help="only the GPT-OSS shape with bf16 and MX FP8 activations")
    ap.add_argument("--profile", action="store_true", help="short run for rocprofv3 plus a calibration copy")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"))
    ap.add_argument("--pmc-out", default=PMC_SUMMARY, help="where --summarize-pmc writes its summary")
    args = ap.parse_args()

    if args.tokens_only:
        print(json.dumps([token_sweep(n) for n in ("ds", "qwen", "gpt")] + [token_sweep("gpt", act_fmt=1)]))
        return 0
    if args.mx_only:
        print(json.dumps([token_sweep("gpt"), token_sweep("gpt", act_fmt=1), shape_sweep("gpt", [8, 32, 64, 128]),
                          shape_sweep("gpt", [8, 32, 64, 128], act_fmt=1)]))
        return 0
    if args.stack_only:
        import torch
        st = Stack()
        print(json.dumps(st.measure(max(10, args.steps // 2), 3)))
        return 0
    if args.summarize_pmc:
        summarize_pmc(args.summarize_pmc[0], args.summarize_pmc[1], args.pmc_out)
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

    Us = sorted(set([args.U] + ([] if (args.no_sweep or args.profile) else [int(u) for u in args.sweep.split(",")])))
    wl = Workload(args.T, Us, n_pool=16, n_shared_copies=4)
    sh = wl.sh

    if args.profile:
        # The headline's own steps: W warm-ups, then K steps (as the timed region runs them).
        for i in range(args.warmup):
            wl.step(args.U, i)
        torch.cuda.synchronize()
        for i in range(args.steps):
            wl.step(args.U, args.warmup + i)
        # Calibration copy for the HBM counters: one elementwise kernel that reads and
        # writes COPY_BYTES each, with a name nothing else in the run uses.
        src = torch.ones(COPY_BYTES // 4, dtype=torch.int32, device=wl.dev)
        dst = torch.empty_like(src)
        torch.bitwise_not(src, out=dst)
        torch.cuda.synchronize()
        log("profile run done")
        return 0

    # Headline: plain steps (two events), then the same steps with per-kernel marks.
    ms, _ = wl.time_steps(args.U, args.steps, args.warmup, marks=False)
    _, per = wl.time_steps(args.U, args.steps, args.warmup, marks=True)
    B = step_alg_bytes(sh, args.T, args.U)
    gu_ms = sum(per["gateup"]) / len(per["gateup"])
    gu_bytes = gateup_alg_bytes(sh, args.T, args.U)
    gu_gbs = gu_bytes / (gu_ms * 1e-3) / 1e9
    log(f"U={args.U}: step {ms * 1e3:.1f} us, {B / (ms * 1e-3) / 1e9:.0f} GB/s; gate/up {gu_ms * 1e3:.1f} us "
        f"({gu_gbs:.0f} GB/s), down {1e3 * sum(per['down']) / len(per['down']):.1f} us")

    sweep = []
    for U in Us:
        if U == args.U:
            p = per
        else:
            _, p = wl.time_steps(U, max(10, args.steps // 2), 3, marks=True)
        med = pct(p["step"], 0.5)
        sweep.append({"U": U, "step_us": {"p10": pct(p["step"], 0.1) * 1e3, "median": med * 1e3,
                                          "p90": pct(p["step"], 0.9) * 1e3},
                      "verify_us": pct(p["verify"], 0.5) * 1e3, "gateup_us": pct(p["gateup"], 0.5) * 1e3,
                      "down_us": pct(p["down"], 0.5) * 1e3, "combine_us": pct(p["combine"], 0.5) * 1e3,
                      "route_union_us": pct(p["route_union"], 0.5) * 1e3,
                      "fixup_us": pct(p["gateup_fixup"], 0.5) * 1e3,
                      "alg_bytes": step_alg_bytes(sh, args.T, U),
                      "GB_s": step_alg_bytes(sh, args.T, U) / (med * 1e-3) / 1e9,
                      "frac_of_8TBs": step_alg_bytes(sh, args.T, U) / (med * 1e-3) / 1e9 / PEAK_HBM_GBS})
        log(f"  U={U:4d}: step {med * 1e3:8.1f} us  {sweep[-1]['GB_s']:7.0f} GB/s")
    fit = None
    if len(sweep) >= 3:
        a, b, r2 = linfit([s["U"] for s in sweep], [s["step_us"]["median"] for s in sweep])
        fit = {"us_intercept": a, "us_per_expert": b, "r2": r2,
               "GB_s_marginal": expert_bytes(sh.d, sh.d_ff) / (b * 1e-6) / 1e9 if b > 0 else None}

    # Batch scaling: scattered routing (i.i.d. logits), T = 8 .. 256 (T > 64 splits an
    # expert's tokens into groups of 64, each streaming the expert once).
    sweep_t = []
    if not args.no_sweep:
        for T in (8, 16, 32, 64, 128, 256):
            wt = TSweep(wl, T)
            med, uniq = wt.time(max(10, args.steps // 2), 3)
            sweep_t.append({"T": T, "unique_experts_median": uniq, "step_us": med,
                            "GB_s": wt.alg_bytes(uniq) / (med * 1e-6) / 1e9})
            log(f"  T={T:4d}: U~{uniq:5.0f} step {med:8.1f} us")
            del wt

    router = router_timing(wl)
    log(f"router from hidden states {router['router_from_hidden_us']:.1f} us, "
        f"top-k from logits {router['route_from_logits_us']:.1f} us")

    cpu, err = (None, None)
    if not args.no_cpu:
        log("timing the oracle on the host ...")
        cpu, err = cpu_baseline(wl, args.U, args.cpu_tokens)

    variants, others, tokens = None, None, None
    if not args.no_sweep:
        del wl
        torch.cuda.empty_cache()
        variants = variant_timing()
        others = [shape_sweep("qwen", [8, 32, 64, 128]), shape_sweep("gpt", [8, 32, 64, 128]),
                  shape_sweep("gpt", [8, 32, 64, 128], act_fmt=1)]
        tokens = [token_sweep(n) for n in ("ds", "qwen", "gpt")] + [token_sweep("gpt", act_fmt=1)]
        log(f"GPT-OSS layer T=64: plain {variants['gpt_oss_T64_clustered']['plain_swiglu_us']:.1f} us, "
            f"GPT-OSS expert {variants['gpt_oss_T64_clustered']['gpt_oss_expert_us']:.1f} us; "
            f"grouped routing {variants['ds_routing_T64']['grouped_us']:.1f} us")

    stack = None
    if not args.no_stack:
        if "wl" in locals():
            del wl
        torch.cuda.empty_cache()
        st = Stack()
        stack = st.measure(max(10, args.steps // 2), 3)
        del st
        torch.cuda.empty_cache()

    traffic = read_pmc_summary()
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
                     "kernel": "expert_ffn_kernel (FP8 gate/up + SwiGLU)", "alg_bytes_per_launch": gu_bytes,
                     "avg_launch_us": gu_ms * 1e3,
                     "traffic_GB_s": None if traffic is None else traffic / (gu_ms * 1e-3) / 1e9},
        "cpu_baseline": cpu,
        "parity_sampled_rows_max_rel_err": err,
        "kernels_us": {k: 1e3 * sum(v) / len(v) for k, v in per.items()},
        "sweep_T64": sweep,
        "linear_fit_us_vs_U": fit,
        "sweep_T_scattered": sweep_t,
        "stack_8_layers_T16": stack,
        "router": router,
        "variants": variants,
        "sweep_other_shapes_T64": others,
        "sweep_tokens_per_expert_U32": tokens,
    }
    print(json.dumps(out))
    return 0


if __name__ == "__main__":
    sys.exit(main())
