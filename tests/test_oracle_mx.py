"""Pins for the oracle's MX activation quantiser and the act_fmt 1 layer (CPU only).

The optional MX activation mode quantises the inputs of both projections to
OCP MX FP8: e4m3fn elements with one power-of-two scale 2^E per block of 32
consecutive elements, E = floor(log2(amax)) - 8, nearest value with ties to the
even code, magnitudes of 448 and more saturating.  The reference here builds the
e4m3fn value grid from the format's definition, takes the exponent from
math.frexp, picks the nearest grid value by search, and lists each block's
elements explicitly, so that a wrong exponent, a wrong rounding direction, a
lost tie rule or a wrong block grouping in the oracle fails.  PyTorch's
float8_e4m3fn cast serves as a library cross-check of the rounding.
"""
import math

import numpy as np
import pytest
import scipy.special as sp
import torch

import oracle
import synth

from test_oracle_verify import _dense


def _e4m3_grid():
    """Non-negative finite e4m3fn values and their codes (exponent bias 7, no infinities,
    S.1111.111 is NaN; exponent field 0 holds the subnormals m/8 * 2^-6)."""
    vals = []
    for e in range(16):
        for m in range(8):
            if e == 15 and m == 7:
                continue
            v = (m / 8.0) * 2.0 ** -6 if e == 0 else (1.0 + m / 8.0) * 2.0 ** (e - 7)
            vals.append((v, (e << 3) | m))
    return sorted(vals)


GRID = _e4m3_grid()
GRID_V = np.array([v for v, _ in GRID])


def _nearest(a):
    if a >= 448.0:
        return 448.0
    i = int(np.searchsorted(GRID_V, a))
    if GRID_V[i] == a:
        return a
    lo, hi = GRID[i - 1], GRID[i]
    dl, dh = a - lo[0], hi[0] - a
    if dl != dh:
        return lo[0] if dl < dh else hi[0]
    return lo[0] if lo[1] % 2 == 0 else hi[0]


def _blocks(K):
    return [[i for i in range(32 * b, 32 * b + 32) if i < K] for b in range((K + 31) // 32)]


def ref_quant(v):
    v = np.asarray(v, np.float64)
    out = v.copy()
    exps = []
    for blk in _blocks(v.size):
        amax = max((abs(v[i]) for i in blk), default=0.0)
        if amax == 0.0:
            E = -127
        else:
            E = min(127, max(-127, math.frexp(amax)[1] - 1 - 8))
        exps.append(E)
        for i in blk:
            q = _nearest(abs(v[i]) / 2.0 ** E)
            out[i] = math.copysign(q, v[i]) * 2.0 ** E if v[i] != 0 else 0.0
    return out, np.array(exps)


def _rows(seed, K, n):
    rng = np.random.default_rng(seed)
    rows = []
    for _ in range(n):
        v = rng.standard_normal(K) * np.exp2(rng.integers(-30, 30, size=K // 8 + 1).repeat(8)[:K])
        v[rng.random(K) < 0.05] = 0.0
        rows.append(v)
    return rows


@pytest.mark.parametrize("K", [128, 256, 2880, 96, 200, 50])
def test_quantiser_matches_brute_force(K):
    for v in _rows(K, K, 4):
        for row in (v, torch.tensor(v).to(torch.bfloat16).to(torch.float64).numpy()):
            q, e = oracle.mx_quantize(row)
            rq, re = ref_quant(row)
            assert np.array_equal(e, re)
            assert np.array_equal(q, rq)


def test_quantiser_agrees_with_torch_float8_cast():
    # In-range rounding (|v / 2^E| < 448) against PyTorch's float32 -> float8_e4m3fn cast.
    for v in _rows(7, 1024, 6):
        q, e = oracle.mx_quantize(v)
        scale = np.repeat(np.exp2(e.astype(np.float64)), 32)
        a = v / scale
        ok = np.abs(a) < 448
        t = torch.tensor(a[ok], dtype=torch.float32).to(torch.float8_e4m3fn).to(torch.float64).numpy()
        assert np.array_equal(q[ok], t * scale[ok])


def test_closed_forms_and_ties():
    v = np.zeros(128)
    v[[0, 1, 2, 3]] = [1.0, 1.0 / 3.0, -2.5, 1.925]          # block 0: amax 2.5 -> E = -7
    v[32:38] = [256.0, 8.5, 9.5, -8.5, 500.0 / 512, 0.0]      # block 1: amax 256 -> E = 0
    v[96] = 300.0                                             # block 3: E = 0
    v[127] = 2.0 ** -20                                       # block 3 as well: tiny next to 300
    q, e = oracle.mx_quantize(v)
    assert list(e) == [-7, 0, -127, 0]
    assert list(q[:4]) == [1.0, 0.34375, -2.5, 1.875]        # 128; 42.67 -> 44; 320; 246.4 -> 240 (x 2^-7)
    # 8.5 and 9.5 are ties (to the even code: 8, 10); 0.977 rounds up to 1.0 on the 1/16 grid
    assert list(q[32:38]) == [256.0, 8.0, 10.0, -8.0, 1.0, 0.0]
    assert q[96] == 288.0 and q[127] == 0.0                  # 300 -> 288 (step 32); 2^-20 underflows
    # Saturation: a block whose maximum lies in [448, 512) * 2^E.
    s = np.zeros(64)
    s[5], s[20] = 500.0 * 2.0 ** -3, -470.0 * 2.0 ** -3
    q, e = oracle.mx_quantize(s)
    assert e[0] == -3 and q[5] == 448.0 * 2.0 ** -3 and q[20] == -448.0 * 2.0 ** -3


def test_block_grouping():
    # One large element raises the exponent of its own block of 32 only.
    rng = np.random.default_rng(3)
    v = rng.standard_normal(384)
    q0, e0 = oracle.mx_quantize(v)
    for pos in (229, 63, 64, 0, 383):
        w = v.copy()
        w[pos] = 1e6
        q, e = oracle.mx_quantize(w)
        assert np.nonzero(e != e0)[0].tolist() == [pos // 32]
        others = np.setdiff1d(np.arange(384), np.arange(pos // 32 * 32, pos // 32 * 32 + 32))
        assert np.array_equal(q[others], q0[others])


def test_representable_rows_are_unchanged_and_zero_blocks():
    rng = np.random.default_rng(5)
    for E in (-127, -40, 0, 50, 120):
        v = np.array([GRID_V[rng.integers(len(GRID_V))] for _ in range(256)]) * rng.choice([-1, 1], 256)
        v[7] = 448.0  # the block maximum fixes E exactly for block 0
        v = v * 2.0 ** E
        q, e = oracle.mx_quantize(v)
        assert e[0] == E
        blk0 = _blocks(256)[0]  # every element of block 0 lies on its grid
        assert np.array_equal(q[blk0], v[blk0])
    q, e = oracle.mx_quantize(np.zeros(200))
    assert np.all(q == 0) and np.all(e == -127) and e.size == 7


def _ffn_mx(x, Wg, Wu, Wd):
    g = x @ Wg.T
    v = x @ Wu.T
    h, _ = ref_quant(g * sp.expit(g) * v)
    return h @ Wd.T


def test_act_fmt1_layer_is_quantised_dense_swiglu():
    sh = synth.Shape("mxq", 320, 160, 8, 3, synth.FMT_MXFP4, 0, False)
    layer = synth.layer_weights(sh, seed=4)
    T = 5
    x = synth.activations(T, sh.d, seed=6)
    lg = synth.logits_scattered(T, sh.E, seed=8)
    idx, w = oracle.route(lg, sh.k, sh.score)
    y = oracle.verify_tokens(dict(layer, act_fmt=1), x, idx, w, threads=4)
    y_plain = oracle.verify_tokens(layer, x, idx, w, threads=4)
    xd = x.to(torch.float64).numpy()
    ref = np.zeros((T, sh.d))
    for t in range(T):
        xq, _ = ref_quant(xd[t])
        for j in range(sh.k):
            e = int(idx[t, j])
            mats = [_dense(sh.fmt, layer[n][e], layer["s_" + n][e]) for n in ("gate", "up", "down")]
            ref[t] += w[t, j] * _ffn_mx(xq, *mats)
    scale = np.abs(ref).max()
    assert np.abs(y - ref).max() <= 1e-12 * scale
    # The mode changes the result (it is not the exact-input layer), by a few percent.
    rel = np.abs(y - y_plain).max() / np.abs(y_plain).max()
    assert 1e-4 < rel < 0.2
