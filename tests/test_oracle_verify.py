"""Pins for the oracle's verify layer (CPU only).

The reference here is a dense numpy SwiGLU MLP on matrices decoded by
independent routes (PyTorch's bf16/float8 conversions, a numpy nibble unpack
and np.kron / np.repeat scale expansion), combined with scipy gate weights,
so that a dropped term, a transposed operand, a wrong scale index or a wrong
sign in the oracle fails.
"""
import numpy as np
import pytest
import scipy.special as sp
import torch

import oracle
import synth

E2M1 = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0, -0.0, -0.5, -1.0, -1.5, -2.0, -3.0, -4.0, -6.0])


def _dense(fmt, w, s):
    """Decode one [N, K] matrix to float64 without the oracle."""
    if fmt == 0:
        return w.to(torch.float64).numpy()
    if fmt == 1:
        q = w.view(torch.float8_e4m3fn).to(torch.float64).numpy()
        return q * np.kron(s.to(torch.float64).numpy(), np.ones((128, 128)))
    p = w.numpy()
    codes = np.empty((p.shape[0], p.shape[1] * 2), np.uint8)
    codes[:, 0::2] = p & 15
    codes[:, 1::2] = p >> 4
    return E2M1[codes] * np.repeat(np.exp2(s.numpy().astype(np.float64) - 127.0), 32, axis=1)


def _ffn_np(x, Wg, Wu, Wd):
    g = x @ Wg.T
    v = x @ Wu.T
    return (g * sp.expit(g) * v) @ Wd.T


def _ref_y(layer, x, idx, w):
    fmt = layer["fmt"]
    xd = x.to(torch.float64).numpy()
    y = np.zeros((x.shape[0], layer["d"]))
    mats = {}
    for e in sorted(set(idx.reshape(-1).tolist())):
        mats[e] = [_dense(fmt, layer[n][e], layer.get("s_" + n, [None] * (e + 1))[e]) for n in ("gate", "up", "down")]
    for t in range(x.shape[0]):
        for j in range(idx.shape[1]):
            y[t] += w[t, j] * _ffn_np(xd[t], *mats[int(idx[t, j])])
        if layer.get("sh_gate") is not None:
            sh = [_dense(fmt, layer["sh_" + n][0], layer["sh_s_" + n][0] if fmt else None) for n in ("gate", "up", "down")]
            y[t] += _ffn_np(xd[t], *sh)
    return y


SMALL = {
    "bf16": synth.Shape("bf16", 256, 128, 8, 2, 0, 0, False),
    "fp8": synth.Shape("fp8", 256, 256, 6, 3, 1, 1, True),
    "mxfp4": synth.Shape("mxfp4", 192, 96, 8, 4, 2, 0, False),
}


@pytest.mark.parametrize("name", list(SMALL))
def test_verify_matches_dense_numpy(name):
    sh = SMALL[name]
    T = 5
    layer = synth.layer_weights(sh, seed=11)
    x = synth.activations(T, sh.d, seed=11)
    lg = synth.logits_scattered(T, sh.E, seed=11).numpy()
    idx, w = oracle.route(lg, sh.k, sh.score)
    y = oracle.verify_tokens(layer, x, idx, w, threads=2)
    ref = _ref_y(layer, x, idx, w)
    np.testing.assert_allclose(y, ref, rtol=1e-10, atol=1e-12 * np.abs(ref).max())


def test_single_token_single_expert_is_dense_swiglu():
    sh = synth.Shape("one", 128, 64, 1, 1, 0, 0, False)
    layer = synth.layer_weights(sh, seed=12)
    x = synth.activations(1, 128, seed=12)
    y = oracle.verify_tokens(layer, x, np.zeros((1, 1), np.int32), np.ones((1, 1)))
    Wg, Wu, Wd = (layer[n][0].to(torch.float64).numpy() for n in ("gate", "up", "down"))
    xd = x.to(torch.float64).numpy()[0]
    g, v = Wg @ xd, Wu @ xd
    ref = Wd @ (g / (1 + np.exp(-g)) * v)
    np.testing.assert_allclose(y[0], ref, rtol=1e-12, atol=1e-15)


def test_fp8_unit_scales_is_plain_e4m3_matrix():
    sh = synth.Shape("fp8u", 128, 128, 2, 1, 1, 0, False)
    layer = synth.layer_weights(sh, seed=13)
    for n in ("gate", "up", "down"):
        layer["s_" + n] = torch.ones_like(layer["s_" + n])
    x = synth.activations(2, 128, seed=13)
    idx = np.array([[1], [0]], np.int32)
    y = oracle.verify_tokens(layer, x, idx, np.ones((2, 1)))
    for t in range(2):
        e = int(idx[t, 0])
        Wg, Wu, Wd = (layer[n][e].view(torch.float8_e4m3fn).to(torch.float64).numpy() for n in ("gate", "up", "down"))
        np.testing.assert_allclose(y[t], _ffn_np(x[t].to(torch.float64).numpy(), Wg, Wu, Wd), rtol=1e-11)


def test_mxfp4_code127_is_plain_e2m1_grid():
    sh = synth.Shape("fp4u", 64, 64, 1, 1, 2, 0, False)
    layer = synth.layer_weights(sh, seed=14)
    for n in ("gate", "up", "down"):
        layer["s_" + n] = torch.full_like(layer["s_" + n], 127)
    x = synth.activations(1, 64, seed=14)
    y = oracle.verify_tokens(layer, x, np.zeros((1, 1), np.int32), np.ones((1, 1)))
    mats = []
    for n in ("gate", "up", "down"):
        p = layer[n][0].numpy()
        codes = np.stack([p & 15, p >> 4], axis=-1).reshape(p.shape[0], -1)
        mats.append(E2M1[codes])
    np.testing.assert_allclose(y[0], _ffn_np(x[0].to(torch.float64).numpy(), *mats), rtol=1e-12)


def test_token_subset_and_thread_count_do_not_change_rows():
    sh = SMALL["fp8"]
    T = 6
    layer = synth.layer_weights(sh, seed=15)
    x = synth.activations(T, sh.d, seed=15)
    idx, w = oracle.route(synth.logits_scattered(T, sh.E, seed=15).numpy(), sh.k, sh.score)
    full = oracle.verify_tokens(layer, x, idx, w, threads=1)
    sub = oracle.verify_tokens(layer, x, idx, w, tokens=[4, 1], threads=3)
    assert np.array_equal(sub, full[[4, 1]])


def test_token_permutation_equivariance():
    sh = SMALL["bf16"]
    T = 4
    layer = synth.layer_weights(sh, seed=16)
    x = synth.activations(T, sh.d, seed=16)
    idx, w = oracle.route(synth.logits_scattered(T, sh.E, seed=16).numpy(), sh.k, 0)
    y = oracle.verify_tokens(layer, x, idx, w)
    pi = np.array([2, 0, 3, 1])
    y2 = oracle.verify_tokens(layer, x[pi], idx[pi], w[pi])
    assert np.array_equal(y2, y[pi])


def test_expert_dict_input_equals_stacked_input():
    sh = SMALL["mxfp4"]
    T = 3
    layer = synth.layer_weights(sh, seed=17)
    x = synth.activations(T, sh.d, seed=17)
    idx, w = oracle.route(synth.logits_scattered(T, sh.E, seed=17).numpy(), sh.k, 0)
    used = sorted(set(idx.reshape(-1).tolist()))
    compact = {"fmt": 2, "d": sh.d, "d_ff": sh.d_ff}
    for n in ("gate", "up", "down", "s_gate", "s_up", "s_down"):
        compact[n] = {e: layer[n][e].clone() for e in used}
    assert np.array_equal(oracle.verify_tokens(compact, x, idx, w), oracle.verify_tokens(layer, x, idx, w))


# --------------------------------------------------------------------------- GPT-OSS expert variant

def _ffn_oai(x, Wg, Wu, Wd, bg, bu, bd, alpha, limit):
    g = np.minimum(x @ Wg.T + bg, limit)
    v = np.clip(x @ Wu.T + bu, -limit, limit)
    return (g * sp.expit(alpha * g) * (v + 1.0)) @ Wd.T + bd


def _with_biases(layer, sh, seed):
    out = dict(layer)
    out["b_gate"] = synth.expert_biases(sh.E, sh.d_ff, seed, "bg")
    out["b_up"] = synth.expert_biases(sh.E, sh.d_ff, seed, "bu")
    out["b_down"] = synth.expert_biases(sh.E, sh.d, seed, "bd")
    out["act"], out["alpha"], out["limit"] = 1, 1.702, 7.0
    return out


def test_oai_single_expert_is_dense_clamped_swiglu():
    sh = synth.Shape("one", 128, 64, 1, 1, 0, 0, False)
    layer = synth.layer_weights(sh, seed=31)
    for n in ("gate", "up", "down"):  # large weights so that both clamps bind on some rows
        layer[n] = (layer[n].float() * 40).to(torch.bfloat16)
    layer = _with_biases(layer, sh, 31)
    x = synth.activations(1, 128, seed=31)
    y = oracle.verify_tokens(layer, x, np.zeros((1, 1), np.int32), np.ones((1, 1)))
    Wg, Wu, Wd = (layer[n][0].to(torch.float64).numpy() for n in ("gate", "up", "down"))
    bg, bu, bd = (layer[n][0].double().numpy() for n in ("b_gate", "b_up", "b_down"))
    xd = x.to(torch.float64).numpy()[0]
    g, v = Wg @ xd + bg, Wu @ xd + bu
    assert (g > 7.0).any() and (v > 7.0).any() and (v < -7.0).any()
    ref = _ffn_oai(xd, Wg, Wu, Wd, bg, bu, bd, 1.702, 7.0)
    np.testing.assert_allclose(y[0], ref, rtol=1e-12, atol=1e-12 * np.abs(ref).max())


def test_oai_clamp_free_limit_differs_from_swiglu_by_silu_term():
    # limit = inf, alpha = 1, no biases: g sigma(g) (v + 1) = silu(g) v + silu(g), so the two
    # activations differ by W_down silu(W_gate x) exactly.
    sh = synth.Shape("one", 64, 32, 1, 1, 0, 0, False)
    layer = synth.layer_weights(sh, seed=32)
    x = synth.activations(1, 64, seed=32)
    one = (np.zeros((1, 1), np.int32), np.ones((1, 1)))
    y0 = oracle.verify_tokens(layer, x, *one)
    y1 = oracle.verify_tokens(dict(layer, act=1, alpha=1.0, limit=float("inf")), x, *one)
    Wg, Wd = (layer[n][0].to(torch.float64).numpy() for n in ("gate", "down"))
    g = Wg @ x.to(torch.float64).numpy()[0]
    np.testing.assert_allclose(y1[0] - y0[0], Wd @ (g * sp.expit(g)), rtol=1e-9, atol=1e-14)


def test_oai_mxfp4_layer_matches_dense_numpy():
    sh = synth.Shape("gpt", 192, 96, 8, 4, 2, 0, False)
    layer = _with_biases(synth.layer_weights(sh, seed=33), sh, 33)
    T = 4
    x = synth.activations(T, sh.d, seed=33)
    idx, w = oracle.route(synth.logits_scattered(T, sh.E, seed=33).numpy(), sh.k, 0)
    y = oracle.verify_tokens(layer, x, idx, w)
    xd = x.to(torch.float64).numpy()
    ref = np.zeros_like(y)
    for t in range(T):
        for j in range(sh.k):
            e = int(idx[t, j])
            mats = [_dense(2, layer[n][e], layer["s_" + n][e]) for n in ("gate", "up", "down")]
            bias = [layer[n][e].double().numpy() for n in ("b_gate", "b_up", "b_down")]
            ref[t] += w[t, j] * _ffn_oai(xd[t], *mats, *bias, 1.702, 7.0)
    np.testing.assert_allclose(y, ref, rtol=1e-10, atol=1e-12 * np.abs(ref).max())
