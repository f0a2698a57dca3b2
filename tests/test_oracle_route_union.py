"""Pins for the oracle's router top-k and expert union / grouping (CPU only).

Independent references: numpy's stable argsort (selection order and stable
grouping), Python sets and bincount (Eq. 1 union, counts), scipy's softmax and
expit (gate weights), plus invariants the paper fixes: one token touches
exactly k experts (AR rows of Tables 1 and 3), and k <= U <= min(E, T*k).
"""
import numpy as np
import pytest
import scipy.special as sp
import torch

import oracle
import synth


def _ref_topk(row, k):
    return np.argsort(-row.astype(np.float64), kind="stable")[:k]


@pytest.mark.parametrize("T,E,k", [(8, 16, 2), (5, 128, 8), (3, 256, 8), (4, 128, 4), (2, 7, 7), (6, 33, 1)])
@pytest.mark.parametrize("kind", ["scattered", "ties"])
def test_topk_matches_stable_argsort(T, E, k, kind):
    lg = (synth.logits_scattered(T, E, seed=3) if kind == "scattered" else synth.logits_tie_grid(T, E, seed=3)).numpy()
    idx, w = oracle.route(lg, k, 0)
    for t in range(T):
        assert list(idx[t]) == list(_ref_topk(lg[t], k))


def test_negative_zero_ties_by_index():
    lg = np.array([[0.0, -0.0, 0.0, -0.0, -1.0]], np.float32)
    lg[0, 1] = -0.0
    idx, _ = oracle.route(lg, 4, 0)
    assert list(idx[0]) == [0, 1, 2, 3]


def test_nan_sorts_last_and_ties_by_index():
    lg = np.array([[np.nan, -np.inf, 1.0, np.nan, -3.0]], np.float32)
    idx, _ = oracle.route(lg, 5, 0)
    assert list(idx[0]) == [2, 4, 1, 0, 3]


@pytest.mark.parametrize("score", [0, 1])
def test_weights_match_scipy_and_sum_to_one(score):
    T, E, k = 16, 256, 8
    lg = synth.logits_scattered(T, E, seed=5).numpy()
    idx, w = oracle.route(lg, k, score)
    sel = np.take_along_axis(lg.astype(np.float64), idx.astype(np.int64), axis=1)
    ref = sp.softmax(sel, axis=1) if score == 0 else sp.expit(sel) / sp.expit(sel).sum(1, keepdims=True)
    np.testing.assert_allclose(w, ref, rtol=1e-13, atol=0)
    np.testing.assert_allclose(w.sum(1), 1.0, atol=1e-12)


def test_softmax_weights_shift_invariant_and_equal_to_full_softmax_renorm():
    T, E, k = 4, 128, 8
    lg = synth.logits_scattered(T, E, seed=6).numpy()
    idx, w = oracle.route(lg, k, 0)
    idx2, w2 = oracle.route(lg + np.float32(3.0), k, 0)
    assert np.array_equal(idx, idx2)
    np.testing.assert_allclose(w, w2, rtol=1e-6)
    full = sp.softmax(lg.astype(np.float64), axis=1)
    top = np.take_along_axis(full, idx.astype(np.int64), axis=1)
    np.testing.assert_allclose(w, top / top.sum(1, keepdims=True), rtol=1e-12)


def test_single_selection_has_weight_one():
    lg = synth.logits_scattered(3, 16, seed=7).numpy()
    for score in (0, 1):
        _, w = oracle.route(lg, 1, score)
        assert np.all(w == 1.0)


@pytest.mark.parametrize("T,E,k,gen", [(8, 16, 2, "scattered"), (64, 256, 8, "scattered"), (32, 128, 8, "clustered"),
                                       (64, 128, 4, "clustered"), (1, 256, 8, "scattered"), (16, 256, 8, "exact24")])
def test_union_grouping_brute_force(T, E, k, gen):
    if gen == "scattered":
        idx, _ = oracle.route(synth.logits_scattered(T, E, seed=8).numpy(), k, 0)
    elif gen == "clustered":
        idx = synth.routes_clustered(T, E, k, 0.8, seed=8).astype(np.int32)
    else:
        idx = synth.routes_exact_u(T, E, k, 24, seed=8).astype(np.int32)
    r = oracle.union(idx, E)
    flat = idx.reshape(-1)
    U = len(set(flat.tolist()))
    assert r["n_unique"] == U
    assert k <= U <= min(E, T * k)
    assert list(r["union_ids"][:U]) == sorted(set(flat.tolist()))
    assert np.all(r["union_ids"][U:] == -1)
    assert np.array_equal(r["counts"], np.bincount(flat, minlength=E))
    cnt_u = r["counts"][r["union_ids"][:U]]
    assert np.array_equal(r["offsets"][:U + 1], np.concatenate([[0], np.cumsum(cnt_u)]))
    assert np.all(r["offsets"][U:] == T * k)
    assert np.array_equal(r["perm"], np.argsort(flat, kind="stable"))
    if gen == "exact24":
        assert U == 24


def test_one_token_touches_k_experts(golden):
    # AR rows: a single verified token activates exactly k experts per layer.
    ar = golden["paper_numbers"]["ar_unique_experts"]
    t13 = golden["paper_numbers"]["table13"]
    for name in ("ds", "qwen", "gpt"):
        E, k = t13[name]["experts"], t13[name]["top_k"]
        assert ar[name] == float(k)
        idx, _ = oracle.route(synth.logits_scattered(1, E, seed=9).numpy(), k, 0)
        assert oracle.union(idx, E)["n_unique"] == k


def test_exact_u_and_routes_to_logits_roundtrip():
    for (T, E, k, U) in [(8, 256, 8, 8), (16, 256, 8, 100), (64, 256, 8, 256), (4, 128, 4, 16)]:
        routes = synth.routes_exact_u(T, E, k, U, seed=1)
        lg = synth.routes_to_logits(routes, E, seed=1).numpy()
        idx, _ = oracle.route(lg, k, 1)
        assert np.array_equal(idx, routes)
        assert oracle.union(idx, E)["n_unique"] == U


def test_invalid_expert_index_rejected():
    with pytest.raises(ValueError):
        oracle.union(np.array([[0, 16]], np.int32), 16)


# --------------------------------------------------------------------------- router logits (Section 1)

def _bf16_values(t):
    return t.float().double().numpy()


@pytest.mark.parametrize("T,d,E", [(1, 32, 1), (3, 96, 5), (7, 256, 16), (2, 544, 33)])
def test_router_logits_match_numpy_fp64_product(T, d, E):
    x = synth.activations(T, d, seed=11)
    w = synth.router_weight(E, d, seed=11, std=0.5)
    ref = _bf16_values(x) @ _bf16_values(w).T
    got = oracle.router_logits(x, w)
    assert got.shape == (T, E)
    np.testing.assert_allclose(got, ref, rtol=1e-13, atol=1e-13)


def test_router_logits_one_hot_rows_pick_weight_columns():
    T, d, E = 5, 64, 9
    w = synth.router_weight(E, d, seed=12, std=1.0)
    cols = [0, 17, 31, 32, 63]
    x = torch.zeros(T, d, dtype=torch.bfloat16)
    for t, c in enumerate(cols):
        x[t, c] = 1.0
    got = oracle.router_logits(x, w)
    for t, c in enumerate(cols):
        assert np.array_equal(got[t], _bf16_values(w)[:, c])


def test_router_logits_orientation_rows_are_experts():
    # W_r[e] = (e + 1) everywhere and x[t] = t-th small integer pattern:
    # logit[t][e] = (e + 1) * sum_c x[t][c]; a transposed operand breaks this.
    T, d, E = 3, 32, 6
    w = torch.arange(1, E + 1, dtype=torch.float32)[:, None].expand(E, d).to(torch.bfloat16)
    x = torch.stack([torch.full((d,), float(t + 1)) * ((torch.arange(d) % 3) - 1) for t in range(T)])
    x[:, 0] = 5.0
    x = x.to(torch.bfloat16)
    got = oracle.router_logits(x, w)
    rs = _bf16_values(x).sum(1)
    assert np.array_equal(got, rs[:, None] * np.arange(1, E + 1)[None, :])
