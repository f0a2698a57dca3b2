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


# --------------------------------------------------------------------------- group-limited routing

def test_grouped_route_hand_example():
    # E=8 in G=4 pairs, keep 2 groups, k=4.  All logits 0 -> s = 0.5 and c = 0.5 + bias.
    # Group scores (top-2 sums): g0 0.95+0.5=1.45, g1 0.8+0.75=1.55, g2 0.55+0.5=1.05, g3 0.7+0.7=1.4.
    # Kept: g1, g0 -> candidates 0..3, ranked by c: 0 (0.95), 2 (0.8), 3 (0.75), 1 (0.5).  Plain top-4
    # of c would take expert 6 (0.7) instead of 1.  Weights: equal s, so 2.5 / 4 each.
    lg = np.zeros((1, 8), np.float32)
    b = np.array([0.45, 0, 0.3, 0.25, 0, 0.05, 0.2, 0.2], np.float32)
    idx, w = oracle.route_grouped(lg, b, 4, 4, 2, 2.5)
    assert list(idx[0]) == [0, 2, 3, 1]
    np.testing.assert_allclose(w[0], [0.625] * 4, rtol=0, atol=1e-15)
    # The bias steers the choice but not the weights: raise s of expert 2 (logit ln 3 -> s = 3/4).
    lg[0, 2] = np.float32(np.log(3.0))
    idx, w = oracle.route_grouped(lg, b, 4, 4, 2, 1.0)
    assert list(idx[0]) == [2, 0, 3, 1]  # c: 1.05, 0.95, 0.75, 0.5
    s2 = 1.0 / (1.0 + np.exp(-np.float64(lg[0, 2])))
    np.testing.assert_allclose(w[0], np.array([s2, 0.5, 0.5, 0.5]) / (s2 + 1.5), rtol=1e-15)


def test_grouped_route_one_group_is_plain_sigmoid_topk():
    T, E, k = 16, 64, 6
    lg = synth.logits_scattered(T, E, seed=21).numpy()
    idx, w = oracle.route_grouped(lg, None, k, 1, 1, 1.0)
    idx_p, w_p = oracle.route(lg, k, 1)
    assert np.array_equal(idx, idx_p)
    np.testing.assert_allclose(w, w_p, rtol=1e-13)


def _grouped_brute(lg, b, k, G, TG, scale):
    """Best TG-subset of groups by enumeration, then a full sort of the candidates."""
    import itertools
    T, E = lg.shape
    gs = E // G
    out_i, out_w = [], []
    for t in range(T):
        s = 1.0 / (1.0 + np.exp(-lg[t].astype(np.float64)))
        c = s + (0.0 if b is None else b.astype(np.float64))
        gsc = np.sort(c.reshape(G, gs), axis=1)[:, ::-1][:, :2].sum(1)
        best = max(itertools.combinations(range(G), TG), key=lambda sub: gsc[list(sub)].sum())
        cand = np.concatenate([np.arange(g * gs, (g + 1) * gs) for g in sorted(best)])
        sel = cand[np.argsort(-c[cand], kind="stable")[:k]]
        out_i.append(sel)
        out_w.append(scale * s[sel] / s[sel].sum())
    return np.array(out_i), np.array(out_w)


@pytest.mark.parametrize("E,G,TG,k,bias", [(256, 8, 4, 8, True), (32, 4, 2, 4, False), (64, 16, 3, 5, True),
                                           (24, 3, 3, 7, True), (256, 8, 1, 8, True)])
def test_grouped_route_matches_subset_enumeration(E, G, TG, k, bias):
    T = 12
    lg = synth.logits_scattered(T, E, seed=E + G).numpy()
    b = synth.router_bias(E, seed=E).numpy() if bias else None
    idx, w = oracle.route_grouped(lg, b, k, G, TG, 2.5)
    ri, rw = _grouped_brute(lg, b, k, G, TG, 2.5)
    assert np.array_equal(idx, ri)
    np.testing.assert_allclose(w, rw, rtol=1e-13)
    # invariants: at most TG groups touched, weights sum to the scale
    assert all(len(set(int(e) // (E // G) for e in row)) <= TG for row in idx)
    np.testing.assert_allclose(w.sum(1), 2.5, rtol=1e-13)


def test_grouped_route_rejects_bad_shapes():
    lg = np.zeros((1, 12), np.float32)
    for args in [(4, 5, 2), (4, 12, 2), (4, 4, 5), (7, 4, 2), (4, 4, 0)]:  # E%G, E/G<2, TG>G, k>TG*E/G, TG<1
        with pytest.raises(ValueError):
            oracle.route_grouped(lg, None, args[0], args[1], args[2], 1.0)
