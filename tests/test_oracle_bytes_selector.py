"""Pins for the expert byte counts and the selection oracle (CPU only).

Bytes: the paper prints 44.04 MB per DeepSeek-V3.1 FP8 expert (Fig. 1(c)),
about 0.5 GB saved per 0.2 experts per layer over 58 layers (Section 3), and
the per-step HBM reductions of Table 2, which follow from the unique-expert
counts of Table 3 times the layer count of Table 13 times the expert size.

Selection: the worked example of Fig. 3, the prefix-consistency property of
Section 4.2, and reductions of Eq. 9 / Eq. 10 to the confidence order.
"""
import itertools

import numpy as np
import pytest

import oracle
from oracle import select as sel
import synth


def test_ds_expert_is_44_04_MB(golden):
    pn = golden["paper_numbers"]
    wb, sb = oracle.expert_bytes(1, pn["ds_shape"]["d"], pn["ds_shape"]["d_ff"])
    assert wb == 44_040_192
    assert round(wb / 1e6, 2) == pn["ds_expert_fp8_MB"]["value"]
    assert sb == 10_752


def test_point_two_experts_is_half_a_GB(golden):
    pn = golden["paper_numbers"]
    wb, _ = oracle.expert_bytes(1, 7168, 2048)
    g = pn["traffic_per_0p2_experts_GB"]
    assert round(g["experts"] * g["layers"] * wb / 1e9, 1) == g["value"]


def test_table2_reductions_from_table3_and_table13(golden):
    pn = golden["paper_numbers"]
    dims = {"qwen": (0, 4096, 1536), "gpt": (2, 2880, 2880), "ds": (1, 7168, 2048)}
    for name, (fmt, d, f) in dims.items():
        wb, sb = oracle.expert_bytes(fmt, d, f)
        dE = pn["table3_unique_experts"][name]["baseline"] - pn["table3_unique_experts"][name]["ecospec"]
        gb = dE * pn["table13"][name]["moe_layers"] * (wb + sb) / 1e9
        # Table 3 prints unique-expert means to one decimal, so allow 0.2 GB.
        assert abs(gb - pn["table2_reduction_GB"][name]) < 0.2, (name, gb)


def test_fig3_worked_example(golden):
    f = golden["fig3_selection"]
    S, costs = sel.select(f["parent"], f["P"], f["pred"], f["budget"], eps=f["eps"], mode="cost_ratio")
    assert S == f["expect_cost_ratio"]
    S2, _ = sel.select(f["parent"], f["P"], f["pred"], f["budget"], eps=f["eps"], mode="confidence")
    assert S2 == f["expect_confidence"]
    B = sel.traj(f["parent"], f["pred"], 0)
    for node, c in f["expect_costs_step2"].items():
        cost = len(sel.traj(f["parent"], f["pred"], int(node)) - B)
        assert cost == c
        assert round(f["P"][int(node)] / (cost + f["eps"]), 2) == f["expect_scores_step2"][node]


def _random_case(seed, n=30, L=3, E=32, K=4, branching=3):
    parent, P = synth.draft_tree(n, branching, seed=seed)
    pred = synth.tree_expert_sets(parent, L, E, K, 0.6, seed=seed)
    return parent, P, pred


@pytest.mark.parametrize("mode", sel.MODES)
def test_selection_is_prefix_closed(mode):
    for seed in range(20):
        parent, P, pred = _random_case(seed)
        S, _ = sel.select(parent, P, pred, 12, mode=mode, lam=0.01)
        chosen = set()
        for i in S:
            assert parent[i] < 0 or parent[i] in chosen, (mode, seed, S)
            chosen.add(i)


def test_child_never_outscores_parent():
    for seed in range(10):
        parent, P, pred = _random_case(seed)
        B = set()
        for i in range(1, len(parent)):
            p = parent[i]
            cp = len(sel.traj(parent, pred, p) - B)
            cc = len(sel.traj(parent, pred, i) - B)
            assert cp <= cc and P[i] <= P[p]
            assert P[i] / (cc + 0.1) <= P[p] / (cp + 0.1)


def test_identical_sets_reduce_to_confidence_order():
    for seed in range(10):
        parent, P, _ = _random_case(seed)
        pred = np.tile(np.array([[[1, 2, 3, 4]] * 2]), (len(parent), 1, 1))
        a, _ = sel.select(parent, P, pred, 10, mode="cost_ratio")
        b, _ = sel.select(parent, P, pred, 10, mode="confidence")
        assert a == b
        # Confidence order is the stable sort by (P desc, depth asc, id asc).
        assert b == sorted(range(len(parent)), key=lambda i: (-P[i], len(sel._path(parent, i)), i))[:10]


def test_global_cost_is_eq10_static_order():
    for seed in range(10):
        parent, P, pred = _random_case(seed)
        S, _ = sel.select(parent, P, pred, 8, mode="global_cost", eps=0.1)
        key = lambda i: (-(P[i] / (len(sel.traj(parent, pred, i)) + 0.1)), len(sel._path(parent, i)), i)
        assert S == sorted(range(len(parent)), key=key)[:8]


def test_greedy_step_is_argmax_over_all_unselected():
    # Brute force one greedy step over every node and every buffer state reached.
    for seed in range(5):
        parent, P, pred = _random_case(seed, n=12)
        S, costs = sel.select(parent, P, pred, 6)
        B = set()
        for step, pick in enumerate(S):
            cands = [i for i in range(len(parent)) if i not in S[:step]]
            scores = {i: P[i] / (len(sel.traj(parent, pred, i) - B) + 0.1) for i in cands}
            best = max(scores.values())
            assert scores[pick] == best
            assert costs[step] == len(sel.traj(parent, pred, pick) - B)
            B |= sel.traj(parent, pred, pick)


def test_budget_larger_than_tree_selects_all():
    parent, P, pred = _random_case(1, n=7)
    S, _ = sel.select(parent, P, pred, 50)
    assert sorted(S) == list(range(7))


def test_initial_buffer_discounts_costs():
    parent, P, pred = _random_case(2, n=10)
    B0 = sel.traj(parent, pred, 0)
    S, costs = sel.select(parent, P, pred, 3, B0=B0)
    assert S[0] == 0 and costs[0] == 0


@pytest.mark.parametrize("case", ["one_layer", "two_layers"])
@pytest.mark.parametrize("mode", sel.MODES)
def test_hand_worked_tree_every_mode(golden, case, mode):
    # Picks and marginal costs worked out by hand (tests/golden/selector_modes.json): Eq. 9 with the buffer
    # update of Algorithm 1, the confidence order, Eq. 10 without the buffer, and P - lambda * DeltaCost.
    g = golden["selector_modes"][case]
    S, costs = sel.select(g["parent"], g["P"], g["pred"], g["budget"], eps=g["eps"], mode=mode, lam=g["lambda"])
    assert S == g["expect"][mode]["nodes"]
    assert costs == g["expect"][mode]["costs"]


def test_hand_worked_tree_scores(golden):
    # The footprints and round-2 scores of the hand computation (four decimals as written there).
    g = golden["selector_modes"]["one_layer"]
    par, P, pred, eps, lam = g["parent"], g["P"], g["pred"], g["eps"], g["lambda"]
    assert [len(sel.traj(par, pred, i)) for i in range(4)] == [4, 8, 6, 9]
    for node, s in g["expect_global_scores"].items():
        i = int(node)
        assert round(P[i] / (len(sel.traj(par, pred, i)) + eps), 4) == s
    B = sel.traj(par, pred, 0)
    for node, s in g["expect_scores_round2"]["cost_ratio"].items():
        i = int(node)
        assert round(P[i] / (len(sel.traj(par, pred, i) - B) + eps), 4) == s
    for node, s in g["expect_scores_round2"]["cost_diff"].items():
        i = int(node)
        assert round(P[i] - lam * len(sel.traj(par, pred, i) - B), 4) == s
