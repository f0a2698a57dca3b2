"""Host selector (moe_select_tree, C++) against the step-by-step Algorithm 1
oracle on random draft trees, every mode; plus the paper's Fig. 3 example."""
import numpy as np
import pytest

import paper_2607_12696_amd as moe
from oracle import select as osel
import synth

MODES = {"cost_ratio": moe.MOE_SEL_COST_RATIO, "confidence": moe.MOE_SEL_CONFIDENCE,
         "global_cost": moe.MOE_SEL_GLOBAL_COST, "cost_diff": moe.MOE_SEL_COST_DIFF}


def test_fig3_example(golden):
    f = golden["fig3_selection"]
    pred = np.array(f["pred"], np.int32)
    s, c = moe.moe_select_tree(f["parent"], f["P"], pred, 16, f["budget"], eps=f["eps"])
    assert list(s) == f["expect_cost_ratio"]
    assert list(c) == [4, 2]
    s, _ = moe.moe_select_tree(f["parent"], f["P"], pred, 16, f["budget"], eps=f["eps"], mode=moe.MOE_SEL_CONFIDENCE)
    assert list(s) == f["expect_confidence"]


@pytest.mark.parametrize("mode", list(MODES))
def test_matches_oracle_on_random_trees(mode):
    rng = np.random.default_rng(123)
    for case in range(250):
        n = int(rng.integers(1, 40))
        L = int(rng.integers(1, 4))
        E = int(rng.choice([8, 16, 64, 70, 256]))
        K = int(rng.integers(1, min(E, 8) + 1))
        branching = int(rng.integers(1, 5))
        parent, P = synth.draft_tree(n, branching, seed=case)
        if case % 5 == 0:  # force exact score ties
            P = np.round(P * 4) / 4
            P[0] = 1.0
            for i in range(1, n):
                P[i] = min(P[i], P[parent[i]])
        pred = synth.tree_expert_sets(parent, L, E, K, float(rng.uniform(0, 1)), seed=case)
        budget = int(rng.integers(0, n + 3))
        lam = float(rng.uniform(0, 0.05))
        B0 = None
        if case % 7 == 3:
            W = (E + 63) // 64
            B0 = rng.integers(0, 2**63, size=(L, W), dtype=np.uint64)
            B0 &= np.uint64(0x5555555555555555)
            if E % 64:
                B0[:, -1] &= np.uint64((1 << (E % 64)) - 1)
        B0_set = None
        if B0 is not None:
            B0_set = {(l, e) for l in range(L) for e in range(E) if (int(B0[l, e // 64]) >> (e % 64)) & 1}
        want, wcost = osel.select(parent, P, pred, budget, eps=0.1, B0=B0_set, mode=mode, lam=lam)
        got, gcost = moe.moe_select_tree(parent, P, pred, E, budget, eps=0.1, lam=lam, mode=MODES[mode], B0=B0)
        assert list(got) == want, (mode, case)
        assert list(gcost) == wcost, (mode, case)


def test_rejects_bad_trees():
    pred = np.zeros((3, 1, 1), np.int32)
    with pytest.raises(moe.MoeError):
        moe.moe_select_tree([0, 0, 1], [1, .5, .2], pred, 4, 2)          # root has a parent
    with pytest.raises(moe.MoeError):
        moe.moe_select_tree([-1, 2, 0], [1, .5, .2], pred, 4, 2)         # parent after child
    with pytest.raises(moe.MoeError):
        moe.moe_select_tree([-1, 0, 0], [1, .5, .2], pred + 4, 4, 2)     # expert id out of range
    with pytest.raises(moe.MoeError):
        moe.moe_select_tree([-1, 0, 0], [1, .5, .2], pred, 4, 2, eps=0.0)  # eps must be > 0 for Eq. 9
    with pytest.raises(moe.MoeError):
        moe.moe_select_tree([-1, 0, 0], [1, .5, .2], pred, 4, 2, mode=7)


@pytest.mark.parametrize("case", ["one_layer", "two_layers"])
@pytest.mark.parametrize("mode", list(MODES))
def test_hand_worked_tree_every_mode(golden, case, mode):
    g = golden["selector_modes"][case]
    pred = np.array(g["pred"], np.int32)
    s, c = moe.moe_select_tree(g["parent"], g["P"], pred, g["E"], g["budget"], eps=g["eps"], lam=g["lambda"],
                               mode=MODES[mode])
    assert list(s) == g["expect"][mode]["nodes"]
    assert list(c) == g["expect"][mode]["costs"]
