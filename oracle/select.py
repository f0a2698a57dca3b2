"""Cost-aware draft selection, step by step -- TEST INFRASTRUCTURE ONLY.

Plain-Python oracle of the paper's draft-tree selection (Section 4.2 and
Algorithm 1 in the appendix):

  * Eq. 4  E_pred(t)     = {(l, e) : e in the top-K predicted experts of layer l}
  * Eq. 7  E_traj(t)     = union of E_pred over the root-to-t path
  * Eq. 8  DeltaCost(t|B) = |E_traj(t) minus B|
  * Eq. 9  S(t)          = P(t) / (DeltaCost(t|B) + eps)
  * Algorithm 1: start from S = {} and B = B0; while |S| < gamma, score every
    unselected node, take the best, add it to S and add E_traj(best) to B.

Modes besides Eq. 9 ("cost_ratio"):
  * "confidence"  rank by P(t) alone (the confidence-driven baseline the paper
    compares against, Sections 1 and 4.2);
  * "global_cost" Eq. 10 of the ablation (Section 5.4): P / (|E_traj| + eps),
    the buffer is never used;
  * "cost_diff"   P - lambda * DeltaCost (a difference form of the trade-off).

Readings where the paper is silent: eps defaults to 0.1; ties in the score go
to the shallower node, then the lower node id; every unselected node is a
candidate; cost counts (layer, expert) pairs over all layers; the loop stops
early if the tree has fewer nodes than the budget.
"""
from __future__ import annotations

MODES = ("cost_ratio", "confidence", "global_cost", "cost_diff")


def _path(parent, i):
    out = []
    while i >= 0:
        out.append(i)
        i = int(parent[i])
    return out[::-1]


def _pred_set(pred, i):
    """E_pred of node i as a set of (layer, expert) pairs (Eq. 4)."""
    return {(l, int(e)) for l in range(len(pred[i])) for e in pred[i][l]}


def traj(parent, pred, i):
    """E_traj of node i (Eq. 7)."""
    s = set()
    for tau in _path(parent, i):
        s |= _pred_set(pred, tau)
    return s


def select(parent, P, pred, budget, eps=0.1, B0=None, mode="cost_ratio", lam=0.0):
    """Returns (selected node ids in pick order, marginal cost of each pick at pick time)."""
    if mode not in MODES:
        raise ValueError(mode)
    n = len(parent)
    depth = [len(_path(parent, i)) - 1 for i in range(n)]
    trajs = [traj(parent, pred, i) for i in range(n)]
    B = set(B0 or ())
    S, costs = [], []
    while len(S) < budget and len(S) < n:
        best, best_key, best_cost = None, None, None
        for i in range(n):
            if i in S:
                continue
            cost = len(trajs[i] - B)
            if mode == "cost_ratio":
                score = P[i] / (cost + eps)
            elif mode == "confidence":
                score = P[i]
            elif mode == "global_cost":
                score = P[i] / (len(trajs[i]) + eps)
            else:
                score = P[i] - lam * cost
            key = (score, -depth[i], -i)
            if best_key is None or key > best_key:
                best, best_key, best_cost = i, key, cost
        S.append(best)
        costs.append(best_cost)
        # The buffer is always tracked so that the reported cost is the true
        # number of new pairs; the confidence and global-cost scores never read it.
        B |= trajs[best]
    return S, costs


def footprint(parent, pred, nodes):
    """Per-layer number of distinct experts over the paths of the given nodes (Eq. 1 per layer)."""
    L = len(pred[0]) if len(pred) else 0
    per = [set() for _ in range(L)]
    for i in nodes:
        for (l, e) in traj(parent, pred, i):
            per[l].add(e)
    return [len(s) for s in per]
