// Cost-aware draft-tree selection on the host (EcoSpec, Section 4.2 and
// Algorithm 1; the global-cost variant is Eq. 10 of Section 5.4).
//
// Each node's path footprint E_traj (Eq. 7) is a bitset of (layer, expert)
// pairs: [L][ceil(E/64)] 64-bit words, built once from the parent's bitset OR
// the node's own predicted sets (Eq. 4).  The expert buffer B is a bitset of
// the same shape; DeltaCost (Eq. 8) is popcount(traj & ~B).  Every round
// scores all unselected nodes and takes the best by (score desc, depth asc,
// id asc); the buffer then absorbs the pick's footprint.
#include "ecospec_moe.h"

#include <stdint.h>

#include <vector>

namespace {

constexpr long kMaxWords = 1L << 24;  // bitset storage cap: 128 MiB

}  // namespace

extern "C" moe_status_t moe_select_tree(int n, const int32_t *parent, const double *P, int L, int K,
                                        const int32_t *pred, int E, const uint64_t *B0, int budget, double eps,
                                        double lambda, int mode, int32_t *selected, int32_t *marginal_cost,
                                        int32_t *n_selected)
{
    if (n < 1 || n > 65536 || !parent || !P || !pred || L < 1 || K < 1 || (long)L * K > 65536 || E < 1 ||
        E > 4096 || budget < 0 || (budget > 0 && !selected))
        return MOE_ERR_INVALID_ARG;
    if (mode < MOE_SEL_COST_RATIO || mode > MOE_SEL_COST_DIFF) return MOE_ERR_INVALID_ARG;
    if ((mode == MOE_SEL_COST_RATIO || mode == MOE_SEL_GLOBAL_COST) && !(eps > 0.0)) return MOE_ERR_INVALID_ARG;
    if (parent[0] != -1) return MOE_ERR_INVALID_ARG;
    for (int i = 1; i < n; ++i)
        if (parent[i] < 0 || parent[i] >= i) return MOE_ERR_INVALID_ARG;
    for (long q = 0; q < (long)n * L * K; ++q)
        if (pred[q] < 0 || pred[q] >= E) return MOE_ERR_INVALID_ARG;
    const int W = (E + 63) / 64;
    const long words = (long)L * W;
    if (words * n > kMaxWords) return MOE_ERR_UNSUPPORTED;

    // Footprints and depths; parents precede children, so one forward pass suffices.
    std::vector<uint64_t> traj((size_t)words * n, 0ull);
    std::vector<int> depth(n, 0);
    for (int i = 0; i < n; ++i) {
        uint64_t *ti = &traj[(size_t)i * words];
        if (i > 0) {
            const uint64_t *tp = &traj[(size_t)parent[i] * words];
            for (long w = 0; w < words; ++w) ti[w] = tp[w];
            depth[i] = depth[parent[i]] + 1;
        }
        for (int l = 0; l < L; ++l)
            for (int j = 0; j < K; ++j) {
                const int e = pred[((size_t)i * L + l) * K + j];
                ti[(size_t)l * W + e / 64] |= 1ull << (e % 64);
            }
    }
    std::vector<int> size(n);
    for (int i = 0; i < n; ++i) {
        int c = 0;
        for (long w = 0; w < words; ++w) c += __builtin_popcountll(traj[(size_t)i * words + w]);
        size[i] = c;
    }

    std::vector<uint64_t> B((size_t)words, 0ull);
    if (B0)
        for (long w = 0; w < words; ++w) B[w] = B0[w];
    std::vector<char> taken(n, 0);
    const int want = budget < n ? budget : n;
    for (int r = 0; r < want; ++r) {
        int best = -1, best_cost = 0;
        double best_score = 0.0;
        for (int i = 0; i < n; ++i) {
            if (taken[i]) continue;
            const uint64_t *ti = &traj[(size_t)i * words];
            int cost = 0;
            for (long w = 0; w < words; ++w) cost += __builtin_popcountll(ti[w] & ~B[w]);
            double score;
            switch (mode) {
            case MOE_SEL_COST_RATIO: score = P[i] / ((double)cost + eps); break;
            case MOE_SEL_CONFIDENCE: score = P[i]; break;
            case MOE_SEL_GLOBAL_COST: score = P[i] / ((double)size[i] + eps); break;
            default: score = P[i] - lambda * (double)cost; break;
            }
            // Nodes are visited in increasing id, so a later node wins only on a
            // strictly larger score, or an equal score at a smaller depth.
            if (best < 0 || score > best_score || (score == best_score && depth[i] < depth[best])) {
                best = i;
                best_score = score;
                best_cost = cost;
            }
        }
        taken[best] = 1;
        selected[r] = best;
        if (marginal_cost) marginal_cost[r] = best_cost;
        const uint64_t *tb = &traj[(size_t)best * words];
        for (long w = 0; w < words; ++w) B[w] |= tb[w];
    }
    if (n_selected) *n_selected = want;
    return MOE_OK;
}
