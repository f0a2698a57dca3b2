// Host build of the expert kernels' split bookkeeping (paper_2607_12696_amd/csrc/split.hpp) for the CPU
// tests: the same header the kernels compile, behind plain C entry points.
#include "split.hpp"

using namespace ecospec::split;

extern "C" {
long split_first_unit(const int *cw, int n_groups, long K, long W, long long target)
{
    return first_unit(cw, n_groups, K, W, target);
}
int split_owner_of(const int *cw, int n_groups, long K, int W, long x) { return owner_of(cw, n_groups, K, W, x); }
long long split_contributors(const int *cw, const long long *bound, int n_groups, long K, int W, long ib, long ie)
{
    return contributors(cw, bound, n_groups, K, W, ib, ie);
}
int split_piece_slot(int v, long v0, long v1, long ib, long ie) { return piece_slot(v, v0, v1, ib, ie); }
long split_finished_item(long x0, long x1, long ns) { return finished_item(x0, x1, ns); }
long long split_div_floor(long long a, long long b) { return div_floor(a, b); }
}
