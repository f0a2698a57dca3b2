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
unsigned long long split_out_cut(const int *cw, const long long *bound, int n_groups, long K, int W, long ib, long ie)
{
    return out_cut(cw, bound, n_groups, K, W, ib, ie);
}
unsigned long long split_out_whole(unsigned p) { return out_whole(p); }
unsigned long long split_out_with_row(unsigned long long code, int r) { return out_with_row(code, r); }
// Decoded fields of a descriptor: kind, pos, row, count, slot 0..2, w0, w1, tail0.
void split_out_fields(unsigned long long code, int *f)
{
    f[0] = out_kind(code);
    f[1] = (int)out_pos(code);
    f[2] = out_row(code);
    f[3] = out_count(code);
    for (int i = 0; i < 3; ++i) f[4 + i] = out_slot(code, i);
    f[7] = out_w0(code);
    f[8] = out_w1(code);
    f[9] = out_tail0(code);
}
}
