// Integer bookkeeping of the cost-weighted split of the expert kernels
// (plain C++, no HIP: constexpr functions are callable from device code, and
// the host build of the unit tests compiles this header as it is).
//
// A launch's work is a sequence of units (one macro step of one item); the
// units of token group g come in a run of K (bands x steps) and each costs
// c_g.  cw[0..n_groups] is the exclusive cost prefix over the groups
// (cw[n_groups] = C, the total per unit of K), so unit x = g*K + r starts at
// cost P_x = cw[g]*K + r*c_g.  Workgroup w of W takes the units with
// C*K*w <= P_x*W < C*K*(w+1): contiguous ranges, every unit exactly once,
// an item cut only where a range starts or ends.
//
// An item cut between workgroups leaves one partial sum per overlapping range
// in the workspace: slot 2*v + 0 if range v starts inside the item (its head
// piece), 2*v + 1 if it starts before (its tail piece).  contributors()
// encodes the overlapping ranges of an item: up to three slots packed, else
// only the first and last workgroup (the finisher then walks the ranges).
#pragma once

#include <stdint.h>

namespace ecospec {
namespace split {

// floor(a / b) for 0 <= a < 2^53 and 0 < b < 2^53: the double quotient is
// within one of it (its relative error is below 2^-53 and a / b < 2^53), so
// one correction makes it exact.  Cheaper on the GPU than a 64-bit division.
constexpr long long div_floor(long long a, long long b)
{
    long long q = (long long)((double)a / (double)b);
    if (q * b > a)
        --q;
    else if ((q + 1) * b <= a)
        ++q;
    return q;
}

// First unit x with P_x * W >= target (0 <= target <= C*K*W); n_groups*K if none.
constexpr long first_unit(const int *cw, int n_groups, long K, long W, long long target)
{
    const long long C = (long long)cw[n_groups] * K;
    if (target <= 0) return 0;
    if (target >= C * W) return (long)n_groups * K;
    int lo = 0, hi = n_groups - 1;  // last group g with cw[g] * K * W < target
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if ((long long)cw[mid] * K * W < target) lo = mid; else hi = mid - 1;
    }
    const long long base = (long long)cw[lo] * K * W, cg = cw[lo + 1] - cw[lo];
    const long long r = div_floor(target - base + cg * W - 1, cg * W);
    return r >= K ? (long)(lo + 1) * K : (long)lo * K + (long)r;
}

// Workgroup whose range holds unit x (0 <= x < n_groups*K).
constexpr int owner_of(const int *cw, int n_groups, long K, int W, long x)
{
    const int g = (int)(x / K);
    const long long cg = cw[g + 1] - cw[g];
    const long long px = (long long)cw[g] * K + (x - (long long)g * K) * cg;
    return (int)div_floor(px * W, (long long)cw[n_groups] * K);
}

// Partial-sum slot of range [v0, v1) for the item of units [ib, ie), or -1 if
// the range is empty (a workgroup with no units).
constexpr int piece_slot(int v, long v0, long v1, long ib, long ie)
{
    return v0 >= v1 ? -1 : 2 * v + ((ib <= v0 && v0 < ie) ? 0 : 1);
}

// Encoding of an item's contributors, bound[w] being workgroup w's first unit
// (bound[W] = all units): up to three slots, 20 bits each in workgroup order,
// their count in bits 60-61 and bit 62 set; past three, bits 62-63 clear and
// (w0 << 16 | w1), the first and last workgroup of the item.
constexpr long long contributors(const int *cw, const long long *bound, int n_groups, long K, int W, long ib, long ie)
{
    const int w0 = owner_of(cw, n_groups, K, W, ib);
    const int w1 = owner_of(cw, n_groups, K, W, ie - 1);
    long long packed = 0;
    int cnt = 0;
    for (int v = w0; v <= w1; ++v) {
        const int s = piece_slot(v, (long)bound[v], (long)bound[v + 1], ib, ie);
        if (s < 0) continue;
        if (cnt < 3) packed |= (long long)s << (20 * cnt);
        ++cnt;
    }
    return cnt <= 3 ? ((1ll << 62) | ((long long)cnt << 60) | packed) : (long long)((w0 << 16) | w1);
}

// The cut item a range finishes, or -1: the item holding the range's first
// unit x0 if it started before x0 and ends inside the range (items of ns
// units).  Every cut item is finished by exactly one range: its last.
constexpr long finished_item(long x0, long x1, long ns)
{
    if (x0 >= x1) return -1;
    const long item = x0 / ns, ib = item * ns, ie = ib + ns;
    return (ib < x0 && ie <= x1) ? item : -1;
}

// Where the combine kernel reads one row of a down item (an 8-byte output
// descriptor, written by the range that holds the item's last unit):
//   kind 0, whole item: bits 0-31 its row of O (the row's routed slot, or
//     T * k + t for the shared expert's row of token t);
//   kind 1, cut over two or three ranges: their slots (10 bits each, bits 0-29,
//     in workgroup order), their count (bits 30-31) and the row r of the group
//     (bits 32-37), the row's place in each slot;
//   kind 2, cut over more than three ranges, none of them empty: the first and
//     last workgroup w0, w1 (bits 0-9, 10-19), bit 20 set if w0's piece is its
//     tail piece (slot 2*w0 + 1, else 2*w0), and r; every later range v adds its
//     head piece, slot 2*v;
//   kind 3: as kind 2, but some range between w0 and w1 is empty, so the
//     reader asks piece_slot() for each of them.
// Workgroups are fewer than 1024 (10 bits).
constexpr uint64_t kOutKindShift = 62;

constexpr uint64_t out_whole(uint32_t p) { return (uint64_t)p; }

// Descriptor of the rows of the cut item [ib, ie) without its row field.
constexpr uint64_t out_cut(const int *cw, const long long *bound, int n_groups, long K, int W, long ib, long ie)
{
    const int w0 = owner_of(cw, n_groups, K, W, ib);
    const int w1 = owner_of(cw, n_groups, K, W, ie - 1);
    uint64_t packed = 0;
    int cnt = 0;
    bool empty = false;
    for (int v = w0; v <= w1; ++v) {
        const int s = piece_slot(v, (long)bound[v], (long)bound[v + 1], ib, ie);
        if (s < 0) {
            empty = true;
            continue;
        }
        if (cnt < 3) packed |= (uint64_t)s << (10 * cnt);
        ++cnt;
    }
    if (cnt <= 3) return (1ull << kOutKindShift) | ((uint64_t)cnt << 30) | packed;
    const bool tail0 = bound[w0] < ib;  // w0's range starts before the item: its tail piece
    return ((empty ? 3ull : 2ull) << kOutKindShift) | ((uint64_t)w1 << 10) | (uint64_t)w0 |
           ((uint64_t)(tail0 ? 1 : 0) << 20);
}

constexpr uint64_t out_with_row(uint64_t code, int r) { return code | ((uint64_t)r << 32); }
constexpr int out_kind(uint64_t code) { return (int)(code >> kOutKindShift); }
constexpr uint32_t out_pos(uint64_t code) { return (uint32_t)code; }
constexpr int out_row(uint64_t code) { return (int)(code >> 32) & 63; }
constexpr int out_count(uint64_t code) { return (int)(code >> 30) & 3; }
constexpr int out_slot(uint64_t code, int i) { return (int)(code >> (10 * i)) & 1023; }
constexpr int out_w0(uint64_t code) { return (int)code & 1023; }
constexpr int out_w1(uint64_t code) { return (int)(code >> 10) & 1023; }
constexpr int out_tail0(uint64_t code) { return (int)(code >> 20) & 1; }

constexpr bool packed_contributors(long long code) { return (code >> 62) != 0; }
constexpr int packed_count(long long code) { return (int)((code >> 60) & 3); }
constexpr int packed_slot(long long code, int i) { return (int)((code >> (20 * i)) & 0xfffff); }
constexpr int first_worker(long long code) { return (int)(code >> 16) & 0xffff; }
constexpr int last_worker(long long code) { return (int)code & 0xffff; }

}  // namespace split
}  // namespace ecospec
