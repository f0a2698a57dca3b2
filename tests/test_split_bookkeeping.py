"""CPU test of the expert kernels' work split (paper_2607_12696_amd/csrc/split.hpp).

The kernels lay all (item, macro step) units of a launch end to end and cut
them into one range per workgroup by modelled cost; an item cut between
workgroups is finished from the partial sums its ranges park, and which sums
get added is decided by this integer bookkeeping alone.  The header is
compiled here for the host (g++) and checked against a brute-force statement
of the split:

  * unit x of group g (offset r) starts at cost P_x = cw[g]*K + r*c_g and
    belongs to the workgroup w with C*K*w <= P_x*W < C*K*(w+1);
  * a range parks a cut item's piece in slot 2w if the item holds the range's
    first unit, else 2w + 1 (the kernel's rule: item start <= range start);
  * the contributors of an item are the ranges that hold its units, in
    workgroup order; up to three are packed, past three the first and last
    workgroup are stored and the finisher walks the ranges between;
  * each cut item has exactly one finisher, the range that holds its last unit;
  * the down launch's output descriptor of a cut item's rows names the same
    slots: packed up to three, else the first and last workgroup and whether
    the first one's piece is its tail piece, every later non-empty range
    adding its head piece (and a flag that some range between is empty).

Cases span W in {256, 512} (one or two workgroups per compute unit) and small
grids, group costs of the kernels' form (A + 2 * token blocks) and arbitrary,
and shapes where one item is spread over many workgroups (the > 3 encoding).
"""
import ctypes as C
import os
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_12696_amd", "csrc")


@pytest.fixture(scope="module")
def lib(tmp_path_factory):
    out = str(tmp_path_factory.mktemp("split") / "libsplit.so")
    src = os.path.join(ROOT, "tests", "split_shim.cpp")
    subprocess.run(["g++", "-O1", "-std=c++17", "-shared", "-fPIC", f"-I{CSRC}", src, "-o", out], check=True)
    L = C.CDLL(out)
    p, i, l, ll = C.c_void_p, C.c_int, C.c_long, C.c_longlong
    L.split_first_unit.argtypes = [p, i, l, l, ll]
    L.split_first_unit.restype = l
    L.split_owner_of.argtypes = [p, i, l, i, l]
    L.split_owner_of.restype = i
    L.split_contributors.argtypes = [p, p, i, l, i, l, l]
    L.split_contributors.restype = ll
    L.split_piece_slot.argtypes = [i, l, l, l, l]
    L.split_piece_slot.restype = i
    L.split_finished_item.argtypes = [l, l, l]
    L.split_finished_item.restype = l
    L.split_div_floor.argtypes = [ll, ll]
    L.split_div_floor.restype = ll
    u = C.c_ulonglong
    L.split_out_cut.argtypes = [p, p, i, l, i, l, l]
    L.split_out_cut.restype = u
    L.split_out_whole.argtypes = [C.c_uint]
    L.split_out_whole.restype = u
    L.split_out_with_row.argtypes = [u, i]
    L.split_out_with_row.restype = u
    L.split_out_fields.argtypes = [u, p]
    L.split_out_fields.restype = None
    return L


def out_fields(lib, code):
    f = np.zeros(10, np.int32)
    lib.split_out_fields(code, f.ctypes.data)
    return dict(zip(("kind", "pos", "row", "count", "s0", "s1", "s2", "w0", "w1", "tail0"), f.tolist()))


def out_slots(lib, code, bound):
    """The partial-sum slots a reader of the output descriptor adds, in order (what the combine kernel
    does: kind 3 consults the ranges, the others do not)."""
    f = out_fields(lib, code)
    if f["kind"] == 1:
        return [f["s0"], f["s1"], f["s2"]][:f["count"]]
    assert f["kind"] in (2, 3), f
    slots = [2 * f["w0"] + f["tail0"]]
    for v in range(f["w0"] + 1, f["w1"] + 1):
        if f["kind"] == 2 or bound[v] < bound[v + 1]:
            slots.append(2 * v)
    return slots


def brute_owner(costs, K, W):
    """Owner of every unit straight from the definition: the number of workgroup start thresholds
    C*K*w (w = 1..W-1) at or below P_x*W."""
    costs = np.asarray(costs, np.int64)
    cw = np.concatenate([[0], np.cumsum(costs)])
    C_tot = int(cw[-1])
    g = np.repeat(np.arange(len(costs)), K)
    r = np.tile(np.arange(K), len(costs))
    px = cw[g] * K + r * costs[g]
    thr = C_tot * K * np.arange(1, W, dtype=np.int64)
    return (px[:, None] * W >= thr[None, :]).sum(1)


def run_case(lib, costs, nbands, nsteps, W):
    n = len(costs)
    K = nbands * nsteps
    cw = np.concatenate([[0], np.cumsum(costs)]).astype(np.int32)
    cwp = cw.ctypes.data
    owner = brute_owner(costs, K, W)
    units = n * K
    # Ranges: bound[w] = first unit whose owner is >= w.
    bound = np.searchsorted(owner, np.arange(W + 1), side="left").astype(np.int64)
    C_tot = int(cw[-1])
    got_bound = np.array([lib.split_first_unit(cwp, n, K, W, C_tot * K * w) for w in range(W + 1)], np.int64)
    assert np.array_equal(got_bound, bound)
    sample = range(units) if units <= 4000 else np.random.default_rng(units).integers(0, units, 4000)
    for x in sample:
        assert lib.split_owner_of(cwp, n, K, W, int(x)) == owner[x], int(x)

    # What each range parks (kernel rule) and which cut items it finishes.
    parked = {}      # item -> list of (workgroup, slot) in workgroup order
    finisher = {}
    for w in range(W):
        x0, x1 = int(bound[w]), int(bound[w + 1])
        if x0 >= x1:
            assert lib.split_finished_item(x0, x1, nsteps) == -1
            continue
        slots = []
        for item in range(x0 // nsteps, (x1 - 1) // nsteps + 1):
            ib, ie = item * nsteps, (item + 1) * nsteps
            if ib >= x0 and ie <= x1:
                continue  # whole in this range: finished in registers
            slot = 2 * w + (0 if ib <= x0 else 1)
            slots.append(slot)
            parked.setdefault(item, []).append((w, slot))
        assert len(set(slots)) == len(slots), (w, slots)  # a range never parks two pieces in one slot
        f = lib.split_finished_item(x0, x1, nsteps)
        if f >= 0:
            finisher.setdefault(f, []).append(w)
    bptr = bound.ctypes.data
    wide = 0
    for item, pieces in parked.items():
        assert len(pieces) >= 2
        assert finisher.get(item) == [pieces[-1][0]], (item, pieces, finisher.get(item))
        ib, ie = item * nsteps, (item + 1) * nsteps
        code = lib.split_contributors(cwp, bptr, n, K, W, ib, ie)
        want = [s for _, s in pieces]
        if (code >> 62) & 1:
            cnt = (code >> 60) & 3
            got = [(code >> (20 * i)) & 0xFFFFF for i in range(cnt)]
            assert len(want) <= 3
        else:
            assert code >= 0 and len(want) > 3
            wide += 1
            w0, w1 = (code >> 16) & 0xFFFF, code & 0xFFFF
            got = []
            for v in range(w0, w1 + 1):
                s = lib.split_piece_slot(v, int(bound[v]), int(bound[v + 1]), ib, ie)
                if s >= 0:
                    got.append(s)
        assert got == want, (item, got, want)
        # The down launch's output descriptor of the item's rows names the same slots, for every row.
        desc = lib.split_out_cut(cwp, bptr, n, K, W, ib, ie)
        assert out_slots(lib, desc, bound) == want, (item, hex(desc), want)
        w0, w1 = int(owner[ib]), int(owner[ie - 1])
        empty = any(bound[v] >= bound[v + 1] for v in range(w0, w1 + 1))
        assert out_fields(lib, desc)["kind"] == (1 if len(want) <= 3 else 3 if empty else 2)
        for r in (0, 1, 37, 63):
            f = out_fields(lib, lib.split_out_with_row(desc, r))
            assert f["row"] == r and out_slots(lib, lib.split_out_with_row(desc, r), bound) == want
    # Items nobody parked are whole in exactly one range, and no cut item lacks a finisher.
    assert set(finisher) == set(parked)
    return wide


KERNEL_COST = {"bf16": 29, "fp8": 12, "fp4": 8, "fp4_mx": 16}


def kernel_costs(fmt, Ms):
    return [KERNEL_COST[fmt] + 2 * ((m + 15) // 16) for m in Ms]


# (fmt, tokens per group, nbands, nsteps): the launches of the full shapes and of a small shape that spreads
# one item over many workgroups.
SHAPE_CASES = [
    ("fp8", [16] * 32 + [64], 16, 56, "DeepSeek-V3.1 gate/up, T 64, U 32 + shared"),
    ("fp8", [16] * 32 + [64], 28, 16, "DeepSeek-V3.1 down, T 64, U 32 + shared"),
    ("fp8", [1] * 8 + [1], 16, 56, "DeepSeek-V3.1 gate/up, T 1"),
    ("fp8", [1] * 8 + [1], 28, 16, "DeepSeek-V3.1 down, T 1"),
    ("bf16", [1] * 8, 12, 32, "Qwen3 gate/up, T 1"),
    ("bf16", [1] * 8, 16, 12, "Qwen3 down, T 1"),
    ("fp4", [1] * 4, 23, 12, "GPT-OSS gate/up, T 1 (two 128-wide blocks per step)"),
    ("fp4", [1] * 4, 12, 12, "GPT-OSS down, T 1"),
    ("bf16", [1], 16, 16, "bf16 d = d_ff = 2048, one expert, T 1: gate/up"),
    ("bf16", [1], 8, 16, "bf16 d = d_ff = 2048, one expert, T 1: down"),
    ("fp8", [64, 64, 64, 64, 30, 7, 1], 16, 56, "uneven token groups"),
]


@pytest.mark.parametrize("fmt,Ms,nbands,nsteps,what", SHAPE_CASES, ids=[c[4] for c in SHAPE_CASES])
@pytest.mark.parametrize("W", [256, 512])
def test_split_of_kernel_shapes(lib, fmt, Ms, nbands, nsteps, what, W):
    run_case(lib, kernel_costs(fmt, Ms), nbands, nsteps, W)


def test_wide_items_reach_the_walk_encoding(lib):
    # T = 1 shapes put four or more ranges on one item: the encoding the finisher walks must be reached.
    wide = 0
    for fmt, Ms, nb, ns, _ in SHAPE_CASES:
        if Ms[0] == 1:
            wide += run_case(lib, kernel_costs(fmt, Ms), nb, ns, 256)
    assert wide > 0


def test_random_costs_and_grids(lib):
    rng = np.random.default_rng(7)
    wide = 0
    for case in range(150):
        n = int(rng.integers(1, 40))
        costs = rng.integers(1, 120, n).tolist()
        nbands = int(rng.integers(1, 12))
        nsteps = int(rng.integers(1, 30))
        W = int(rng.choice([1, 2, 3, 7, 64, 256, 512]))
        wide += run_case(lib, costs, nbands, nsteps, W)
    assert wide > 0


def test_whole_item_descriptor(lib):
    # A whole item's row: kind 0 and its grouped position, for positions up to the largest a call has.
    for p in (0, 1, 4095, 2**24 + 2**18, 2**25 - 1):
        f = out_fields(lib, lib.split_out_whole(p))
        assert f["kind"] == 0 and f["pos"] == p


def test_descriptor_walk_with_empty_ranges(lib):
    # More workgroups than units: ranges between an item's first and last contributor are empty, and the
    # descriptor must say so (kind 3) for the reader to skip them.
    kinds = set()
    for W in (64, 256, 512):
        for costs, nb, ns in (([200, 1, 1], 1, 3), ([5], 2, 3), ([1, 90], 1, 7)):
            run_case(lib, costs, nb, ns, W)
            K = nb * ns
            cw = np.concatenate([[0], np.cumsum(costs)]).astype(np.int32)
            owner = brute_owner(costs, K, W)
            bound = np.searchsorted(owner, np.arange(W + 1), side="left").astype(np.int64)
            for item in range(len(costs) * nb):
                ib, ie = item * ns, (item + 1) * ns
                if owner[ib] != owner[ie - 1]:
                    kinds.add(out_fields(lib, lib.split_out_cut(cw.ctypes.data, bound.ctypes.data, len(costs), K, W,
                                                                ib, ie))["kind"])
    assert 3 in kinds


def test_div_floor_is_exact(lib):
    # The split's divisions go through a double quotient corrected by one step; its operands stay
    # below 2^45 (cost total x units per group x workgroups).  Exact against Python integers,
    # including quotients that sit on or next to an integer, where the double rounds either way.
    rng = np.random.default_rng(11)
    cases = [(0, 1), (1, 1), (2**45, 1), (2**45 - 1, 3), (2**52, 2**52 - 1), (2**52 - 1, 2**52)]
    for _ in range(3000):
        b = int(rng.integers(1, 2**int(rng.integers(1, 45))))
        q = int(rng.integers(0, 2**45 // b + 1))
        for a in (q * b - 1, q * b, q * b + 1, q * b + b - 1):
            if 0 <= a < 2**52:
                cases.append((a, b))
    for a, b in cases:
        assert lib.split_div_floor(a, b) == a // b, (a, b)


def test_first_unit_at_large_magnitudes(lib):
    # Targets near the largest the kernels produce (4096 groups, 2^17 units per group, 512
    # workgroups): first_unit against the definition in exact integers.
    rng = np.random.default_rng(5)
    for _ in range(40):
        n = int(rng.integers(1, 4097))
        costs = rng.integers(8, 42, n)
        cw = np.concatenate([[0], np.cumsum(costs)]).astype(np.int32)
        K = int(rng.integers(1, 2**17))
        W = int(rng.choice([256, 512]))
        C_tot = int(cw[-1]) * K
        for w in rng.integers(0, W + 1, 16).tolist():
            target = C_tot * int(w)
            # smallest unit x = g*K + r with (cw[g]*K + r*c_g) * W >= target
            if target <= 0:
                want = 0
            elif target >= C_tot * W:
                want = n * K
            else:
                g = int(np.searchsorted(cw[:-1].astype(np.int64) * K * W, target, side="left")) - 1
                base, cg = int(cw[g]) * K * W, int(costs[g])
                r = -(-(target - base) // (cg * W))
                want = (g + 1) * K if r >= K else g * K + r
            got = lib.split_first_unit(cw.ctypes.data, n, K, W, target)
            assert got == want, (n, K, W, w)
