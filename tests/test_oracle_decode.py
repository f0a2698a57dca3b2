"""Pins for the oracle's exact decoders (CPU only).

Each decoder is checked against something other than itself: the OCP format
tables (golden fixture), PyTorch's independent float8/bfloat16 conversions for
every code, and a numpy expansion of the block scales.
"""
import numpy as np
import pytest
import torch

import oracle


def _same(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    both_nan = np.isnan(a) & np.isnan(b)
    eq = (a == b) & (np.signbit(a) == np.signbit(b))
    return bool(np.all(both_nan | eq))


def test_e4m3fn_all_codes_match_torch():
    mine = oracle.decode_table(0)
    ref = torch.arange(256, dtype=torch.int32).to(torch.uint8).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    assert _same(mine, ref)


def test_e4m3fn_spec_values(golden):
    t = oracle.decode_table(0)
    for code, val in golden["ocp_formats"]["e4m3fn"].items():
        if code == "nan":
            for c in val:
                assert np.isnan(t[int(c, 16)])
            continue
        assert t[int(code, 16)] == val and np.signbit(t[int(code, 16)]) == np.signbit(val)
    assert np.nanmax(t) == 448.0 and np.isnan(t).sum() == 2


def test_e2m1_table_matches_spec(golden):
    assert _same(oracle.decode_table(1), golden["ocp_formats"]["e2m1"])


def test_e8m0_spec_values(golden):
    t = oracle.decode_table(2)
    for code, val in golden["ocp_formats"]["e8m0"].items():
        if code == "nan":
            assert all(np.isnan(t[c]) for c in val)
        else:
            assert t[int(code)] == val
    # consecutive codes double
    assert np.all(t[1:255] == 2.0 * t[0:254])


def test_bf16_all_codes_match_torch():
    mine = oracle.decode_table(3)
    ref = torch.arange(65536, dtype=torch.int32).to(torch.int16).view(torch.bfloat16).to(torch.float64).numpy()
    assert _same(mine, ref)


def test_fp8_block_scale_indexing():
    # Distinct scale per 128x128 block: a transposed or swapped scale index fails.
    rng = np.random.default_rng(1)
    N, K = 256, 384
    q = rng.integers(0, 256, (N, K), dtype=np.uint8)
    q[(q & 0x7F) == 0x7F] = 0x3C
    s = (np.arange(1, 1 + (N // 128) * (K // 128), dtype=np.float32) * 0.37).reshape(N // 128, K // 128)
    dq = torch.from_numpy(q).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    ref = dq * np.kron(s.astype(np.float64), np.ones((128, 128)))
    for (n, c) in [(0, 0), (127, 127), (128, 0), (0, 128), (255, 383), (130, 260), (5, 300), (200, 10)]:
        assert oracle.weight_at(1, q, s, n, c) == ref[n, c]


def test_mxfp4_nibble_order_and_scale_indexing(golden):
    rng = np.random.default_rng(2)
    N, K = 8, 128
    packed = rng.integers(0, 256, (N, K // 2), dtype=np.uint8)
    sc = rng.integers(118, 124, (N, K // 32), dtype=np.uint8)
    grid = np.array(golden["ocp_formats"]["e2m1"])
    codes = np.empty((N, K), np.uint8)
    codes[:, 0::2] = packed & 15
    codes[:, 1::2] = packed >> 4
    ref = grid[codes] * np.repeat(np.exp2(sc.astype(np.float64) - 127.0), 32, axis=1)
    for n in range(N):
        for c in range(0, K, 7):
            assert oracle.weight_at(2, packed, sc, n, c) == ref[n, c]


@pytest.mark.parametrize("fmt", [0, 1, 2])
def test_expert_byte_formula_matches_generator(fmt):
    import synth
    for (d, f) in [(7168, 2048), (4096, 1536), (2880, 2880), (256, 128)]:
        if fmt == 1 and (d % 128 or f % 128):
            continue
        assert oracle.expert_bytes(fmt, d, f) == synth.expert_bytes(d, f, fmt)
