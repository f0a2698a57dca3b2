"""GPU parity of the MXFP4 path at the edges of the e8m0 scale code (OCP MX: code c scales by 2^(c-127),
code 0 by 2^-127, code 255 is NaN), against the oracle's decode of the same codes."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_12696_amd as moe
import synth

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

DEV = torch.device("cuda:0")
YTOL = 1e-2
MX = synth.Shape("mxfp4", 320, 160, 16, 4, synth.FMT_MXFP4, 0, False)
MX_K1 = synth.Shape("mxfp4_k1", 320, 160, 4, 1, synth.FMT_MXFP4, 0, False)


def _dev(layer):
    return moe.pack_layer({k: (v.to(DEV) if hasattr(v, "to") else v) for k, v in layer.items()})


def _run(layer, sh, T, seed):
    x = synth.activations(T, sh.d, seed=seed)
    lg = synth.logits_scattered(T, sh.E, seed=seed + 1)
    y, _ = moe.moe_verify_step(x.to(DEV), lg.to(DEV), _dev(layer), sh.k, sh.score)
    torch.cuda.synchronize()
    idx, w = oracle.route(lg.numpy(), sh.k, sh.score)
    return y.float().cpu().numpy(), oracle.verify_tokens(layer, x, idx, w, threads=8), idx


def _codes(shape, lo, hi, seed):
    g = torch.Generator().manual_seed(seed)
    return torch.randint(lo, hi + 1, shape, generator=g, dtype=torch.int32).to(torch.uint8)


@pytest.mark.parametrize("T", [8, 64])
def test_wide_range_of_scale_codes(T):
    """Scale codes spread over 2^-15 .. 2^15 on every matrix: each code's power of two is applied."""
    layer = synth.layer_weights(MX, seed=31)
    for i, nm in enumerate(("s_gate", "s_up", "s_down")):
        layer[nm] = _codes(tuple(layer[nm].shape), 112, 142, 100 + i)
    y, ref, _ = _run(layer, MX, T, seed=T)
    err = np.abs(y - ref).max() / np.abs(ref).max()
    print(f"T={T}: rel err {err:.3e}", flush=True)
    assert err <= YTOL


def test_smallest_scale_code_on_the_down_projection():
    """Code 0 (2^-127) and 1 on every down block, one expert per token: y is made of those blocks alone,
    decoded to subnormal and smallest-normal bf16 weights."""
    layer = synth.layer_weights(MX_K1, seed=32)
    layer["s_down"] = _codes(tuple(layer["s_down"].shape), 0, 1, 7)
    y, ref, _ = _run(layer, MX_K1, 16, seed=5)
    assert np.isfinite(y).all()
    err = np.abs(y - ref).max() / np.abs(ref).max()
    print(f"rel err {err:.3e}, max|y| {np.abs(ref).max():.3e}", flush=True)
    assert err <= YTOL


def test_nan_scale_code_reaches_exactly_the_routed_tokens():
    """Code 255 (NaN) on one block of one gate row of one expert: exactly the tokens routed to that expert
    get NaN rows; the others match the oracle."""
    layer = synth.layer_weights(MX, seed=33)
    T = 32
    _, _, idx = _run(layer, MX, T, seed=9)
    e = int(idx[0, 0])
    sg = layer["s_gate"].clone()
    sg[e, 5, 3] = 255
    layer["s_gate"] = sg
    y, ref, idx = _run(layer, MX, T, seed=9)
    hit = (idx == e).any(axis=1)
    assert np.isnan(ref[hit]).all() and not np.isnan(ref[~hit]).any()
    assert np.array_equal(np.isnan(y).all(axis=1), hit) and not np.isnan(y[~hit]).any()
    err = np.abs(y[~hit] - ref[~hit]).max() / np.abs(ref[~hit]).max()
    assert err <= YTOL
