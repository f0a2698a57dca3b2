"""moe_verify_layer_noalloc (the entry point that allocates nothing: its workspace is the library's fixed
per-GPU scratch) against moe_verify_layer with a caller workspace, through the C ABI: two calls in a row
on each shape, the second with fewer tokens, bit for bit the same y; and a call beyond the scratch is
refused on the host."""
import numpy as np
import pytest
import torch

import paper_2607_12696_amd as moe
import synth

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

DEV = torch.device("cuda:0")

SHAPES = {
    "fp8": (synth.Shape("fp8", 256, 256, 16, 4, synth.FMT_FP8, 1, True), 0),
    "mxfp4_mx": (synth.Shape("mxfp4", 320, 160, 16, 4, synth.FMT_MXFP4, 0, False), 1),
    "wide": (synth.Shape("wide", 2048, 2048, 4, 1, synth.FMT_BF16, 0, False), 0),
}


def _pair(sh, dl, T, seed):
    x = synth.activations(T, sh.d, seed=seed).to(DEV)
    lg = synth.logits_scattered(T, sh.E, seed=seed + 1).to(DEV)
    r = moe.moe_route_union(lg, sh.k, sh.score)
    y_ref = moe.moe_verify_layer(x, dl, r)
    y_na = moe.moe_verify_layer_noalloc(x, dl, r)
    torch.cuda.synchronize()
    return y_ref, y_na


@pytest.mark.parametrize("name", list(SHAPES))
def test_noalloc_matches_workspace_entry(name):
    sh, act_fmt = SHAPES[name]
    print(f"noalloc shape={name}", flush=True)
    layer = synth.layer_weights(sh, seed=5)
    dl = dict(moe.pack_layer({k: (v.to(DEV) if hasattr(v, "to") else v) for k, v in layer.items()}),
              act_fmt=act_fmt)
    for T, seed in ((64, 1), (9, 2), (1, 3)):  # each call smaller than the one before
        y_ref, y_na = _pair(sh, dl, T, seed)
        assert torch.equal(y_ref, y_na), (name, T)
        assert torch.isfinite(y_na.float()).all()


def test_noalloc_full_deepseek_shape():
    sh = synth.SHAPES["ds"]
    print("noalloc full DeepSeek-V3.1 shape", flush=True)
    dl = moe.pack_layer(synth.layer_weights(sh, seed=0, device=DEV))
    for T, U, seed in ((64, 32, 1), (8, 12, 2)):
        x = synth.activations(T, sh.d, seed=seed).to(DEV)
        lg = synth.routes_to_logits(synth.routes_exact_u(T, sh.E, sh.k, U, seed=seed), sh.E, seed=seed).to(DEV)
        r = moe.moe_route_union(lg, sh.k, sh.score)
        y_ref = moe.moe_verify_layer(x, dl, r)
        y_na = moe.moe_verify_layer_noalloc(x, dl, r)
        torch.cuda.synchronize()
        assert int(r.n_unique.item()) == U
        assert torch.equal(y_ref, y_na), T
    # Beyond the scratch (T = 256 needs more than MOE_NOALLOC_SCRATCH_BYTES): refused before any launch.
    T = 256
    assert moe.moe_verify_workspace_size(dl, T, sh.k) > (64 << 20)
    x = synth.activations(T, sh.d, seed=4).to(DEV)
    r = moe.moe_route_union(synth.logits_scattered(T, sh.E, seed=4).to(DEV), sh.k, sh.score)
    y = torch.zeros_like(x)
    with pytest.raises(moe.MoeError) as e:
        moe.moe_verify_layer_noalloc(x, dl, r, y=y)
    assert e.value.status == moe.MOE_ERR_WORKSPACE and "scratch" in str(e.value)
    torch.cuda.synchronize()
    assert int(y.view(torch.int16).abs().sum().item()) == 0  # nothing was written
