"""C ABI checks that need no GPU: the library loads, exports every function the
header declares, and rejects invalid arguments on the host before any launch."""
import ctypes as C
import os
import re

import pytest

import paper_2607_12696_amd as moe

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ecospec_moe.h")

# Any non-null value: validation fails before the pointer is ever used.
FAKE = 0x10000


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(moe_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    L = moe.lib()
    names = declared_functions()
    assert set(names) == set(moe.EXPORTED)
    for n in names:
        assert hasattr(L, n), n


def test_status_strings():
    L = moe.lib()
    for s in range(5):
        assert L.moe_status_string(s)
    assert L.moe_status_string(99) == b"unknown status"


@pytest.mark.parametrize("T,E,k,score,null", [
    (0, 16, 2, 0, False), (4, 0, 1, 0, False), (4, 16, 0, 0, False), (4, 16, 17, 0, False),
    (4, 1025, 8, 0, False), (4, 128, 65, 0, False), (4, 16, 2, 2, False), (4, 16, 2, 0, True)])
def test_route_topk_rejects(T, E, k, score, null):
    L = moe.lib()
    p = 0 if null else FAKE
    assert L.moe_route_topk(p, T, E, k, score, FAKE, FAKE, None) == moe.MOE_ERR_INVALID_ARG


@pytest.mark.parametrize("T,E,k,G,TG,scale,null", [
    (0, 256, 8, 8, 4, 2.5, False), (4, 256, 0, 8, 4, 2.5, False), (4, 256, 65, 8, 4, 2.5, False),
    (4, 1025, 8, 8, 4, 2.5, False), (4, 256, 8, 0, 4, 2.5, False), (4, 256, 8, 128, 4, 2.5, False),
    (4, 250, 8, 8, 4, 2.5, False), (4, 16, 2, 16, 4, 2.5, False), (4, 256, 8, 8, 0, 2.5, False),
    (4, 256, 8, 8, 9, 2.5, False), (4, 256, 33, 8, 1, 2.5, False), (4, 256, 8, 8, 4, float("nan"), False),
    (4, 256, 8, 8, 4, float("inf"), False), (4, 256, 8, 8, 4, 2.5, True)])
def test_route_topk_grouped_rejects(T, E, k, G, TG, scale, null):
    L = moe.lib()
    p = 0 if null else FAKE
    assert L.moe_route_topk_grouped(p, None, T, E, k, G, TG, scale, FAKE, FAKE, None) == moe.MOE_ERR_INVALID_ARG


def test_router_workspace_size():
    L = moe.lib()
    n = C.c_size_t()
    assert L.moe_router_workspace_size(64, 7168, 256, C.byref(n)) == moe.MOE_OK
    assert n.value == 14 * 64 * 256 * 4  # 14 slices of 512 along d
    assert L.moe_router_workspace_size(3, 544, 33, C.byref(n)) == moe.MOE_OK and n.value == 2 * 3 * 33 * 4
    assert L.moe_router_workspace_size(4, 80, 16, C.byref(n)) == moe.MOE_ERR_UNSUPPORTED
    for T, d, E in [(0, 64, 16), (4, 0, 16), (4, 64, 0), (4, 64, 1025)]:
        assert L.moe_router_workspace_size(T, d, E, C.byref(n)) == moe.MOE_ERR_INVALID_ARG
    assert L.moe_router_workspace_size(4, 64, 16, None) == moe.MOE_ERR_INVALID_ARG


@pytest.mark.parametrize("T,d,E,k,score,status", [
    (0, 64, 16, 2, 0, moe.MOE_ERR_INVALID_ARG), (4, 64, 0, 1, 0, moe.MOE_ERR_INVALID_ARG),
    (4, 64, 16, 0, 0, moe.MOE_ERR_INVALID_ARG), (4, 64, 16, 17, 0, moe.MOE_ERR_INVALID_ARG),
    (4, 64, 1025, 8, 0, moe.MOE_ERR_INVALID_ARG), (4, 64, 128, 65, 0, moe.MOE_ERR_INVALID_ARG),
    (4, 64, 16, 2, 2, moe.MOE_ERR_INVALID_ARG), (4, 80, 16, 2, 0, moe.MOE_ERR_UNSUPPORTED),
    (4, 64, 16, 2, 0, moe.MOE_ERR_WORKSPACE)])
def test_route_topk_hidden_rejects(T, d, E, k, score, status):
    L = moe.lib()
    # workspace of 16 bytes: too small for any valid shape here
    assert L.moe_route_topk_hidden(FAKE, FAKE, T, d, E, k, score, FAKE, FAKE, None, FAKE, 16, None) == status


def test_route_topk_hidden_rejects_null_and_misaligned():
    L = moe.lib()
    big = 1 << 20
    assert L.moe_route_topk_hidden(0, FAKE, 4, 64, 16, 2, 0, FAKE, FAKE, None, FAKE, big, None) == moe.MOE_ERR_INVALID_ARG
    assert L.moe_route_topk_hidden(FAKE, FAKE, 4, 64, 16, 2, 0, FAKE, FAKE, None, 0, big, None) == moe.MOE_ERR_INVALID_ARG
    assert L.moe_route_topk_hidden(FAKE + 8, FAKE, 4, 64, 16, 2, 0, FAKE, FAKE, None, FAKE, big,
                                   None) == moe.MOE_ERR_INVALID_ARG
    assert L.moe_route_topk_hidden(FAKE, FAKE + 2, 4, 64, 16, 2, 0, FAKE, FAKE, None, FAKE, big,
                                   None) == moe.MOE_ERR_INVALID_ARG


@pytest.mark.parametrize("T,k,E", [(0, 2, 16), (4, 0, 16), (4, 65, 128), (4, 2, 0), (4, 2, 1025), (1 << 20, 32, 64)])
def test_expert_union_rejects(T, k, E):
    L = moe.lib()
    assert L.moe_expert_union(FAKE, T, k, E, FAKE, FAKE, FAKE, FAKE, FAKE, None) == moe.MOE_ERR_INVALID_ARG


@pytest.mark.parametrize("T,E,k,score,null", [
    (0, 16, 2, 0, False), (4, 0, 1, 0, False), (4, 16, 0, 0, False), (4, 16, 17, 0, False),
    (4, 1025, 8, 0, False), (4, 128, 65, 0, False), (4, 16, 2, 2, False), (4, 16, 2, 0, True)])
def test_route_union_rejects(T, E, k, score, null):
    L = moe.lib()
    p = 0 if null else FAKE
    assert L.moe_route_union(FAKE, T, E, k, score, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, p, None) == moe.MOE_ERR_INVALID_ARG


def test_expert_union_rejects_null_output():
    L = moe.lib()
    assert L.moe_expert_union(FAKE, 4, 2, 16, FAKE, 0, FAKE, FAKE, FAKE, None) == moe.MOE_ERR_INVALID_ARG


def _weights(fmt=0, d=256, d_ff=128, E=16, shared=False, scales=True):
    w = moe.moe_weights_t()
    w.fmt, w.d, w.d_ff, w.E = fmt, d, d_ff, E
    w.w_gate = w.w_up = w.w_down = FAKE
    if fmt and scales:
        w.s_gate = w.s_up = w.s_down = FAKE
    if shared:
        w.sh_gate = w.sh_up = w.sh_down = FAKE
        if fmt:
            w.sh_s_gate = w.sh_s_up = w.sh_s_down = FAKE
    return w


def _routing(T=8, k=2, E=16):
    r = moe.moe_routing_t()
    r.T, r.k, r.E = T, k, E
    for n in ("topk_idx", "topk_w", "counts", "union_ids", "n_unique", "offsets", "perm"):
        setattr(r, n, FAKE)
    return r


def _ws(w, T, k):
    n = C.c_size_t()
    st = moe.lib().moe_verify_workspace_size(C.byref(w), T, k, C.byref(n))
    return st, n.value


def test_workspace_size_formula():
    st, n = _ws(_weights(0, 256, 128, 16), 8, 2)
    assert st == moe.MOE_OK
    rows = 8 * 2
    h = rows * 128 * 2
    o = rows * 256 * 4
    # H (bf16) and O (fp32) rows at least, 256-byte granular.
    assert n >= h + o and n % 256 == 0
    st, n2 = _ws(_weights(1, 7168, 2048, 256, shared=True), 64, 8)
    assert st == moe.MOE_OK and n2 >= (64 * 8 + 64) * (2048 * 2 + 7168 * 4)


def test_workspace_rejects_too_many_token_groups():
    # 1025 + ceil((T*k + T) / 64) token groups at most 4096.
    assert _ws(_weights(), 21000, 8)[0] == moe.MOE_OK
    assert _ws(_weights(), 32768, 8)[0] == moe.MOE_ERR_UNSUPPORTED


@pytest.mark.parametrize("kw,status", [
    (dict(fmt=3), moe.MOE_ERR_INVALID_ARG),
    (dict(d=0), moe.MOE_ERR_INVALID_ARG),
    (dict(E=1025), moe.MOE_ERR_INVALID_ARG),
    (dict(d=80), moe.MOE_ERR_UNSUPPORTED),
    (dict(d_ff=48), moe.MOE_ERR_UNSUPPORTED),
    (dict(fmt=1, d=320, d_ff=128), moe.MOE_ERR_UNSUPPORTED),
    (dict(fmt=1, scales=False), moe.MOE_ERR_INVALID_ARG),
    (dict(fmt=2, scales=False), moe.MOE_ERR_INVALID_ARG),
])
def test_weights_validation(kw, status):
    assert _ws(_weights(**kw), 8, 2)[0] == status


def test_partial_shared_expert_rejected():
    w = _weights()
    w.sh_gate = FAKE
    assert _ws(w, 8, 2)[0] == moe.MOE_ERR_INVALID_ARG
    w.sh_gate, w.sh_up, w.sh_down = None, FAKE, FAKE  # sh_up alone cannot stand in for sh_gate
    assert _ws(w, 8, 2)[0] == moe.MOE_ERR_INVALID_ARG


def test_paired_gate_up_accepted():
    # w_up = NULL: W_gate and W_up packed as one pair in w_gate (and sh_up = NULL for the shared expert)
    w = _weights(fmt=1, d=256, d_ff=256, shared=True)
    w.w_up = None
    assert _ws(w, 8, 2)[0] == moe.MOE_OK
    w.sh_up = None
    assert _ws(w, 8, 2)[0] == moe.MOE_OK
    w.s_up = None  # the up scales are still needed
    assert _ws(w, 8, 2)[0] == moe.MOE_ERR_INVALID_ARG


def test_pack_gate_up_rejects():
    L = moe.lib()
    args = [1, 2, 128, 256, FAKE, FAKE, 2 * FAKE, 2 * FAKE, 3 * FAKE, 4 * FAKE, 5 * FAKE, None]
    bad = list(args); bad[6] = None  # no w_up
    assert L.moe_pack_gate_up(*bad) == moe.MOE_ERR_INVALID_ARG
    bad = list(args); bad[8] = FAKE  # packed buffer aliases w_gate
    assert L.moe_pack_gate_up(*bad) == moe.MOE_ERR_INVALID_ARG
    bad = list(args); bad[10] = bad[9]  # both scale outputs the same buffer
    assert L.moe_pack_gate_up(*bad) == moe.MOE_ERR_INVALID_ARG
    bad = list(args); bad[3] = 160  # FP8 needs K % 128 == 0
    assert L.moe_pack_gate_up(*bad) == moe.MOE_ERR_UNSUPPORTED


def test_pack_down_rejects():
    L = moe.lib()
    args = [1, 2, 256, 256, FAKE, FAKE, 2 * FAKE, 3 * FAKE, None]
    bad = list(args); bad[4] = None  # no w
    assert L.moe_pack_down(*bad) == moe.MOE_ERR_INVALID_ARG
    bad = list(args); bad[6] = FAKE  # packed buffer aliases w
    assert L.moe_pack_down(*bad) == moe.MOE_ERR_INVALID_ARG
    bad = list(args); bad[7] = None  # FP8 needs its scales
    assert L.moe_pack_down(*bad) == moe.MOE_ERR_INVALID_ARG
    bad = [0, 2, 48, 256, FAKE, None, 2 * FAKE, None, None]  # 3 row tiles: no whole pairs
    assert L.moe_pack_down(*bad) == moe.MOE_ERR_UNSUPPORTED


def test_down_paired_flag_validated():
    w = _weights()
    for v, st in ((0, moe.MOE_OK), (1, moe.MOE_OK), (2, moe.MOE_ERR_INVALID_ARG), (-1, moe.MOE_ERR_INVALID_ARG)):
        w.down_paired = v
        assert _ws(w, 8, 2)[0] == st


def test_verify_layer_rejects_outputs_past_2gib():
    # O (fp32 rows of T*k + T slots x d) is addressed through a 32-bit buffer range: DS shape with T = 8400
    # gives 75600 x 7168 x 4 bytes = 2.17 GB; every other limit (groups, H, x) still holds.
    L = moe.lib()
    w = _weights(1, 7168, 2048, 256, shared=True)
    T = 8400
    st, need = _ws(w, T, 8)
    assert st == moe.MOE_OK
    r = _routing(T, 8, 256)
    assert L.moe_verify_layer(FAKE, C.byref(w), C.byref(r), 2 * FAKE, 4 * FAKE, need, None) == moe.MOE_ERR_UNSUPPORTED


def test_misaligned_weight_rejected():
    w = _weights()
    w.w_up = FAKE + 8
    assert _ws(w, 8, 2)[0] == moe.MOE_ERR_INVALID_ARG


def test_verify_layer_rejects_before_launch():
    L = moe.lib()
    w, r = _weights(), _routing()
    st, need = _ws(w, 8, 2)
    assert st == moe.MOE_OK
    args = lambda x=FAKE, y=2 * FAKE, ws=4 * FAKE, nb=need: (x, C.byref(w), C.byref(r), y, ws, nb, None)
    assert L.moe_verify_layer(*args(nb=need - 1)) == moe.MOE_ERR_WORKSPACE
    assert L.moe_verify_layer(*args(x=0)) == moe.MOE_ERR_INVALID_ARG
    assert L.moe_verify_layer(*args(y=FAKE)) == moe.MOE_ERR_INVALID_ARG      # y aliases x
    assert L.moe_verify_layer(*args(ws=4 * FAKE + 16)) == moe.MOE_ERR_INVALID_ARG  # workspace not 256-aligned
    r.E = 32
    assert L.moe_verify_layer(*args()) == moe.MOE_ERR_INVALID_ARG
    r.E, r.k = 16, 17
    assert L.moe_verify_layer(*args()) == moe.MOE_ERR_INVALID_ARG
    r.k, r.perm = 2, None
    assert L.moe_verify_layer(*args()) == moe.MOE_ERR_INVALID_ARG


@pytest.mark.parametrize("field,value", [
    ("act", 2), ("act", -1),
    ("alpha", float("nan")), ("limit", float("inf")), ("limit", 0.0), ("limit", -1.0)])
def test_activation_fields_validated(field, value):
    w = _weights()
    w.act, w.alpha, w.limit = moe.MOE_ACT_SWIGLU_OAI, 1.702, 7.0
    assert _ws(w, 8, 2)[0] == moe.MOE_OK
    setattr(w, field, value)
    assert _ws(w, 8, 2)[0] == moe.MOE_ERR_INVALID_ARG


def test_plain_activation_ignores_alpha_and_limit():
    w = _weights()
    w.act, w.alpha, w.limit = moe.MOE_ACT_SWIGLU, float("nan"), 0.0
    assert _ws(w, 8, 2)[0] == moe.MOE_OK


def test_mx_activation_format_validated():
    # act_fmt: 0 or 1; MX FP8 activations only with MXFP4 weights; they need room for the quantised rows.
    w = _weights(fmt=2, d=320, d_ff=160)
    st0, n0 = _ws(w, 64, 2)
    assert st0 == moe.MOE_OK
    w.act_fmt = moe.MOE_ACTQ_MXFP8
    st1, n1 = _ws(w, 64, 2)
    assert st1 == moe.MOE_OK
    # x: 64 rows x 384 codes + 12 scales; H: 128 rows x 256 codes + 8 scales (each region 256-byte aligned).
    assert n1 - n0 == 64 * 384 + 768 + 128 * 256 + 1024
    for bad in (2, -1):
        w.act_fmt = bad
        assert _ws(w, 64, 2)[0] == moe.MOE_ERR_INVALID_ARG
    for fmt in (0, 1):
        w = _weights(fmt=fmt, d=256, d_ff=128)
        w.act_fmt = moe.MOE_ACTQ_MXFP8
        assert _ws(w, 8, 2)[0] == moe.MOE_ERR_UNSUPPORTED


@pytest.mark.parametrize("name", ["b_gate", "b_up", "b_down"])
def test_misaligned_bias_rejected(name):
    w = _weights()
    setattr(w, name, FAKE)
    assert _ws(w, 8, 2)[0] == moe.MOE_OK
    setattr(w, name, FAKE + 4)
    assert _ws(w, 8, 2)[0] == moe.MOE_ERR_INVALID_ARG


@pytest.mark.parametrize("down_bias", [False, True])
def test_verify_needs_topk_idx(down_bias):
    # The combine reads each slot's expert (to skip slots outside [0, E) and to pick the down bias).
    L = moe.lib()
    w, r = _weights(), _routing()
    if down_bias:
        w.b_down = FAKE
    st, need = _ws(w, 8, 2)
    assert st == moe.MOE_OK
    r.topk_idx = None
    assert L.moe_verify_layer(FAKE, C.byref(w), C.byref(r), 2 * FAKE, 4 * FAKE, need, None) == moe.MOE_ERR_INVALID_ARG


def test_down_matrix_over_2GiB_rejected():
    # W_down [d][d_ff] is bounded like W_gate / W_up: with d_ff padded to 128 it can be the larger matrix.
    w = _weights()
    w.fmt, w.d, w.d_ff = 0, 32, 32
    assert _ws(w, 8, 2)[0] == moe.MOE_OK
    w.d, w.d_ff = 262144 + 32, 4064  # W_down 262176 x 4096 bf16 >= 2 GiB, W_gate 4064 x 262176 < 2 GiB (unpaired)
    w.w_up = FAKE
    assert _ws(w, 8, 2)[0] == moe.MOE_ERR_UNSUPPORTED


@pytest.mark.parametrize("fmt,E,N,K,status", [
    (3, 1, 16, 32, moe.MOE_ERR_INVALID_ARG), (0, 0, 16, 32, moe.MOE_ERR_INVALID_ARG),
    (0, 1, 24, 32, moe.MOE_ERR_UNSUPPORTED), (0, 1, 16, 48, moe.MOE_ERR_UNSUPPORTED),
    (1, 1, 64, 128, moe.MOE_ERR_UNSUPPORTED), (1, 1, 128, 160, moe.MOE_ERR_UNSUPPORTED)])
def test_pack_validation(fmt, E, N, K, status):
    wb, sb = C.c_size_t(), C.c_size_t()
    assert moe.lib().moe_packed_size(fmt, E, N, K, C.byref(wb), C.byref(sb)) == status
    assert moe.lib().moe_pack_weights(fmt, E, N, K, FAKE, FAKE, 2 * FAKE, 3 * FAKE, None) == status


def test_packed_sizes():
    assert moe.moe_packed_size(1, 2, 2048, 7168) == (2 * 2048 * 7168, 2 * 16 * 56 * 4)
    assert moe.moe_packed_size(0, 1, 32, 96) == (32 * 128 * 2, 0)
    # MXFP4 scales: 23 blocks of 128 -> 6 quads of 4 blocks, 16 bytes per row and quad
    assert moe.moe_packed_size(2, 1, 2880, 2880) == (2880 * 2944 // 2, 2880 * 6 * 16)


def test_binding_refuses_host_tensors():
    torch = pytest.importorskip("torch")
    with pytest.raises(ValueError):
        moe.moe_route_topk(torch.zeros(2, 16), 2, 0)


def test_workspace_scales_with_tokens():
    # Partial-sum slots hold only the live 16-token blocks and one pair per workgroup of the grid, so a
    # one-token call needs far less than a 64-token one (DeepSeek-V3.1 shape: under 16 MiB at T = 1).
    w = _weights(1, 7168, 2048, 256, shared=True)
    st1, n1 = _ws(w, 1, 8)
    st64, n64 = _ws(w, 64, 8)
    assert st1 == st64 == moe.MOE_OK
    assert n1 < 16 << 20 and n64 < 64 << 20 and n1 < n64 / 4
