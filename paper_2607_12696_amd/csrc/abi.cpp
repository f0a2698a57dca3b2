// C ABI of the verification pass: argument validation, workspace carve-up and
// launch sequencing.  No allocation, no synchronisation.
#include "ecospec_moe.h"

#include <hip/hip_runtime_api.h>
#include <stdio.h>
#include <string.h>

#include "launch.hpp"
#include <math.h>

namespace {

thread_local char g_last_error[256] = "";

moe_status_t from_hip(hipError_t e)
{
    if (e == hipSuccess) return MOE_OK;
    snprintf(g_last_error, sizeof g_last_error, "%s", hipGetErrorString(e));
    return MOE_ERR_HIP;
}

bool aligned(const void *p, size_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

constexpr int kMaxE = 1024;
constexpr int kMaxK = 64;
constexpr long kMaxSlots = 1L << 24;

moe_status_t check_weights(const moe_weights_t *w)
{
    if (!w) return MOE_ERR_INVALID_ARG;
    if (w->fmt < MOE_W_BF16 || w->fmt > MOE_W_MXFP4) return MOE_ERR_INVALID_ARG;
    if (w->d < 1 || w->d_ff < 1 || w->E < 1 || w->E > kMaxE) return MOE_ERR_INVALID_ARG;
    // w_up == NULL: W_gate and W_up packed as one pair in w_gate (moe_pack_gate_up); the same for sh_up.
    if (!w->w_gate || !w->w_down) return MOE_ERR_INVALID_ARG;
    if (w->fmt != MOE_W_BF16 && (!w->s_gate || !w->s_up || !w->s_down)) return MOE_ERR_INVALID_ARG;
    const bool sh = w->sh_gate != nullptr || w->sh_up != nullptr || w->sh_down != nullptr;
    if (sh && (!w->sh_gate || !w->sh_down)) return MOE_ERR_INVALID_ARG;
    if (sh && w->fmt != MOE_W_BF16 && (!w->sh_s_gate || !w->sh_s_up || !w->sh_s_down)) return MOE_ERR_INVALID_ARG;
    // Tile shapes of the kernels: 16-row gate/up bands, 32-row down bands,
    // 32-wide K chunks; FP8 needs whole 128x128 scale blocks.
    if (w->d % 32 || w->d_ff % 32) return MOE_ERR_UNSUPPORTED;
    if (w->fmt == MOE_W_FP8_E4M3_B128 && (w->d % 128 || w->d_ff % 128)) return MOE_ERR_UNSUPPORTED;
    // Every packed matrix is addressed through a 32-bit buffer range below 2^31 bytes.
    const size_t pair = (!w->w_up || (sh && !w->sh_up)) ? 2 : 1;
    if (ecospec::packed_matrix_bytes(w->fmt, w->d_ff, w->d) * pair >= (1UL << 31)) return MOE_ERR_UNSUPPORTED;
    if (ecospec::packed_matrix_bytes(w->fmt, w->d, w->d_ff) >= (1UL << 31)) return MOE_ERR_UNSUPPORTED;
    const void *mats[] = {w->w_gate, w->w_up, w->w_down, w->sh_gate, w->sh_up, w->sh_down};
    for (const void *p : mats)
        if (p && !aligned(p, 16)) return MOE_ERR_INVALID_ARG;
    if (w->fmt == MOE_W_FP8_E4M3_B128) {
        const void *sc[] = {w->s_gate, w->s_up, w->s_down, w->sh_s_gate, w->sh_s_up, w->sh_s_down};
        for (const void *p : sc)
            if (p && !aligned(p, 4)) return MOE_ERR_INVALID_ARG;
    }
    if (w->act != MOE_ACT_SWIGLU && w->act != MOE_ACT_SWIGLU_OAI) return MOE_ERR_INVALID_ARG;
    if (w->act == MOE_ACT_SWIGLU_OAI && (!isfinite(w->alpha) || !isfinite(w->limit) || !(w->limit > 0.f)))
        return MOE_ERR_INVALID_ARG;
    const void *bs[] = {w->b_gate, w->b_up, w->b_down};
    for (const void *p : bs)
        if (p && !aligned(p, 16)) return MOE_ERR_INVALID_ARG;
    if (w->act_fmt != MOE_ACTQ_BF16 && w->act_fmt != MOE_ACTQ_MXFP8) return MOE_ERR_INVALID_ARG;
    if (w->act_fmt == MOE_ACTQ_MXFP8 && w->fmt != MOE_W_MXFP4) return MOE_ERR_UNSUPPORTED;
    if (w->down_paired != 0 && w->down_paired != 1) return MOE_ERR_INVALID_ARG;
    return MOE_OK;
}

}  // namespace

namespace ecospec {

void set_last_error(const char *msg) { snprintf(g_last_error, sizeof g_last_error, "%s", msg); }

}  // namespace ecospec

extern "C" {

const char *moe_status_string(moe_status_t s)
{
    switch (s) {
    case MOE_OK: return "ok";
    case MOE_ERR_INVALID_ARG: return "invalid argument";
    case MOE_ERR_UNSUPPORTED: return "unsupported shape or format";
    case MOE_ERR_WORKSPACE: return "workspace too small";
    case MOE_ERR_HIP: return "HIP error";
    }
    return "unknown status";
}

const char *moe_last_error(void) { return g_last_error; }

moe_status_t moe_route_topk(const float *logits, int T, int E, int k, int score, int32_t *topk_idx, float *topk_w,
                            void *stream)
{
    if (!logits || !topk_idx || !topk_w) return MOE_ERR_INVALID_ARG;
    if (T < 1 || E < 1 || E > kMaxE || k < 1 || k > E || k > kMaxK) return MOE_ERR_INVALID_ARG;
    if ((long)T * E > (1L << 31) - 1 || (long)T * k > kMaxSlots) return MOE_ERR_INVALID_ARG;
    if (score != MOE_SCORE_SOFTMAX && score != MOE_SCORE_SIGMOID) return MOE_ERR_INVALID_ARG;
    return from_hip(
        ecospec::launch_route_topk(logits, 0, T, E, k, score, topk_idx, topk_w, nullptr, (hipStream_t)stream));
}

moe_status_t moe_route_topk_grouped(const float *logits, const float *bias, int T, int E, int k, int n_group,
                                    int topk_group, float scale, int32_t *topk_idx, float *topk_w, void *stream)
{
    if (!logits || !topk_idx || !topk_w) return MOE_ERR_INVALID_ARG;
    if (T < 1 || E < 1 || E > kMaxE || k < 1 || k > kMaxK) return MOE_ERR_INVALID_ARG;
    if ((long)T * E > (1L << 31) - 1 || (long)T * k > kMaxSlots) return MOE_ERR_INVALID_ARG;
    if (n_group < 1 || n_group > 64 || E % n_group || E / n_group < 2) return MOE_ERR_INVALID_ARG;
    if (topk_group < 1 || topk_group > n_group || k > topk_group * (E / n_group)) return MOE_ERR_INVALID_ARG;
    if (!(scale == scale) || scale == INFINITY || scale == -INFINITY) return MOE_ERR_INVALID_ARG;
    return from_hip(ecospec::launch_route_grouped(logits, bias, T, E, k, n_group, topk_group, scale, topk_idx,
                                                  topk_w, (hipStream_t)stream));
}

moe_status_t moe_router_workspace_size(int T, int d, int E, size_t *bytes)
{
    if (!bytes || T < 1 || d < 1 || E < 1 || E > kMaxE) return MOE_ERR_INVALID_ARG;
    if (d % 32) return MOE_ERR_UNSUPPORTED;
    *bytes = (size_t)ecospec::router_slices(d) * T * E * 4;
    return MOE_OK;
}

moe_status_t moe_route_topk_hidden(const void *x, const void *w_router, int T, int d, int E, int k, int score,
                                   int32_t *topk_idx, float *topk_w, float *logits, void *workspace,
                                   size_t workspace_bytes, void *stream)
{
    if (!x || !w_router || !topk_idx || !topk_w || !workspace) return MOE_ERR_INVALID_ARG;
    if (T < 1 || E < 1 || E > kMaxE || k < 1 || k > E || k > kMaxK || d < 1) return MOE_ERR_INVALID_ARG;
    if ((long)T * k > kMaxSlots || (long)T * E > (1L << 31) - 1) return MOE_ERR_INVALID_ARG;
    if (score != MOE_SCORE_SOFTMAX && score != MOE_SCORE_SIGMOID) return MOE_ERR_INVALID_ARG;
    if (!aligned(x, 16) || !aligned(w_router, 16) || !aligned(workspace, 16)) return MOE_ERR_INVALID_ARG;
    if (d % 32) return MOE_ERR_UNSUPPORTED;
    if ((size_t)T * d * 2 >= (1u << 31) || (size_t)E * d * 2 >= (1u << 31)) return MOE_ERR_UNSUPPORTED;
    const size_t need = (size_t)ecospec::router_slices(d) * T * E * 4;
    if (workspace_bytes < need) return MOE_ERR_WORKSPACE;
    float *partial = static_cast<float *>(workspace);
    hipError_t err = ecospec::launch_router_gemm(static_cast<const uint16_t *>(x),
                                                 static_cast<const uint16_t *>(w_router), T, d, E, partial,
                                                 (hipStream_t)stream);
    if (err != hipSuccess) return from_hip(err);
    return from_hip(ecospec::launch_route_topk(partial, ecospec::router_slices(d), T, E, k, score, topk_idx, topk_w,
                                               logits, (hipStream_t)stream));
}

moe_status_t moe_expert_union(const int32_t *topk_idx, int T, int k, int E, int32_t *counts, int32_t *union_ids,
                              int32_t *n_unique, int32_t *offsets, int32_t *perm, void *stream)
{
    if (!topk_idx || !counts || !union_ids || !n_unique || !offsets || !perm) return MOE_ERR_INVALID_ARG;
    if (T < 1 || k < 1 || k > kMaxK || E < 1 || E > kMaxE || (long)T * k > kMaxSlots) return MOE_ERR_INVALID_ARG;
    return from_hip(ecospec::launch_expert_union(topk_idx, T, k, E, counts, union_ids, n_unique, offsets, perm,
                                                 (hipStream_t)stream));
}

moe_status_t moe_route_union(const float *logits, int T, int E, int k, int score, int32_t *topk_idx, float *topk_w,
                             int32_t *counts, int32_t *union_ids, int32_t *n_unique, int32_t *offsets, int32_t *perm,
                             void *stream)
{
    if (!logits || !topk_idx || !topk_w || !counts || !union_ids || !n_unique || !offsets || !perm)
        return MOE_ERR_INVALID_ARG;
    if (T < 1 || E < 1 || E > kMaxE || k < 1 || k > E || k > kMaxK) return MOE_ERR_INVALID_ARG;
    if ((long)T * E > (1L << 31) - 1 || (long)T * k > kMaxSlots) return MOE_ERR_INVALID_ARG;
    if (score != MOE_SCORE_SOFTMAX && score != MOE_SCORE_SIGMOID) return MOE_ERR_INVALID_ARG;
    hipStream_t st = (hipStream_t)stream;
    hipError_t err = ecospec::launch_route_topk(logits, 0, T, E, k, score, topk_idx, topk_w, nullptr, st);
    if (err != hipSuccess) return from_hip(err);
    return from_hip(ecospec::launch_expert_union(topk_idx, T, k, E, counts, union_ids, n_unique, offsets, perm, st));
}

moe_status_t moe_verify_workspace_size(const moe_weights_t *w, int T, int k, size_t *bytes)
{
    if (!bytes) return MOE_ERR_INVALID_ARG;
    const moe_status_t st = check_weights(w);
    if (st != MOE_OK) return st;
    if (T < 1 || k < 1 || k > kMaxK || k > w->E || (long)T * k > kMaxSlots) return MOE_ERR_INVALID_ARG;
    const ecospec::VerifyWorkspace ws =
        ecospec::verify_workspace(w->d, w->d_ff, T, k, w->sh_gate != nullptr, w->act_fmt == MOE_ACTQ_MXFP8,
                                  ecospec::verify_workers());
    if (ws.plan_cap > ecospec::kMaxGroups) return MOE_ERR_UNSUPPORTED;
    *bytes = ws.total;
    return MOE_OK;
}

}  // extern "C"

namespace ecospec {

moe_status_t verify_impl(const void *x, const moe_weights_t *w, const moe_routing_t *r, void *y, void *workspace,
                         size_t workspace_bytes, void *stream, void *const *events)
{
    moe_status_t st = check_weights(w);
    if (st != MOE_OK) return st;
    if (!x || !y || !r || !workspace || x == y) return MOE_ERR_INVALID_ARG;
    if (!aligned(x, 16) || !aligned(y, 16) || !aligned(workspace, 256)) return MOE_ERR_INVALID_ARG;
    if (r->T < 1 || r->k < 1 || r->k > kMaxK || r->k > w->E || r->E != w->E || (long)r->T * r->k > kMaxSlots)
        return MOE_ERR_INVALID_ARG;
    if (!r->topk_idx || !r->topk_w || !r->counts || !r->union_ids || !r->n_unique || !r->offsets || !r->perm)
        return MOE_ERR_INVALID_ARG;
    const bool shared = w->sh_gate != nullptr;
    const ecospec::VerifyWorkspace ws =
        ecospec::verify_workspace(w->d, w->d_ff, r->T, r->k, shared, w->act_fmt == MOE_ACTQ_MXFP8,
                                  ecospec::verify_workers());
    if (ws.plan_cap > ecospec::kMaxGroups) return MOE_ERR_UNSUPPORTED;
    if (workspace_bytes < ws.total) return MOE_ERR_WORKSPACE;
    const long rows = (long)r->T * r->k + (shared ? r->T : 0);
    // x, H and O are addressed through 32-bit buffer ranges.
    if ((long)r->T * w->d * 2 >= (1L << 31) || rows * w->d_ff * 2 >= (1L << 31) || rows * w->d * 4 >= (1L << 31))
        return MOE_ERR_UNSUPPORTED;

    ecospec::VerifyArgs a{};
    a.fmt = w->fmt;
    a.d = w->d;
    a.d_ff = w->d_ff;
    a.E = w->E;
    a.T = r->T;
    a.k = r->k;
    a.w_gate = static_cast<const uint8_t *>(w->w_gate);
    a.w_up = static_cast<const uint8_t *>(w->w_up);
    a.gu_pair = w->w_up == nullptr;
    a.sh_gu_pair = w->sh_gate != nullptr && w->sh_up == nullptr;
    a.w_down = static_cast<const uint8_t *>(w->w_down);
    a.down_pair = w->down_paired == 1;
    a.s_gate = w->s_gate;
    a.s_up = w->s_up;
    a.s_down = w->s_down;
    a.sh_gate = static_cast<const uint8_t *>(w->sh_gate);
    a.sh_up = static_cast<const uint8_t *>(w->sh_up);
    a.sh_down = static_cast<const uint8_t *>(w->sh_down);
    a.sh_s_gate = w->sh_s_gate;
    a.sh_s_up = w->sh_s_up;
    a.sh_s_down = w->sh_s_down;
    a.topk_w = r->topk_w;
    a.topk_idx = r->topk_idx;
    a.act = w->act;
    a.alpha = w->alpha;
    a.limit = w->limit;
    a.b_gate = w->b_gate;
    a.b_up = w->b_up;
    a.b_down = w->b_down;
    a.act_fmt = w->act_fmt;
    a.counts = r->counts;
    a.union_ids = r->union_ids;
    a.n_unique = r->n_unique;
    a.offsets = r->offsets;
    a.perm = r->perm;
    a.x = static_cast<const uint16_t *>(x);
    a.y = static_cast<uint16_t *>(y);
    hipEvent_t ev[ecospec::kTimingMarks] = {};
    if (events)
        for (int i = 0; i < ecospec::kTimingMarks; ++i) ev[i] = (hipEvent_t)events[i];
    return from_hip(ecospec::launch_verify(a, workspace, ws, (hipStream_t)stream, events ? ev : nullptr));
}

}  // namespace ecospec

extern "C" {

moe_status_t moe_verify_layer(const void *x, const moe_weights_t *w, const moe_routing_t *r, void *y,
                              void *workspace, size_t workspace_bytes, void *stream)
{
    return ecospec::verify_impl(x, w, r, y, workspace, workspace_bytes, stream, nullptr);
}

moe_status_t moe_verify_layer_timed(const void *x, const moe_weights_t *w, const moe_routing_t *r, void *y,
                                    void *workspace, size_t workspace_bytes, void *stream, void *const *events)
{
    return ecospec::verify_impl(x, w, r, y, workspace, workspace_bytes, stream, events);
}

static moe_status_t check_pack(int fmt, int E, int N, int K)
{
    if (fmt < MOE_W_BF16 || fmt > MOE_W_MXFP4 || E < 1 || N < 16 || K < 32) return MOE_ERR_INVALID_ARG;
    if (N % 16 || K % 32) return MOE_ERR_UNSUPPORTED;
    if (fmt == MOE_W_FP8_E4M3_B128 && (N % 128 || K % 128)) return MOE_ERR_UNSUPPORTED;
    if (ecospec::packed_matrix_bytes(fmt, N, K) >= (1UL << 31)) return MOE_ERR_UNSUPPORTED;
    return MOE_OK;
}

moe_status_t moe_packed_size(int fmt, int E, int N, int K, size_t *weight_bytes, size_t *scale_bytes)
{
    if (!weight_bytes || !scale_bytes) return MOE_ERR_INVALID_ARG;
    const moe_status_t st = check_pack(fmt, E, N, K);
    if (st != MOE_OK) return st;
    *weight_bytes = (size_t)E * ecospec::packed_matrix_bytes(fmt, N, K);
    *scale_bytes = (size_t)E * ecospec::packed_scale_bytes(fmt, N, K);
    return MOE_OK;
}

moe_status_t moe_pack_weights(int fmt, int E, int N, int K, const void *w, const void *s, void *w_packed,
                              void *s_packed, void *stream)
{
    const moe_status_t st = check_pack(fmt, E, N, K);
    if (st != MOE_OK) return st;
    if (!w || !w_packed || w == w_packed || !aligned(w, 16) || !aligned(w_packed, 16)) return MOE_ERR_INVALID_ARG;
    if (fmt != MOE_W_BF16 && (!s || !s_packed || s == s_packed)) return MOE_ERR_INVALID_ARG;
    return from_hip(ecospec::launch_pack(fmt, E, N, K, w, s, w_packed, s_packed, (hipStream_t)stream));
}

moe_status_t moe_pack_down(int fmt, int E, int N, int K, const void *w, const void *s, void *w_packed, void *s_packed,
                           void *stream)
{
    const moe_status_t st = check_pack(fmt, E, N, K);
    if (st != MOE_OK) return st;
    if (N % 32) return MOE_ERR_UNSUPPORTED;  // whole pairs of 16-row tiles
    if (!w || !w_packed || w == w_packed || !aligned(w, 16) || !aligned(w_packed, 16)) return MOE_ERR_INVALID_ARG;
    if (fmt != MOE_W_BF16 && (!s || !s_packed || s == s_packed)) return MOE_ERR_INVALID_ARG;
    return from_hip(ecospec::launch_pack_down(fmt, E, N, K, w, s, w_packed, s_packed, (hipStream_t)stream));
}

moe_status_t moe_pack_gate_up(int fmt, int E, int N, int K, const void *w_gate, const void *s_gate, const void *w_up,
                              const void *s_up, void *w_packed, void *s_gate_packed, void *s_up_packed, void *stream)
{
    const moe_status_t st = check_pack(fmt, E, N, K);
    if (st != MOE_OK) return st;
    if (ecospec::packed_matrix_bytes(fmt, N, K) * 2 >= (1UL << 31)) return MOE_ERR_UNSUPPORTED;
    if (!w_gate || !w_up || !w_packed || w_gate == w_packed || w_up == w_packed) return MOE_ERR_INVALID_ARG;
    if (!aligned(w_gate, 16) || !aligned(w_up, 16) || !aligned(w_packed, 16)) return MOE_ERR_INVALID_ARG;
    if (fmt != MOE_W_BF16 && (!s_gate || !s_up || !s_gate_packed || !s_up_packed || s_gate_packed == s_up_packed))
        return MOE_ERR_INVALID_ARG;
    return from_hip(ecospec::launch_pack_gate_up(fmt, E, N, K, w_gate, s_gate, w_up, s_up, w_packed, s_gate_packed,
                                                 s_up_packed, (hipStream_t)stream));
}

}  // extern "C"
