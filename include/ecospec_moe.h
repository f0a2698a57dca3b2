/*
 * ecospec_moe.h -- C ABI of the MoE verification pass on MI355X (gfx950).
 *
 * The library computes, for one MoE layer, what a speculative-decoding
 * verifier must do for T draft tokens (EcoSpec, arXiv 2607.12696):
 *   router top-k          -> moe_route_topk (or moe_route_topk_hidden from x,
 *                            moe_route_topk_grouped for group-limited routing)
 *   expert union, Eq. 1   -> moe_expert_union (moe_route_union: route + union in one call)
 *   grouped SwiGLU experts streaming every activated expert's weights from
 *   HBM once, gate-weighted combine -> moe_verify_layer
 * and, on the host, the cost-aware draft-tree selection of Section 4.2
 * (Eq. 7-9, Algorithm 1) -> moe_select_tree.
 *
 * Conventions for every call:
 *   - Device pointers point to HIP device memory owned by the caller.  The
 *     library never allocates or frees memory and never synchronises; all
 *     device work is enqueued on `stream` (a hipStream_t; NULL is the null
 *     stream).  Calls are stateless and may run concurrently on different
 *     streams with different buffers.
 *   - Argument errors are detected on the host before anything is enqueued
 *     and return MOE_ERR_INVALID_ARG (or MOE_ERR_UNSUPPORTED for shapes the
 *     kernels do not handle, MOE_ERR_WORKSPACE for a short workspace).  A
 *     failed launch returns MOE_ERR_HIP.  Contents of device arrays are
 *     preconditions, not checked: e.g. topk_idx entries must lie in [0, E).
 *     A violated precondition gives unspecified results but no access
 *     outside the buffers described here.
 *   - Integers are int32, row-major, no padding.  bf16 values are stored as
 *     their 16-bit patterns.
 */
#ifndef ECOSPEC_MOE_H
#define ECOSPEC_MOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    MOE_OK = 0,
    MOE_ERR_INVALID_ARG = 1,
    MOE_ERR_UNSUPPORTED = 2,
    MOE_ERR_WORKSPACE = 3,
    MOE_ERR_HIP = 4
} moe_status_t;

/* Gate-weight rule applied to the k selected router logits l_0..l_{k-1}. */
typedef enum {
    MOE_SCORE_SOFTMAX = 0, /* w_j = exp(l_j - max) / sum_i exp(l_i - max)        */
    MOE_SCORE_SIGMOID = 1  /* w_j = sigmoid(l_j) / sum_i sigmoid(l_i)            */
} moe_score_t;

/* Expert weight storage.  Every matrix is stored out x in with the input
 * (reduction) dimension contiguous: W_gate, W_up are [d_ff][d], W_down is
 * [d][d_ff]; experts are stacked along a leading [E] dimension. */
typedef enum {
    MOE_W_BF16 = 0,          /* bf16 [E][N][K]                                               */
    MOE_W_FP8_E4M3_B128 = 1, /* OCP e4m3fn codes u8 [E][N][K], fp32 scales [E][N/128][K/128];
                                weight = e4m3fn(q[n][c]) * s[n/128][c/128]                      */
    MOE_W_MXFP4 = 2          /* OCP MXFP4: e2m1 codes packed two per byte u8 [E][N][K/2], the
                                low nibble holding the even K index; e8m0 scale codes u8
                                [E][N][K/32]; weight = e2m1 * 2^(code-127)                      */
} moe_wfmt_t;

/* Draft-selection scores (Section 4.2 and the ablation of Section 5.4). */
typedef enum {
    MOE_SEL_COST_RATIO = 0,  /* Eq. 9:  P / (DeltaCost + eps), buffer updated (Algorithm 1) */
    MOE_SEL_CONFIDENCE = 1,  /* P alone: the confidence-driven baseline                     */
    MOE_SEL_GLOBAL_COST = 2, /* Eq. 10: P / (|E_traj| + eps), buffer never consulted        */
    MOE_SEL_COST_DIFF = 3    /* P - lambda * DeltaCost                                      */
} moe_sel_mode_t;

/* Expert activation.  MOE_ACT_SWIGLU: h = silu(g) * u.  MOE_ACT_SWIGLU_OAI:
 * the clamped form of the GPT-OSS family (the GPT-OSS-120B rows of the
 * paper's tables): g = min(g, limit), u = clamp(u, -limit, limit),
 * h = g * sigmoid(alpha * g) * (u + 1). */
typedef enum {
    MOE_ACT_SWIGLU = 0,
    MOE_ACT_SWIGLU_OAI = 1
} moe_act_t;

/* Precision of the projections' inputs (x for gate/up, the activation rows h
 * for down).  MOE_ACTQ_BF16: x as given, h rounded to bf16, exact products.
 * MOE_ACTQ_MXFP8 (opt-in; MOE_W_MXFP4 weights only): both inputs quantised to
 * OCP MX FP8 and multiplied on the scaled FP4 x FP8 matrix-core instruction.
 * A row is taken in blocks of 32 consecutive elements (the OCP MX block, and
 * the K block the instruction's scales apply to).  A block's scale is 2^E,
 * E = floor(log2(max |v|)) - 8 clamped to [-127, 127] (-127 for an all-zero
 * block); each element becomes the e4m3fn value nearest to v / 2^E, ties to
 * the even code, magnitudes from 448 up saturating to 448.  The paper keeps
 * activations exact; this mode trades a few percent of y (relative to
 * max |y|) for matrix-core work without weight decoding. */
typedef enum {
    MOE_ACTQ_BF16 = 0,
    MOE_ACTQ_MXFP8 = 1
} moe_actq_t;

/* Weights of one MoE layer, in the streaming layout written by
 * moe_pack_weights; all pointers are device pointers.  The scale pointers
 * are NULL for MOE_W_BF16.  The sh_* fields describe one always-on shared
 * expert (packed the same way, E = 1) with gate weight 1 that every token
 * uses; all sh_* weight pointers NULL means no shared expert.
 * act / alpha / limit select the activation (moe_act_t; alpha and limit are
 * read for MOE_ACT_SWIGLU_OAI only, finite, limit > 0).  b_gate, b_up
 * [E][d_ff] and b_down [E][d] are optional fp32 biases of the routed experts
 * (NULL: none; 16-byte aligned): g and u get b_gate, b_up before the
 * activation and each expert output gets b_down before the gate weight.
 * The shared expert takes the activation but no biases.  act_fmt selects the
 * precision of the projection inputs (moe_actq_t; MOE_ACTQ_MXFP8 needs
 * MOE_W_MXFP4, else MOE_ERR_UNSUPPORTED).  A zero-initialised struct tail
 * (act 0, NULL biases, act_fmt 0, down_paired 0) is the plain SwiGLU layer
 * with W_down packed by moe_pack_weights; callers zero-initialise the whole
 * struct, since fields are only ever added at its end.
 * w_up == NULL means W_gate and W_up were packed together by
 * moe_pack_gate_up into w_gate (likewise sh_up == NULL with sh_gate set);
 * s_up (sh_s_up) still points to the up scales.  down_paired = 1 means
 * w_down and sh_down were packed by moe_pack_down (0: moe_pack_weights; any
 * other value is MOE_ERR_INVALID_ARG).
 * Requirements: d % 32 == 0, d_ff % 32 == 0, and for FP8 d % 128 == 0 and
 * d_ff % 128 == 0; each packed matrix below 2 GiB; 16-byte aligned pointers.
 * Other shapes return MOE_ERR_UNSUPPORTED. */
typedef struct {
    int fmt; /* moe_wfmt_t */
    int d, d_ff, E;
    const void *w_gate, *w_up, *w_down;
    const void *s_gate, *s_up, *s_down;
    const void *sh_gate, *sh_up, *sh_down;
    const void *sh_s_gate, *sh_s_up, *sh_s_down;
    int act; /* moe_act_t */
    float alpha, limit;
    const float *b_gate, *b_up, *b_down;
    int act_fmt; /* moe_actq_t */
    int down_paired;
} moe_weights_t;

/* Routing of T tokens (device pointers).  Slot s = t*k + j is the j-th
 * expert of token t.  topk_idx and topk_w are moe_route_topk's output; the
 * union and grouping arrays are moe_expert_union's output for that topk_idx.
 * moe_verify_layer reads topk_idx and topk_w and writes the union and
 * grouping arrays itself (the same values moe_expert_union gives), so they
 * need not be filled before the call. */
typedef struct {
    int T, k, E;
    const int32_t *topk_idx; /* [T][k] */
    const float *topk_w;     /* [T][k] */
    int32_t *counts;         /* [E]    */
    int32_t *union_ids;      /* [E]    */
    int32_t *n_unique;       /* [1]    */
    int32_t *offsets;        /* [E+1]  */
    int32_t *perm;           /* [T*k]  */
} moe_routing_t;

/*
 * moe_route_topk followed by moe_expert_union in one call (the two kernels,
 * enqueued back to back).  Same arguments, limits and results as the two
 * calls: logits [T][E] fp32 in; topk_idx, topk_w [T][k] and counts,
 * union_ids, n_unique, offsets, perm out.
 */
moe_status_t moe_route_union(const float *logits, int T, int E, int k, int score, int32_t *topk_idx, float *topk_w,
                             int32_t *counts, int32_t *union_ids, int32_t *n_unique, int32_t *offsets, int32_t *perm,
                             void *stream);

/*
 * Weight packing (done once, when a model is loaded).  Converts E stacked
 * N x K matrices of one tensor (W_gate or W_up: N = d_ff, K = d; W_down:
 * N = d, K = d_ff) from the interchange layout of moe_wfmt_t into the
 * streaming layout the verify kernels read:
 *   K is padded with zero codes to Kp = the next multiple of 128; each
 *   matrix is a row-major grid of blocks of 16 rows x 128 elements, block
 *   (rb, kb) at byte offset (rb*Kp/128 + kb) * B, with B = 4096 (bf16), 2048
 *   (FP8) or 1024 (MXFP4); a block is B/1024 vectors of 1 KiB and the 16
 *   bytes at offset 16*l of vector i (l = c + 16*g, c < 16, g < 4) hold
 *   the weights of row rb*16 + c from element kb*128 + 32*g + i*32*1024/B on,
 *   i.e. exactly the matrix-core operand fragment of lane l.
 *   FP8 scales keep their [N/128][K/128] layout (copied).  MXFP4 scales
 *   become [N/16][ceil(Kp/512)][64][4] bytes: in quad q of row tile rb,
 *   the 4 bytes of lane l = c + 16*g are the codes of row rb*16 + c for the
 *   32-element chunks (4q + j)*4 + g, j = 0..3 (127 in the padding).
 * w, s: device pointers in the interchange layout; w_packed, s_packed:
 * device buffers of the sizes moe_packed_size returns (s may be NULL for
 * bf16).  Requirements: N % 16 == 0, K % 32 == 0 (FP8: N, K % 128 == 0).
 */
moe_status_t moe_packed_size(int fmt, int E, int N, int K, size_t *weight_bytes, size_t *scale_bytes);

/*
 * W_gate and W_up (both E x N x K, N = d_ff, K = d) packed as one pair: the
 * streaming layout of moe_pack_weights, except that block (rb, kb) of the
 * pair is the gate block (B bytes) immediately followed by the up block, so
 * the verify kernel streams both tiles of a step as one contiguous run.
 * w_packed: 2 * weight_bytes of moe_packed_size (per pair of matrices);
 * s_gate_packed, s_up_packed: scale_bytes each (NULL for bf16), laid out as
 * moe_pack_weights lays them out.  A layer packed this way passes w_gate =
 * w_packed and w_up = NULL in moe_weights_t.  Requirements as for
 * moe_pack_weights, and 2 * weight_bytes / E below 2 GiB.
 */
moe_status_t moe_pack_gate_up(int fmt, int E, int N, int K, const void *w_gate, const void *s_gate, const void *w_up,
                              const void *s_up, void *w_packed, void *s_gate_packed, void *s_up_packed, void *stream);

/*
 * W_down (E x N x K, N = d, K = d_ff) with the two 16-row tiles that one
 * down wavefront streams interleaved: the streaming layout of
 * moe_pack_weights, except that block (2p + j, kb), j = 0, 1, sits at byte
 * offset ((p*Kp/128 + kb)*2 + j) * B, so the pair's blocks of one K step
 * form one contiguous run.  Same sizes as moe_pack_weights; the scales are
 * laid out exactly as moe_pack_weights lays them out.  A layer packed this
 * way sets down_paired = 1 in moe_weights_t (for w_down and sh_down alike).
 * Requirements as for moe_pack_weights, and N % 32 == 0
 * (MOE_ERR_UNSUPPORTED otherwise).
 */
moe_status_t moe_pack_down(int fmt, int E, int N, int K, const void *w, const void *s, void *w_packed, void *s_packed,
                           void *stream);
moe_status_t moe_pack_weights(int fmt, int E, int N, int K, const void *w, const void *s, void *w_packed,
                              void *s_packed, void *stream);

/*
 * Router top-k (Section 1: each token goes to a top-k subset of experts;
 * Table 13 gives k per model).
 *   logits   [T][E] fp32, device.
 *   topk_idx [T][k] out: for each token, the experts in routing order --
 *            larger logit first, equal logits (-0 == +0) by lower expert
 *            index, NaN after every number -- slot j holding rank j.
 *   topk_w   [T][k] out: gate weights by `score`, computed in fp32.
 * Limits: T >= 1, 1 <= E <= 1024, 1 <= k <= min(E, 64).
 */
moe_status_t moe_route_topk(const float *logits, int T, int E, int k, int score, int32_t *topk_idx,
                            float *topk_w, void *stream);

/*
 * Group-limited router top-k: the routing rule of the DeepSeek-V3 family (the
 * DeepSeek-V3.1 rows of Tables 1-13; Section 1 only fixes that each token goes
 * to a top-k subset of experts).  Per token, from the fp32 logits l:
 *   s_e = sigmoid(l_e), c_e = s_e + bias_e (bias NULL: zero);
 *   the E experts form n_group contiguous groups of E / n_group; a group's
 *   score is the sum of its two highest c (in routing order: NaN below every
 *   number, so it only counts in a group with fewer than two numbers);
 *   the topk_group groups of highest score stay eligible (ties: lower group);
 *   the k eligible experts of highest c are selected, in order (ties: lower
 *   index), slot j holding rank j;
 *   topk_w[j] = scale * s_j / sum_i s_i over the selected, in fp32.
 *   logits [T][E], bias [E], topk_idx / topk_w [T][k]: fp32 / int32 device.
 * Limits: T >= 1, 1 <= E <= 1024, 1 <= n_group <= 64, E % n_group == 0,
 * E / n_group >= 2, 1 <= topk_group <= n_group, 1 <= k <= min(64,
 * topk_group * E / n_group), scale finite; else MOE_ERR_INVALID_ARG.
 */
moe_status_t moe_route_topk_grouped(const float *logits, const float *bias, int T, int E, int k, int n_group,
                                    int topk_group, float scale, int32_t *topk_idx, float *topk_w, void *stream);

/*
 * Router from hidden states (Section 1: the router scores every expert for
 * each token, and the token goes to the top-k of them): logits = x . W_r^T,
 * then the same top-k and gate weights as moe_route_topk.
 *   x         [T][d] bf16, device, 16-byte aligned.
 *   w_router  [E][d] bf16, device, 16-byte aligned.
 *   topk_idx, topk_w: as for moe_route_topk, ranked on the logits below.
 *   logits    [T][E] fp32 out, device, or NULL: the router logits the top-k
 *             was taken on.  Each is the exact bf16 products summed in fp32;
 *             the reduction order is fixed (within 512-wide slices of d on
 *             the matrix cores, then over the slices in order), so results
 *             are deterministic, but they are not the sequential fp32 sum.
 *   workspace device scratch of moe_router_workspace_size bytes, 16-byte
 *             aligned; its contents on entry do not matter.
 * Limits: T >= 1, 1 <= E <= 1024, 1 <= k <= min(E, 64); d % 32 == 0 and x,
 * W_r each below 2 GiB (else MOE_ERR_UNSUPPORTED).  Two kernels on `stream`,
 * no allocation.
 */
moe_status_t moe_router_workspace_size(int T, int d, int E, size_t *bytes);
moe_status_t moe_route_topk_hidden(const void *x, const void *w_router, int T, int d, int E, int k, int score,
                                   int32_t *topk_idx, float *topk_w, float *logits, void *workspace,
                                   size_t workspace_bytes, void *stream);

/*
 * Expert union and grouping (Section 3, Eq. 1: the verifier must fetch the
 * union of the experts routed to by all verified tokens).
 *   topk_idx  [T][k] in (entries in [0, E)).
 *   counts    [E]    out: slots routed to each expert.
 *   union_ids [E]    out: experts with counts > 0 in ascending order, then -1.
 *   n_unique  [1]    out: U, the number of distinct experts.
 *   offsets   [E+1]  out: offsets[u] = first grouped position of union member
 *                    u; offsets[u] = T*k for u >= U.
 *   perm      [T*k]  out: slot at each grouped position; slots are ordered by
 *                    (expert, slot), i.e. a stable counting sort.
 * Limits: T >= 1, 1 <= k <= 64, 1 <= E <= 1024, T*k <= 2^24.
 */
moe_status_t moe_expert_union(const int32_t *topk_idx, int T, int k, int E, int32_t *counts,
                              int32_t *union_ids, int32_t *n_unique, int32_t *offsets, int32_t *perm,
                              void *stream);

/*
 * Bytes of device workspace moe_verify_layer needs for T tokens and top-k.
 * MOE_ERR_UNSUPPORTED when a call could hold more than 4096 token groups
 * (one per distinct expert, plus one per further 64 tokens of an expert):
 * 1025 + ceil((T*k + T) / 64) > 4096.
 */
moe_status_t moe_verify_workspace_size(const moe_weights_t *w, int T, int k, size_t *bytes);

/*
 * MoE verification layer (Section 3; Fig. 1(a): cost grows with the number
 * of distinct experts).  For every token t:
 *   y[t] = sum_j topk_w[t][j] * FFN_{topk_idx[t][j]}(x[t])  (+ FFN_shared(x[t]))
 *   FFN_e(x) = W_down[e] (silu(W_gate[e] x) * (W_up[e] x))
 * Each distinct routed expert (and the shared one) is streamed from HBM once
 * per call for up to 64 of its tokens (once per 64 tokens beyond that).
 *   x  [T][d] bf16 in, y [T][d] bf16 out (may not alias x), device.
 *   r  routing for the same T, k, E: topk_idx and topk_w in (moe_route_topk);
 *      counts, union_ids, n_unique, offsets and perm out, the union of the
 *      routed experts and the grouping of the slots by expert (Eq. 1), as
 *      moe_expert_union computes them (their contents on entry do not matter).
 *   workspace: device buffer of at least moe_verify_workspace_size bytes,
 *   256-byte aligned; its contents on entry do not matter.
 * Arithmetic: weights decoded exactly to bf16, bf16 matrix cores with fp32
 * accumulation, FP8 block scales applied to fp32 partial sums, the SwiGLU
 * intermediate rounded to bf16, y rounded to bf16.  With act_fmt =
 * MOE_ACTQ_MXFP8 (MXFP4 weights) x and the SwiGLU intermediate are quantised
 * to MX FP8 instead (moe_actq_t) and multiplied on the scaled FP4 x FP8
 * matrix cores, fp32 accumulation.  Deterministic: the same inputs give
 * bit-identical y.
 * Limits: T*d*2, (T*k + T)*d_ff*2 and (T*k + T)*d*4 bytes each below 2 GiB
 * (else MOE_ERR_UNSUPPORTED), plus those of moe_verify_workspace_size.
 */
moe_status_t moe_verify_layer(const void *x, const moe_weights_t *w, const moe_routing_t *r, void *y,
                              void *workspace, size_t workspace_bytes, void *stream);

/*
 * moe_verify_layer without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same arguments, results and limits as
 * moe_verify_layer; the workspace is a fixed array of the library of
 * MOE_NOALLOC_SCRATCH_BYTES per GPU (each GPU the library runs on holds its
 * own copy until the process ends).  A call whose moe_verify_workspace_size
 * exceeds it returns MOE_ERR_WORKSPACE (moe_last_error says how much it
 * needs), before anything is enqueued.  Nothing is allocated, freed or
 * cleared.  All calls on one GPU share the array and it keeps the last call's
 * contents: calls ordered on one stream are safe, calls that overlap on one
 * GPU (other streams, unordered host threads) race.  DeepSeek-V3.1-shaped FP8
 * layers fit up to about T = 96 tokens, Qwen3-shaped bf16 layers up to about
 * T = 128.
 */
#define MOE_NOALLOC_SCRATCH_BYTES (64u << 20)
moe_status_t moe_verify_layer_noalloc(const void *x, const moe_weights_t *w, const moe_routing_t *r, void *y,
                                      void *stream);

/*
 * moe_verify_layer with timing marks: identical work and arguments, and in
 * addition records the caller's events on `stream` around its kernels:
 *   events[0] before the gate/up expert kernel, events[1] after it (before
 *   its fix-up kernel), events[2] before the down expert kernel, events[3]
 *   after it (before the combine kernel), events[4] after the combine kernel.
 * events is an array of 5 hipEvent_t handles created by the caller (any
 * entry may be NULL to skip that mark).
 */
moe_status_t moe_verify_layer_timed(const void *x, const moe_weights_t *w, const moe_routing_t *r, void *y,
                                    void *workspace, size_t workspace_bytes, void *stream, void *const *events);

/*
 * Cost-aware draft-tree selection on the host (Section 4.2, Eq. 7-9,
 * Algorithm 1 in the appendix; Eq. 10 of Section 5.4 for the global mode).
 *   n       number of tree nodes; parent[n] (-1 for the root, parent ids
 *           smaller than the child's), P[n] cumulative path probability.
 *   pred    [n][L][K] predicted expert ids per node and layer (Eq. 4), each
 *           in [0, E).
 *   B0      initial buffer as a bitset [L][ceil(E/64)] uint64 (bit e of word
 *           e/64 set = expert e of that layer already covered), or NULL.
 *   budget  number of nodes to select (gamma); fewer if n < budget.
 *   eps     the epsilon of Eq. 9/10; lambda weights the cost in COST_DIFF.
 *   selected       [budget] out: node ids in pick order.
 *   marginal_cost  [budget] out or NULL: number of (layer, expert) pairs of
 *                  the pick's path not covered by B0 and earlier picks.
 *   n_selected     out or NULL: number of entries written.
 * The score of every unselected node is computed each round; ties go to the
 * shallower node, then to the lower id, so the result is prefix-closed.
 * Host memory only; limits: n <= 65536, L*K <= 65536, E <= 4096.
 */
moe_status_t moe_select_tree(int n, const int32_t *parent, const double *P, int L, int K,
                             const int32_t *pred, int E, const uint64_t *B0, int budget, double eps,
                             double lambda, int mode, int32_t *selected, int32_t *marginal_cost,
                             int32_t *n_selected);

/* Static description of a status code. */
const char *moe_status_string(moe_status_t status);

/* Message of the last HIP error seen by this thread (empty if none). */
const char *moe_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* ECOSPEC_MOE_H */
