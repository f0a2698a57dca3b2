/*
 * CPU oracle for the MoE verification pass -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow, obviously correct fp64 reference of what the verification
 * pass over T draft tokens computes in one MoE layer.  Only the test suite,
 * the smoke check and the benchmark's CPU-baseline leg use it; the product
 * library never links or calls it, and it includes nothing from the product
 * sources (nor they from here).
 *
 * Paper: "Less Experts, Faster Decoding: Cost-Aware Speculative Decoding for
 * Mixture-of-Experts" (EcoSpec).
 *   - Section 1 (Introduction): a router sends each token to a top-k subset
 *     of the layer's experts.
 *   - Section 3, Eq. 1: the experts a verification pass must read at layer l
 *     are the union, over the verified tokens, of each token's routed set.
 *   - Fig. 1(c) and Section 3: every extra expert costs its full weight bytes
 *     (44.04 MB for a DeepSeek-V3.1 FP8 expert).
 * The paper never writes the layer formula out.  The readings used here: the
 * expert is a SwiGLU FFN, y_t = sum_j w_tj * W_down(silu(W_gate x) * (W_up x))
 * (+ an always-on shared expert with weight 1 for DeepSeek-V3.1); top-k is taken
 * on the raw fp32 router logits ordered by (value desc, index asc), NaN last;
 * weights are a softmax over the k selected logits or sigmoid(l)/sum sigmoid.
 *
 * Storage formats (input formats, decoded exactly here):
 *   0 bf16        W[n][c] = bf16 bits, K (=c) contiguous
 *   1 FP8 e4m3fn  W[n][c] = e4m3fn(q[n][c]) * s[n/128][c/128]   (OCP FP8, bias 7, max 448)
 *   2 MXFP4       W[n][c] = e2m1(nibble) * 2^(e8m0[n][c/32]-127) (OCP MX; two codes per byte,
 *                 low nibble = even c)
 *
 * Optional MX activation mode (act_fmt 1; not in the paper, an opt-in numeric
 * mode): the inputs of both projections are quantised to OCP MX FP8 first (see
 * orc_mx_quant below).
 *
 * Parity status: route, union, decode, the MX activation quantiser and the
 * verify layer are pinned by the tests under tests/ (brute force, closed forms,
 * library cross-checks and the paper's 44.04 MB byte count).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------ decode */

double orc_bf16(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
}

/* OCP FP8 E4M3 ("fn": no infinities; S.1111.111 is NaN). */
double orc_e4m3fn(uint8_t c)
{
    int s = c >> 7, e = (c >> 3) & 15, m = c & 7;
    double v;
    if (e == 15 && m == 7)
        return NAN;
    if (e == 0)
        v = ldexp((double)m / 8.0, -6);            /* subnormal: 0.m * 2^(1-7) */
    else
        v = ldexp(1.0 + (double)m / 8.0, e - 7);   /* normal: 1.m * 2^(e-7) */
    return s ? -v : v;
}

/* OCP MX E2M1 (FP4): S.EE.M, bias 1. */
double orc_e2m1(uint8_t nib)
{
    int s = (nib >> 3) & 1, e = (nib >> 1) & 3, m = nib & 1;
    double v = (e == 0) ? 0.5 * m : ldexp(1.0 + 0.5 * m, e - 1);
    return s ? -v : v;
}

/* OCP MX E8M0 shared scale: 2^(code-127), 0xFF is NaN. */
double orc_e8m0(uint8_t c)
{
    return c == 255 ? NAN : ldexp(1.0, (int)c - 127);
}

/* Writes the decoded value of every code of a format (kind 0: e4m3fn, 256
 * codes; 1: e2m1, 16 codes; 2: e8m0, 256 codes; 3: bf16, 65536 codes). */
int orc_decode_table(int kind, double *out)
{
    int i;
    switch (kind) {
    case 0: for (i = 0; i < 256; i++) out[i] = orc_e4m3fn((uint8_t)i); return 256;
    case 1: for (i = 0; i < 16; i++) out[i] = orc_e2m1((uint8_t)i); return 16;
    case 2: for (i = 0; i < 256; i++) out[i] = orc_e8m0((uint8_t)i); return 256;
    case 3: for (i = 0; i < 65536; i++) out[i] = orc_bf16((uint16_t)i); return 65536;
    default: return -1;
    }
}

/* Decoded element (n, c) of one N x K weight matrix stored in format fmt. */
static double weight_at(int fmt, const void *w, const void *s, int N, int K, int n, int c)
{
    (void)N;
    switch (fmt) {
    case 0:
        return orc_bf16(((const uint16_t *)w)[(size_t)n * K + c]);
    case 1:
        return orc_e4m3fn(((const uint8_t *)w)[(size_t)n * K + c]) *
               (double)((const float *)s)[(size_t)(n / 128) * (K / 128) + c / 128];
    case 2: {
        uint8_t byte = ((const uint8_t *)w)[(size_t)n * (K / 2) + c / 2];
        uint8_t nib = (c % 2 == 0) ? (byte & 15) : (byte >> 4);
        return orc_e2m1(nib) * orc_e8m0(((const uint8_t *)s)[(size_t)n * (K / 32) + c / 32]);
    }
    }
    return NAN;
}

/* Decoded element, exported for the tests. */
double orc_weight_at(int fmt, const void *w, const void *s, int N, int K, int n, int c)
{
    return weight_at(fmt, w, s, N, K, n, c);
}

/* ------------------------------------------------------------------ routing */

/* Does (a, ia) come before (b, ib) in the routing order?  Larger logit first,
 * -0 equal to +0, NaN after every number, equal values by lower index. */
static int before(float a, int ia, float b, int ib)
{
    int na = isnan(a), nb = isnan(b);
    if (na || nb)
        return (na && nb) ? ia < ib : nb;
    if (a != b)
        return a > b;
    return ia < ib;
}

static const float *g_sort_row;
static int cmp_experts(const void *pa, const void *pb)
{
    int a = *(const int *)pa, b = *(const int *)pb;
    if (a == b) return 0;
    return before(g_sort_row[a], a, g_sort_row[b], b) ? -1 : 1;
}

/* Router top-k (Section 1; Table 13 gives k per model).  For each token the E
 * experts are sorted in routing order and the first k kept, slot j = rank j.
 * score 0: w_j = exp(l_j - m) / sum_i exp(l_i - m) over the k selected logits,
 * m = their max; score 1: w_j = sigmoid(l_j) / sum_i sigmoid(l_i).  fp64. */
int orc_route(const float *logits, int T, int E, int k, int score, int32_t *idx, double *w)
{
    int t, j, *order;
    if (T < 0 || E < 1 || k < 1 || k > E || (score != 0 && score != 1))
        return 1;
    order = (int *)malloc(sizeof(int) * (size_t)E);
    for (t = 0; t < T; t++) {
        const float *row = logits + (size_t)t * E;
        double m, sum = 0.0;
        for (j = 0; j < E; j++) order[j] = j;
        g_sort_row = row;
        qsort(order, (size_t)E, sizeof(int), cmp_experts);
        for (j = 0; j < k; j++) idx[(size_t)t * k + j] = order[j];
        if (score == 0) {
            m = -INFINITY;
            for (j = 0; j < k; j++) if ((double)row[order[j]] > m) m = (double)row[order[j]];
            for (j = 0; j < k; j++) sum += exp((double)row[order[j]] - m);
            for (j = 0; j < k; j++) w[(size_t)t * k + j] = exp((double)row[order[j]] - m) / sum;
        } else {
            for (j = 0; j < k; j++) sum += 1.0 / (1.0 + exp(-(double)row[order[j]]));
            for (j = 0; j < k; j++)
                w[(size_t)t * k + j] = (1.0 / (1.0 + exp(-(double)row[order[j]]))) / sum;
        }
    }
    free(order);
    return 0;
}

/* Routing order on fp64 scores: larger first, NaN after every number, equal
 * values by lower index. */
static int before_d(double a, int ia, double b, int ib)
{
    int na = isnan(a), nb = isnan(b);
    if (na || nb)
        return (na && nb) ? ia < ib : nb;
    if (a != b)
        return a > b;
    return ia < ib;
}

static const double *g_sort_d;
static int cmp_d(const void *pa, const void *pb)
{
    int a = *(const int *)pa, b = *(const int *)pb;
    if (a == b) return 0;
    return before_d(g_sort_d[a], a, g_sort_d[b], b) ? -1 : 1;
}

/* Group-limited top-k (DeepSeek-V3 routing; the paper routes each token to a
 * top-k subset of experts, Section 1, and this is the rule of its DeepSeek
 * model family).  Per token: s_e = sigmoid(l_e), c_e = s_e + bias_e; the E
 * experts form G contiguous groups of E/G; a group's score is the sum of its
 * two highest c (routing order); the TG groups of highest score (ties: lower
 * group) are kept and the k experts of highest c among them (ties: lower
 * index) are selected, slot j = rank j.  Weights: w_j = scale * s_j / sum_i
 * s_i over the selected.  fp64.  bias may be NULL (zero). */
int orc_route_grouped(const float *logits, const float *bias, int T, int E, int k, int G, int TG, double scale,
                      int32_t *idx, double *w)
{
    int t, e, g, j, gs;
    double *sv, *cv, *gsc;
    int *order, *gorder, *cand;
    if (T < 0 || E < 1 || G < 1 || E % G || E / G < 2 || TG < 1 || TG > G || k < 1 || k > TG * (E / G))
        return 1;
    gs = E / G;
    sv = (double *)malloc(sizeof(double) * (size_t)E);
    cv = (double *)malloc(sizeof(double) * (size_t)E);
    gsc = (double *)malloc(sizeof(double) * (size_t)G);
    order = (int *)malloc(sizeof(int) * (size_t)E);
    gorder = (int *)malloc(sizeof(int) * (size_t)G);
    cand = (int *)malloc(sizeof(int) * (size_t)E);
    for (t = 0; t < T; t++) {
        int nc = 0;
        double sum = 0.0;
        for (e = 0; e < E; e++) {
            sv[e] = 1.0 / (1.0 + exp(-(double)logits[(size_t)t * E + e]));
            cv[e] = sv[e] + (bias ? (double)bias[e] : 0.0);
        }
        g_sort_d = cv;
        for (g = 0; g < G; g++) {
            for (j = 0; j < gs; j++) order[j] = g * gs + j;
            qsort(order, (size_t)gs, sizeof(int), cmp_d);
            gsc[g] = cv[order[0]] + cv[order[1]];
        }
        for (g = 0; g < G; g++) gorder[g] = g;
        g_sort_d = gsc;
        qsort(gorder, (size_t)G, sizeof(int), cmp_d);
        for (g = 0; g < TG; g++)
            for (j = 0; j < gs; j++) cand[nc++] = gorder[g] * gs + j;
        g_sort_d = cv;
        qsort(cand, (size_t)nc, sizeof(int), cmp_d);
        for (j = 0; j < k; j++) {
            idx[(size_t)t * k + j] = cand[j];
            sum += sv[cand[j]];
        }
        for (j = 0; j < k; j++) w[(size_t)t * k + j] = scale * sv[cand[j]] / sum;
    }
    free(sv); free(cv); free(gsc); free(order); free(gorder); free(cand);
    return 0;
}

/* Router logits (Section 1: the router scores every expert for each token):
 * logits[t][e] = sum_c x[t][c] * W_r[e][c], x [T][d] and W_r [E][d] bf16
 * bits, summed in fp64 in index order. */
int orc_router_logits(const uint16_t *x, const uint16_t *w, int T, int d, int E, double *logits)
{
    int t, e, c;
    if (T < 0 || d < 1 || E < 1)
        return 1;
    for (t = 0; t < T; t++)
        for (e = 0; e < E; e++) {
            double acc = 0.0;
            for (c = 0; c < d; c++)
                acc += orc_bf16(x[(size_t)t * d + c]) * orc_bf16(w[(size_t)e * d + c]);
            logits[(size_t)t * E + e] = acc;
        }
    return 0;
}

/* ------------------------------------------------------------------ union and grouping */

/* Expert union of the verified tokens (Section 3, Eq. 1), with the grouping the
 * expert FFN needs.  Slots are s = t*k + j.
 *   counts[e]    number of slots routed to expert e (e in [0, E))
 *   union_ids[u] the u-th expert with counts > 0, ascending; -1 for u >= U
 *   n_unique[0]  U = |union|
 *   offsets[u]   first grouped position of union member u, u in [0, E];
 *                offsets[u] = T*k for u >= U
 *   perm[p]      slot at grouped position p: slots ordered by (expert, slot). */
int orc_union(const int32_t *idx, int T, int k, int E, int32_t *counts, int32_t *union_ids,
              int32_t *n_unique, int32_t *offsets, int32_t *perm)
{
    int e, u, s, U = 0, p = 0, S = T * k;
    if (T < 0 || k < 1 || E < 1)
        return 1;
    for (e = 0; e < E; e++) counts[e] = 0;
    for (s = 0; s < S; s++) {
        if (idx[s] < 0 || idx[s] >= E) return 2;
        counts[idx[s]]++;
    }
    for (e = 0; e < E; e++) union_ids[e] = -1;
    for (e = 0; e < E; e++)
        if (counts[e] > 0) union_ids[U++] = e;
    *n_unique = U;
    for (u = 0; u <= E; u++) offsets[u] = S;
    for (u = 0; u < U; u++) {
        offsets[u] = p;
        for (s = 0; s < S; s++)
            if (idx[s] == union_ids[u]) perm[p++] = s;
    }
    return 0;
}

/* ------------------------------------------------------------------ MX activation quantisation */

/* OCP MX FP8 quantisation of one activation row of length K, in place
 * (optional activation mode act_fmt 1; the paper does not quantise
 * activations).  The row is split into blocks of 32 consecutive elements (the
 * last one zero-padded), the OCP MX block, which is also the K block the
 * scales of CDNA4's scaled FP4 x FP8 matrix-core instruction apply to.  A
 * block's scale is 2^E with E = floor(log2(amax)) - 8 (8: exponent of 448, the
 * largest e4m3fn normal), clamped to [-127, 127], and E = -127 when amax = 0.
 * Each element becomes the e4m3fn value nearest to v / 2^E, ties to the even
 * code, magnitudes of 448 and more saturating to 448, subnormals (multiples of
 * 2^-9) kept; the quantised value is that e4m3fn value times 2^E.  exps
 * (optional) receives E of every block: (K + 31) / 32 entries. */
static double e4m3_nearest(double a)  /* a >= 0, a < 448 */
{
    int p;
    double step;
    if (a == 0.0) return 0.0;
    (void)frexp(a, &p);                  /* a = m 2^p, m in [0.5, 1): floor(log2 a) = p - 1 */
    step = p - 1 < -6 ? ldexp(1.0, -9)   /* subnormal binade: multiples of 2^-9 */
                      : ldexp(1.0, p - 1 - 3);
    return rint(a / step) * step;        /* a / step < 16 is exact; rint rounds half to even */
}

int orc_mx_quant(double *v, int K, int32_t *exps)
{
    int nblocks = (K + 31) / 32, b, i;
    if (!v || K < 0) return 1;
    for (b = 0; b < nblocks; b++) {
        int lo = 32 * b, hi = 32 * b + 32 < K ? 32 * b + 32 : K, E;
        double amax = 0.0, scale;
        for (i = lo; i < hi; i++)
            if (fabs(v[i]) > amax) amax = fabs(v[i]);
        if (amax == 0.0) {
            E = -127;
        } else {
            int p;
            (void)frexp(amax, &p);
            E = p - 1 - 8;
            if (E < -127) E = -127;
            if (E > 127) E = 127;
        }
        if (exps) exps[b] = E;
        scale = ldexp(1.0, E);
        for (i = lo; i < hi; i++) {
            double a = fabs(v[i]) / scale, q = a >= 448.0 ? 448.0 : e4m3_nearest(a);
            v[i] = (v[i] < 0.0 ? -q : q) * scale;
        }
    }
    return 0;
}

/* ------------------------------------------------------------------ verify layer */

typedef struct {
    int fmt, d, d_ff, n_experts;
    const void *const *gate;   /* [n_experts] base of expert e's [d_ff][d] matrix, NULL = absent */
    const void *const *up;     /* [n_experts] [d_ff][d] */
    const void *const *down;   /* [n_experts] [d][d_ff] */
    const void *const *s_gate; /* scales per expert (NULL array for bf16) */
    const void *const *s_up;
    const void *const *s_down;
    const void *sh_gate, *sh_up, *sh_down;       /* shared expert, or NULL */
    const void *sh_s_gate, *sh_s_up, *sh_s_down;
    int act;                   /* 0: SwiGLU; 1: clamped SwiGLU of GPT-OSS (alpha, limit, up + 1) */
    double alpha, limit;
    const void *const *b_gate; /* fp32 biases per routed expert ([d_ff], [d_ff], [d]); NULL array = none */
    const void *const *b_up;
    const void *const *b_down;
    int act_fmt;               /* 0: exact bf16 inputs; 1: x and h quantised by orc_mx_quant */
} orc_layer;

/* One expert FFN.  g_n = sum_c x_c W_gate[n][c] + bg_n, v_n = sum_c x_c W_up[n][c] + bu_n
 * (biases NULL: zero).  act 0: h_n = silu(g_n) * v_n.  act 1 (GPT-OSS): g clamped
 * from above at `limit`, v clamped to [-limit, limit], h_n = g sigmoid(alpha g) (v + 1).
 * act_fmt 1: h quantised by orc_mx_quant (x is quantised by the caller).
 * o[m] = sum_n h_n W_down[m][n] + bd_m. */
static void swiglu_expert(int fmt, int d, int d_ff, const void *wg, const void *wu, const void *wd,
                          const void *sg, const void *su, const void *sd, int act, double alpha,
                          double limit, const float *bg, const float *bu, const float *bd, int act_fmt,
                          const double *x, double *h, double *o)
{
    int n, c, m;
    for (n = 0; n < d_ff; n++) {
        double g = 0.0, v = 0.0;
        for (c = 0; c < d; c++) {
            g += x[c] * weight_at(fmt, wg, sg, d_ff, d, n, c);
            v += x[c] * weight_at(fmt, wu, su, d_ff, d, n, c);
        }
        if (bg) g += (double)bg[n];
        if (bu) v += (double)bu[n];
        if (act == 0) {
            h[n] = g / (1.0 + exp(-g)) * v;
        } else {
            if (g > limit) g = limit;
            if (v > limit) v = limit;
            if (v < -limit) v = -limit;
            h[n] = g / (1.0 + exp(-alpha * g)) * (v + 1.0);
        }
    }
    if (act_fmt == 1) orc_mx_quant(h, d_ff, NULL);
    for (m = 0; m < d; m++) {
        double acc = 0.0;
        for (n = 0; n < d_ff; n++) acc += h[n] * weight_at(fmt, wd, sd, d, d_ff, m, n);
        o[m] = acc + (bd ? (double)bd[m] : 0.0);
    }
}

/* y[i][:] for token tokens[i]: sum_j w[t][j] * FFN_{idx[t][j]}(x_t), j ascending,
 * then + FFN_shared(x_t) when the layer has a shared expert.  x is bf16 [T][d].
 * Independent (token, slot) products run on up to nthreads threads; the sum
 * order is fixed, so the result does not depend on the thread count. */
int orc_verify_tokens(const orc_layer *L, const uint16_t *x, int T, int k, const int32_t *idx,
                      const double *w, int n_sel, const int32_t *tokens, double *y, int nthreads)
{
    int d = L->d, d_ff = L->d_ff, has_sh = L->sh_gate != NULL, per = k + (L->sh_gate != NULL);
    long total = (long)n_sel * per, q;
    double *o;
    int bad = 0;
    if (!L || !x || !idx || !w || !y || n_sel < 0 || k < 1)
        return 1;
    for (q = 0; q < n_sel; q++)
        if (tokens[q] < 0 || tokens[q] >= T) return 1;
    for (q = 0; q < (long)n_sel * k; q++) {
        int e = idx[(size_t)tokens[q / k] * k + q % k];
        if (e < 0 || e >= L->n_experts || !L->gate[e] || !L->up[e] || !L->down[e]) return 2;
    }
    o = (double *)malloc(sizeof(double) * (size_t)total * d);
    if (!o) return 3;
#ifdef _OPENMP
    if (nthreads < 1) nthreads = 1;
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads)
#else
    (void)nthreads;
#endif
    for (q = 0; q < total; q++) {
        int i = (int)(q / per), j = (int)(q % per), t = tokens[i], c;
        double *xt = (double *)malloc(sizeof(double) * (size_t)d);
        double *h = (double *)malloc(sizeof(double) * (size_t)d_ff);
        if (!xt || !h) { bad = 1; free(xt); free(h); continue; }
        for (c = 0; c < d; c++) xt[c] = orc_bf16(x[(size_t)t * d + c]);
        if (L->act_fmt == 1) orc_mx_quant(xt, d, NULL);
        if (j < k) {
            int e = idx[(size_t)t * k + j];
            swiglu_expert(L->fmt, d, d_ff, L->gate[e], L->up[e], L->down[e],
                          L->s_gate ? L->s_gate[e] : NULL, L->s_up ? L->s_up[e] : NULL,
                          L->s_down ? L->s_down[e] : NULL, L->act, L->alpha, L->limit,
                          L->b_gate ? (const float *)L->b_gate[e] : NULL,
                          L->b_up ? (const float *)L->b_up[e] : NULL,
                          L->b_down ? (const float *)L->b_down[e] : NULL, L->act_fmt, xt, h,
                          o + (size_t)q * d);
        } else {
            swiglu_expert(L->fmt, d, d_ff, L->sh_gate, L->sh_up, L->sh_down, L->sh_s_gate,
                          L->sh_s_up, L->sh_s_down, L->act, L->alpha, L->limit, NULL, NULL, NULL, L->act_fmt,
                          xt, h, o + (size_t)q * d);
        }
        free(xt);
        free(h);
    }
    if (!bad) {
        int i, j, m;
        for (i = 0; i < n_sel; i++) {
            int t = tokens[i];
            for (m = 0; m < d; m++) {
                double acc = 0.0;
                for (j = 0; j < k; j++)
                    acc += w[(size_t)t * k + j] * o[((size_t)i * per + j) * d + m];
                if (has_sh)
                    acc += o[((size_t)i * per + k) * d + m];
                y[(size_t)i * d + m] = acc;
            }
        }
    }
    free(o);
    return bad ? 3 : 0;
}

/* Bytes one expert occupies in HBM: weights and scales (Fig. 1(c)). */
void orc_expert_bytes(int fmt, long d, long d_ff, long *weight_bytes, long *scale_bytes)
{
    long n = 3 * d * d_ff;
    switch (fmt) {
    case 0: *weight_bytes = 2 * n; *scale_bytes = 0; break;
    case 1: *weight_bytes = n; *scale_bytes = 4 * 3 * (d / 128) * (d_ff / 128); break;
    case 2: *weight_bytes = n / 2; *scale_bytes = n / 32; break;
    default: *weight_bytes = -1; *scale_bytes = -1;
    }
}
