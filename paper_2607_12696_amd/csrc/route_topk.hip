// Router top-k on gfx950: one 64-lane wavefront per token.
//
// Each token's E logits (E <= 1024) are spread over the lanes of one wave.
// An expert's position in the routing order is a 64-bit key: the upper 32
// bits map the fp32 logit to an unsigned integer that preserves its order
// (-0 folded onto +0, NaN below every number) and the lower 32 bits hold the
// complement of the expert index, so equal logits prefer the lower index and
// all keys are distinct.  k rounds of a wave-wide max pick the experts in
// order; the owner lane clears its key after each round.  Gate weights are
// then a softmax or a renormalised sigmoid over the k selected logits, held
// one per lane, in fp32.
#include "device.hpp"
#include "launch.hpp"
#include "route_common.hpp"

namespace ecospec {

// slices == 0: `logits` is [T][E].  slices > 0: `logits` holds the router's
// K-slice partial sums [slices][T][E], added here in slice order; the sums
// are also stored to logits_out when it is given.
template <int EPL>  // experts per lane: ceil(E / 64)
__global__ __launch_bounds__(256) void route_topk_kernel(const float *__restrict__ logits, int slices, int T, int E,
                                                         int k, int score, int32_t *__restrict__ topk_idx,
                                                         float *__restrict__ topk_w, float *__restrict__ logits_out)
{
    const int lane = lane_id();
    const int t = blockIdx.x * (blockDim.x / kWave) + (threadIdx.x / kWave);
    if (t >= T) return;  // uniform per wave
    const float *row = logits + (size_t)t * E;

    float val[EPL];
    if (slices == 0) {
#pragma unroll
        for (int i = 0; i < EPL; ++i) {
            const int e = lane + kWave * i;
            val[i] = e < E ? row[e] : 0.f;
        }
    } else {
        // Sum the slices in order, CH at a time with all their loads in flight.
        constexpr int CH = EPL >= 8 ? 2 : 8;
#pragma unroll
        for (int i = 0; i < EPL; ++i) val[i] = 0.f;
        for (int s0 = 0; s0 < slices; s0 += CH) {
            float p[EPL][CH];
#pragma unroll
            for (int c = 0; c < CH; ++c)
#pragma unroll
                for (int i = 0; i < EPL; ++i) {
                    const int e = lane + kWave * i;
                    p[i][c] = (s0 + c < slices && e < E) ? logits[((size_t)(s0 + c) * T + t) * E + e] : 0.f;
                }
#pragma unroll
            for (int c = 0; c < CH; ++c)
                if (s0 + c < slices)
#pragma unroll
                    for (int i = 0; i < EPL; ++i) val[i] += p[i][c];
        }
        if (logits_out) {
#pragma unroll
            for (int i = 0; i < EPL; ++i) {
                const int e = lane + kWave * i;
                if (e < E) logits_out[(size_t)t * E + e] = val[i];
            }
        }
    }
    uint64_t key[EPL];
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
        const int e = lane + kWave * i;
        key[i] = e < E ? ((uint64_t)order_key(val[i]) << 32) | (uint32_t)~(uint32_t)e : 0ull;
    }

    const int mine = select_ranks(key, k);
    const float wgt = gate_weight(value_of(val, mine), k, score);
    if (lane < k) {
        topk_idx[(size_t)t * k + lane] = mine;
        topk_w[(size_t)t * k + lane] = wgt;
    }
}

// Group-limited routing (the DeepSeek-V3 rule): sigmoid scores s, choice
// scores c = s + bias; the E experts form G contiguous groups of gs = E / G
// (gs >= 2); a group's score is the sum of its two highest choice scores (in
// the routing order of order_key, so NaN only counts when a group has fewer
// than two numbers); the TG groups of highest score (ties: lower group) stay
// eligible and the k highest choice scores among their experts are selected,
// in order.  Gate weights: scale * s / sum(s) over the selected.  One
// wavefront per token; the choice scores go through LDS so that lane g can
// score group g.
template <int EPL>
__global__ __launch_bounds__(256) void route_grouped_kernel(const float *__restrict__ logits,
                                                            const float *__restrict__ bias, int T, int E, int k,
                                                            int G, int TG, float scale, int32_t *__restrict__ topk_idx,
                                                            float *__restrict__ topk_w)
{
    __shared__ float cs[4][1024];
    const int lane = lane_id(), wv = threadIdx.x / kWave;
    const int t = blockIdx.x * 4 + wv;
    const bool active = t < T;
    const int gs = E / G;
    float sv[EPL], cv[EPL];
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
        const int e = lane + kWave * i;
        const float l = (active && e < E) ? logits[(size_t)t * E + e] : 0.f;
        sv[i] = 1.f / (1.f + expf(-l));
        cv[i] = sv[i] + ((bias && e < E) ? bias[e] : 0.f);
        if (e < E) cs[wv][e] = cv[i];
    }
    __syncthreads();
    if (!active) return;  // uniform per wave, after the block's only barrier

    uint64_t gkey = 0ull;
    if (lane < G) {
        uint32_t k1 = 0u, k2 = 0u;
        float v1 = 0.f, v2 = 0.f;
        bool h1 = false, h2 = false;
        for (int j = 0; j < gs; ++j) {
            const float v = cs[wv][lane * gs + j];
            const uint32_t kv = order_key(v);
            if (!h1 || kv > k1) {
                k2 = k1; v2 = v1; h2 = h1;
                k1 = kv; v1 = v; h1 = true;
            } else if (!h2 || kv > k2) {
                k2 = kv; v2 = v; h2 = true;
            }
        }
        gkey = ((uint64_t)order_key(v1 + v2) << 32) | (uint32_t)~(uint32_t)lane;
    }
    uint64_t gmask = 0ull;  // bit g: group g stays eligible
    for (int r = 0; r < TG; ++r) {
        const uint64_t m = wave_max_u64(gkey);
        const int g = (int)~(uint32_t)m;
        gmask |= 1ull << g;
        if (lane == g) gkey = 0ull;
    }
    uint64_t key[EPL];
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
        const int e = lane + kWave * i;
        key[i] = (e < E && ((gmask >> (e / gs)) & 1ull)) ? ((uint64_t)order_key(cv[i]) << 32) | (uint32_t)~(uint32_t)e
                                                          : 0ull;
    }
    const int mine = select_ranks(key, k);
    const bool sel = lane < k;
    const float sm = value_of(sv, mine);  // every lane takes part in the shuffles
    const float g = sel ? sm : 0.f;
    const float sum = wave_sum(g);
    if (sel) {
        topk_idx[(size_t)t * k + lane] = mine;
        topk_w[(size_t)t * k + lane] = scale * (g / sum);
    }
}

hipError_t launch_route_grouped(const float *logits, const float *bias, int T, int E, int k, int G, int TG,
                                float scale, int32_t *idx, float *w, hipStream_t stream)
{
    const dim3 block(256), grid((T + 3) / 4);
    const int epl = (E + kWave - 1) / kWave;
#define GROUPED_CASE(N)                                                                                         \
    case N:                                                                                                     \
        hipLaunchKernelGGL(route_grouped_kernel<N>, grid, block, 0, stream, logits, bias, T, E, k, G, TG, scale, \
                           idx, w);                                                                             \
        break;
    switch (epl) {
        GROUPED_CASE(1) GROUPED_CASE(2) GROUPED_CASE(3) GROUPED_CASE(4) GROUPED_CASE(5) GROUPED_CASE(6)
        GROUPED_CASE(7) GROUPED_CASE(8) GROUPED_CASE(9) GROUPED_CASE(10) GROUPED_CASE(11) GROUPED_CASE(12)
        GROUPED_CASE(13) GROUPED_CASE(14) GROUPED_CASE(15) GROUPED_CASE(16)
    default: return hipErrorInvalidValue;
    }
#undef GROUPED_CASE
    return hipGetLastError();
}

hipError_t launch_route_topk(const float *logits, int slices, int T, int E, int k, int score, int32_t *idx, float *w,
                             float *logits_out, hipStream_t stream)
{
    const dim3 block(256), grid((T + 3) / 4);
    const int epl = (E + kWave - 1) / kWave;
#define ROUTE_CASE(N)                                                                                          \
    case N:                                                                                                    \
        hipLaunchKernelGGL(route_topk_kernel<N>, grid, block, 0, stream, logits, slices, T, E, k, score, idx, w, \
                           logits_out);                                                                        \
        break;
    switch (epl) {
        ROUTE_CASE(1) ROUTE_CASE(2) ROUTE_CASE(3) ROUTE_CASE(4) ROUTE_CASE(5) ROUTE_CASE(6) ROUTE_CASE(7)
        ROUTE_CASE(8) ROUTE_CASE(9) ROUTE_CASE(10) ROUTE_CASE(11) ROUTE_CASE(12) ROUTE_CASE(13)
        ROUTE_CASE(14) ROUTE_CASE(15) ROUTE_CASE(16)
    default: return hipErrorInvalidValue;
    }
#undef ROUTE_CASE
    return hipGetLastError();
}

}  // namespace ecospec
