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

namespace ecospec {

__device__ __forceinline__ uint32_t order_key(float v)
{
    uint32_t b = __float_as_uint(v);
    if (v != v) return 0u;             // NaN after every number
    if (b == 0x80000000u) b = 0u;      // -0 == +0
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

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

    int mine = -1;  // lane r keeps the expert of rank r
    for (int r = 0; r < k; ++r) {
        uint64_t best = 0ull;
        int bi = -1;
#pragma unroll
        for (int i = 0; i < EPL; ++i)
            if (key[i] > best) { best = key[i]; bi = i; }
        const uint64_t win = wave_max_u64(best);
        if (bi >= 0 && best == win) {
#pragma unroll
            for (int i = 0; i < EPL; ++i)
                if (i == bi) key[i] = 0ull;
        }
        if (lane == r) mine = (int)~(uint32_t)win;
    }

    // The selected logit of each rank, from the lane that holds that expert.
    float v = 0.f;
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
        const int src = mine - kWave * i;  // lane holding `mine` in register i
        const float c = __shfl(val[i], src & (kWave - 1), kWave);
        if (mine >= kWave * i && mine < kWave * (i + 1)) v = c;
    }
    const bool sel = lane < k;
    if (!sel) v = 0.f;
    float g;
    if (score == 0) {
        const float m = __shfl(v, 0, kWave);  // rank 0 holds the largest logit
        g = sel ? expf(v - m) : 0.f;
    } else {
        g = sel ? 1.f / (1.f + expf(-v)) : 0.f;
    }
    const float s = wave_sum(g);
    if (sel) {
        topk_idx[(size_t)t * k + lane] = mine;
        topk_w[(size_t)t * k + lane] = g / s;
    }
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
