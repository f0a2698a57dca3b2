// Routing helpers shared by the top-k kernels (one 64-lane wavefront per
// token; expert e = lane + 64 i sits in register i of its lane).
#pragma once

#include "device.hpp"

namespace ecospec {

__device__ __forceinline__ uint32_t order_key(float v)
{
    uint32_t b = __float_as_uint(v);
    if (v != v) return 0u;             // NaN after every number
    if (b == 0x80000000u) b = 0u;      // -0 == +0
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// k rounds of a wave-wide max over the experts' keys (expert e = lane + 64 i
// in register i; key 0 = not eligible): lane r returns the expert of rank r.
template <int EPL>
__device__ __forceinline__ int select_ranks(uint64_t (&key)[EPL], int k)
{
    const int lane = lane_id();
    int mine = -1;
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
    return mine;
}

// val of expert `mine` (held by lane mine % 64 in register mine / 64).  Call
// it from every lane: a lane-permute reads nothing from inactive lanes.
template <int EPL>
__device__ __forceinline__ float value_of(const float (&val)[EPL], int mine)
{
    float v = 0.f;
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
        const float c = __shfl(val[i], (mine - kWave * i) & (kWave - 1), kWave);
        if (mine >= kWave * i && mine < kWave * (i + 1)) v = c;
    }
    return v;
}

// Gate weight of rank `lane` (< k) from its logit v, held one per lane: a
// softmax over the k selected logits (score 0; rank 0 holds the largest) or a
// renormalised sigmoid (score 1), in fp32.  Every lane must call it.
__device__ __forceinline__ float gate_weight(float v, int k, int score)
{
    const bool sel = lane_id() < k;
    if (!sel) v = 0.f;
    float g;
    if (score == 0) {
        const float m = __shfl(v, 0, kWave);
        g = sel ? expf(v - m) : 0.f;
    } else {
        g = sel ? 1.f / (1.f + expf(-v)) : 0.f;
    }
    return g / wave_sum(g);
}

}  // namespace ecospec
