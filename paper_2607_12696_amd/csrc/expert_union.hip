// Expert union, histogram, scans and stable grouping on gfx950, in one
// workgroup of 1024 threads (E <= 1024, so thread e owns expert e).
//
//  1. LDS histogram of the T*k routed slots (integer atomics: exact).
//  2. Two block-wide exclusive scans over the experts: of the "used" flags
//     (position of each expert in the ascending union) and of the counts
//     (first grouped position of each expert).
//  3. Stable counting sort of the slots into perm: wavefront 0 walks the
//     slots 64 at a time; lanes holding the same expert find each other with
//     one ballot per bit of the expert id, take their rank among the lower
//     lanes, and the highest such lane advances that expert's cursor.  Slots
//     therefore land in ascending order within each expert.
#include "device.hpp"
#include "launch.hpp"

namespace ecospec {

constexpr int kUnionThreads = 1024;

__global__ __launch_bounds__(kUnionThreads) void expert_union_kernel(
    const int32_t *__restrict__ idx, int S, int E, int32_t *__restrict__ counts, int32_t *__restrict__ union_ids,
    int32_t *__restrict__ n_unique, int32_t *__restrict__ offsets, int32_t *__restrict__ perm)
{
    __shared__ int cnt[kUnionThreads];
    __shared__ int cursor[kUnionThreads];
    __shared__ int member_id[kUnionThreads];
    __shared__ int member_start[kUnionThreads];
    __shared__ int wave_tot[kUnionThreads / kWave];
    const int tid = threadIdx.x;

    cnt[tid] = 0;
    __syncthreads();
    for (int s = tid; s < S; s += kUnionThreads) {
        const int e = idx[s];
        if ((unsigned)e < (unsigned)E) atomicAdd(&cnt[e], 1);
    }
    __syncthreads();

    const int c = tid < E ? cnt[tid] : 0;
    int U = 0, placed = 0;
    const int pos = block_exclusive_scan(c > 0 ? 1 : 0, wave_tot, &U);
    const int start = block_exclusive_scan(c, wave_tot, &placed);

    if (tid < E) {
        counts[tid] = c;
        cursor[tid] = start;
        if (c > 0) {
            member_id[pos] = tid;
            member_start[pos] = start;
        }
    }
    __syncthreads();
    for (int u = tid; u <= E; u += kUnionThreads) {
        if (u < E) union_ids[u] = u < U ? member_id[u] : -1;
        offsets[u] = u < U ? member_start[u] : placed;
    }
    if (tid == 0) *n_unique = U;

    if (tid < kWave) {
        const int lane = tid;
        const uint64_t below = (1ull << lane) - 1ull;
        int nbits = 0;
        while ((1 << nbits) < E) ++nbits;
        for (int base = 0; base < S; base += kWave) {
            const int s = base + lane;
            const int e = s < S ? idx[s] : -1;
            const bool ok = (unsigned)e < (unsigned)E;
            uint64_t peers = __ballot(ok);
            for (int b = 0; b < nbits; ++b) {
                const bool bit = ok && ((e >> b) & 1);
                const uint64_t m = __ballot(bit);
                peers &= bit ? m : ~m;
            }
            if (ok) {
                const int rank = __popcll(peers & below);
                const int at = cursor[e];
                perm[at + rank] = s;
                if (lane == 63 - __clzll(peers)) cursor[e] = at + __popcll(peers);
            }
            __threadfence_block();  // cursor updates precede the next chunk's reads
        }
    }
}

hipError_t launch_expert_union(const int32_t *idx, int T, int k, int E, int32_t *counts, int32_t *union_ids,
                               int32_t *n_unique, int32_t *offsets, int32_t *perm, hipStream_t stream)
{
    hipLaunchKernelGGL(expert_union_kernel, dim3(1), dim3(kUnionThreads), 0, stream, idx, T * k, E, counts,
                       union_ids, n_unique, offsets, perm);
    return hipGetLastError();
}

}  // namespace ecospec
