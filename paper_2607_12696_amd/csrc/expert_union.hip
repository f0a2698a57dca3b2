// Expert union, histogram, scans and stable grouping on gfx950, in one
// workgroup of 1024 threads (E <= 1024, so thread e owns expert e).
//
// The routed slots are taken 1024 at a time, one per thread, in slot order
// (wavefront w holds slots 64w .. 64w + 63 of a pass).  Within a wavefront,
// lanes holding the same expert find each other with one ballot per bit of
// the expert id; a lane's rank among the lower such lanes orders equal
// experts by slot, and the highest lane of each expert records the
// wavefront's count in LDS.  A pass then adds, per expert, the counts of the
// earlier wavefronts (and passes): that prefix plus the rank places every slot
// of the pass at once.  So the grouping is a stable counting sort by expert.
//
//  1. Counts per expert: the sum of the per-wavefront counts of all passes.
//  2. Two block-wide exclusive scans over the experts: of the "used" flags
//     (position of each expert in the ascending union) and of the counts
//     (first grouped position of each expert).
//  3. The passes again, placing each slot at first position of its expert +
//     slots of that expert in earlier passes and wavefronts + rank.
// With a single pass (S <= 1024) the matches are kept in registers between
// steps 1 and 3 and the two scans are done as one.
#include "device.hpp"
#include "launch.hpp"

namespace ecospec {

constexpr int kUnionThreads = 1024;
constexpr int kUnionWaves = kUnionThreads / kWave;

// The union, scans and grouping of S routed slots idx[0 .. S) (global or LDS),
// by the whole 1024-thread workgroup.
__device__ __forceinline__ void union_block(const int32_t *idx, int S, int E, int32_t *__restrict__ counts,
                                            int32_t *__restrict__ union_ids, int32_t *__restrict__ n_unique,
                                            int32_t *__restrict__ offsets, int32_t *__restrict__ perm)
{
    __shared__ int wcnt[kUnionWaves][kUnionThreads];  // per-wavefront counts of the current pass
    __shared__ int member_id[kUnionThreads];
    __shared__ int member_start[kUnionThreads];
    __shared__ int wave_tot[kUnionWaves];
    const int tid = threadIdx.x, wave = tid / kWave;
    int nbits = 0;
    while ((1 << nbits) < E) ++nbits;
    const int passes = (S + kUnionThreads - 1) / kUnionThreads;

    if (passes == 1) {
        // One pass (S <= 1024, every verification batch of up to 64 tokens x 16
        // slots): the slots' matches stay in registers from counting to
        // placement, and one scan of (count << 16 | used) gives both prefixes
        // (count, union size and placed slots are all <= 1024 < 2^16).
        for (int w = 0; w < kUnionWaves; ++w) wcnt[w][tid] = 0;
        __syncthreads();
        const int e = tid < S ? idx[tid] : -1;
        const bool ok = (unsigned)e < (unsigned)E;
        int rank, cnt;
        bool top;
        wave_match(e, ok, nbits, rank, top, cnt);
        if (top) wcnt[wave][e] = cnt;
        __syncthreads();
        int c = 0;
        if (tid < E)
            for (int w = 0; w < kUnionWaves; ++w) c += wcnt[w][tid];
        int tot = 0;
        const int ex = block_exclusive_scan((c << 16) | (c > 0 ? 1 : 0), wave_tot, &tot);
        const int pos = ex & 0xffff, start = ex >> 16, U = tot & 0xffff, placed = tot >> 16;
        if (tid < E) {
            counts[tid] = c;
            if (c > 0) {
                member_id[pos] = tid;
                member_start[pos] = start;
            }
            // Per-wavefront counts of expert tid -> first position of each wavefront's slots.
            int run = start;
            for (int w = 0; w < kUnionWaves; ++w) {
                const int n = wcnt[w][tid];
                wcnt[w][tid] = run;
                run += n;
            }
        }
        __syncthreads();
        for (int u = tid; u <= E; u += kUnionThreads) {
            if (u < E) union_ids[u] = u < U ? member_id[u] : -1;
            offsets[u] = u < U ? member_start[u] : placed;
        }
        if (tid == 0) *n_unique = U;
        if (ok) perm[wcnt[wave][e] + rank] = tid;
        return;
    }

    // 1. Counts: per-wavefront matches, summed per expert over wavefronts and passes.
    int total = 0;  // thread e: slots routed to expert e
    for (int ps = 0; ps < passes; ++ps) {
        for (int w = 0; w < kUnionWaves; ++w) wcnt[w][tid] = 0;
        __syncthreads();
        const int s = ps * kUnionThreads + tid;
        const int e = s < S ? idx[s] : -1;
        const bool ok = (unsigned)e < (unsigned)E;
        int rank, cnt;
        bool top;
        wave_match(e, ok, nbits, rank, top, cnt);
        if (top) wcnt[wave][e] = cnt;
        __syncthreads();
        if (tid < E)
            for (int w = 0; w < kUnionWaves; ++w) total += wcnt[w][tid];
        __syncthreads();
    }

    // 2. Union positions and first grouped positions.
    const int c = tid < E ? total : 0;
    int U = 0, placed = 0;
    const int pos = block_exclusive_scan(c > 0 ? 1 : 0, wave_tot, &U);
    const int start = block_exclusive_scan(c, wave_tot, &placed);
    if (tid < E) {
        counts[tid] = c;
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

    // 3. Placement, pass by pass: thread e turns the per-wavefront counts into
    //    first positions (in place), then every slot of the pass is placed.
    int run = start;  // thread e: next position of expert e
    for (int ps = 0; ps < passes; ++ps) {
        for (int w = 0; w < kUnionWaves; ++w) wcnt[w][tid] = 0;
        __syncthreads();
        const int s = ps * kUnionThreads + tid;
        const int e = s < S ? idx[s] : -1;
        const bool ok = (unsigned)e < (unsigned)E;
        int rank, cnt;
        bool top;
        wave_match(e, ok, nbits, rank, top, cnt);
        if (top) wcnt[wave][e] = cnt;
        __syncthreads();
        if (tid < E) {
            for (int w = 0; w < kUnionWaves; ++w) {
                const int n = wcnt[w][tid];
                wcnt[w][tid] = run;
                run += n;
            }
        }
        __syncthreads();
        if (ok) perm[wcnt[wave][e] + rank] = s;
        __syncthreads();
    }
}

__global__ __launch_bounds__(kUnionThreads) void expert_union_kernel(
    const int32_t *__restrict__ idx, int S, int E, int32_t *__restrict__ counts, int32_t *__restrict__ union_ids,
    int32_t *__restrict__ n_unique, int32_t *__restrict__ offsets, int32_t *__restrict__ perm)
{
    union_block(idx, S, E, counts, union_ids, n_unique, offsets, perm);
}

hipError_t launch_expert_union(const int32_t *idx, int T, int k, int E, int32_t *counts, int32_t *union_ids,
                               int32_t *n_unique, int32_t *offsets, int32_t *perm, hipStream_t stream)
{
    hipLaunchKernelGGL(expert_union_kernel, dim3(1), dim3(kUnionThreads), 0, stream, idx, T * k, E, counts,
                       union_ids, n_unique, offsets, perm);
    return hipGetLastError();
}

}  // namespace ecospec
