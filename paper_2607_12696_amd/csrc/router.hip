// Router logits from hidden states on gfx950: logits[t][e] = sum_c x[t][c] *
// W_r[e][c] (bf16 inputs, fp32 accumulation), the scores a top-k routing reads
// (Section 1: a router sends each token to a top-k subset of the experts).
//
// The product is tiny (T x E outputs over K = d) and bound by latency, so it is
// split along K.  Workgroup (16-expert tile, 512-wide K slice, 64-token group)
// has four wavefronts; wavefront w takes the quarter [128w, 128w + 128) of the
// slice for all four 16-token tiles of the group.  It issues every load at once
// (4 operand fragments of W_r and 16 of x, 16 bytes per lane, exactly the lane
// fragments v_mfma_f32_16x16x32_bf16 takes: experts on the 16-row side, tokens
// on the 16-column side), then runs 16 matrix-core steps, so the workgroup
// costs one memory round trip and reads each W_r byte once.  The four quarters
// are added through LDS in wavefront order and each lane stores the four
// consecutive experts it holds with one 16-byte store.  Buffer loads past the
// end of x or W_r return zeros, which covers the expert and token tails.  The
// fp32 partial sums of the slices, [slices][T][E], are added in slice order by
// the routing kernel that follows, so the logits are deterministic.
#include "device.hpp"
#include "launch.hpp"

namespace ecospec {

constexpr int kRouterSlice = 512;  // K elements per slice (4 wavefronts x 4 steps x 32)
constexpr int kRouterTiles = 4;    // 16-token tiles per workgroup
constexpr int kRouterSteps = 4;    // matrix-core steps per wavefront

int router_slices(int d) { return (d + kRouterSlice - 1) / kRouterSlice; }

__global__ __launch_bounds__(256) void router_gemm_kernel(const uint16_t *__restrict__ x, const uint16_t *__restrict__ w,
                                                          int T, int d, int E, float *__restrict__ partial)
{
    __shared__ f32x4 red[4][kRouterTiles][kWave];
    const int lane = lane_id(), wave = threadIdx.x / kWave;
    const int e0 = blockIdx.x * 16, slice = blockIdx.y, tg = blockIdx.z * 16 * kRouterTiles;
    const int k_w = slice * kRouterSlice + wave * 32 * kRouterSteps;  // this wavefront's first K index
    const int r = lane & 15, kq = (lane >> 4) * 8;                    // operand row / column and K offset
    const rsrc_t rw = make_rsrc(w, (uint32_t)((size_t)E * d * 2));
    const rsrc_t rx = make_rsrc(x, (uint32_t)((size_t)T * d * 2));
    const int e = e0 + r;

    u32x4 a[kRouterSteps], b[kRouterTiles][kRouterSteps];
#pragma unroll
    for (int i = 0; i < kRouterSteps; ++i) {
        const int k = k_w + 32 * i;  // d % 32 == 0: a step is wholly in range or wholly out
        a[i] = load16<0>(rw, k < d && e < E ? (uint32_t)(((size_t)e * d + k + kq) * 2) : kOff);
#pragma unroll
        for (int j = 0; j < kRouterTiles; ++j) {
            const int t = tg + 16 * j + r;
            b[j][i] = load16<0>(rx, k < d && t < T ? (uint32_t)(((size_t)t * d + k + kq) * 2) : kOff);
        }
    }
    // Keep every load ahead of the first matrix-core step: the scheduler would
    // otherwise interleave them to save registers and pay several round trips.
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < kRouterTiles; ++j) {
        f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int i = 0; i < kRouterSteps; ++i)
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a[i]),
                                                          __builtin_bit_cast(bf16x8, b[j][i]), acc, 0, 0, 0);
        red[wave][j][lane] = acc;
    }
    __syncthreads();

    // Wavefront j finishes token tile j: quarters added in order 0, 1, 2, 3.
    const int j = wave;
    const int t = tg + 16 * j + r;
    if (t >= T) return;
    f32x4 s = red[0][j][lane];
#pragma unroll
    for (int q4 = 1; q4 < 4; ++q4) s += red[q4][j][lane];
    // Lane (r, q) holds experts e0 + 4q .. e0 + 4q + 3 of token t.
    const int eq = e0 + 4 * (lane >> 4);
    float *dst = partial + ((size_t)slice * T + t) * E + eq;
    if ((E & 3) == 0) {
        if (eq < E) *reinterpret_cast<f32x4 *>(dst) = s;
    } else {
#pragma unroll
        for (int i = 0; i < 4; ++i)
            if (eq + i < E) dst[i] = s[i];
    }
}

hipError_t launch_router_gemm(const uint16_t *x, const uint16_t *w, int T, int d, int E, float *partial,
                              hipStream_t stream)
{
    const dim3 grid((E + 15) / 16, router_slices(d), (T + 16 * kRouterTiles - 1) / (16 * kRouterTiles));
    hipLaunchKernelGGL(router_gemm_kernel, grid, dim3(256), 0, stream, x, w, T, d, E, partial);
    return hipGetLastError();
}

}  // namespace ecospec
