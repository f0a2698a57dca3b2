// Grouped SwiGLU experts of the verification pass on gfx950 (CDNA4).
//
// The pass is bound by HBM bandwidth: every distinct expert routed to by the
// T <= 64 verified tokens must be read once, while each weight is used by
// only M_u <= T tokens (arithmetic intensity <= 2*M_u flop per weight).  The
// kernels are therefore weight streams with a small matrix-core contraction
// attached:
//
//  * A work item is one expert and a band of 16 (gate/up) or 32 (down) weight
//    rows.  One 64-lane wavefront owns an item and walks the full reduction
//    dimension K in macro steps of 128: lane (c, g) = (lane % 16, lane / 16)
//    loads the 32 consecutive weights [k0 + 32 g, k0 + 32 g + 32) of row c of
//    each 16-row tile with 128-bit loads (64, 32 or 16 bytes for bf16, FP8 or
//    MXFP4), so each row contributes a whole 128-byte line per macro step and
//    every weight byte is fetched from HBM exactly once.  Several macro steps
//    are kept in flight per wavefront.
//  * The loaded words are already in the A-operand layout of
//    v_mfma_f32_16x16x32_bf16 (weights on the 16-row side, tokens on the
//    16-column side): weights are decoded exactly to bf16 in registers
//    (v_cvt_scalef32_pk_bf16_fp8 with unit scale, v_cvt_scalef32_pk_bf16_fp4
//    with the e8m0 power of two) and never touch LDS.  The B operand is the
//    gathered activation rows (x for gate/up, the grouped bf16 SwiGLU output
//    H for down), read from L2 in the same K order.
//  * FP8 128x128 block scales are applied to the fp32 partial sum of each
//    macro step (one step = one scale block), so the weights stay exact.
//  * Up to 32 tokens (2 blocks of 16) share one pass over an expert's
//    weights; an expert with more tokens takes further passes.
//  * Grids are persistent: the number of items depends on the union size U,
//    which stays on the device; wavefronts stride over items until U runs out.
//
// Kernel sequence of moe_verify_layer: gateup -> down -> combine.  The down
// kernel writes each slot's weighted expert output to an fp32 buffer and the
// combine kernel sums a token's k slots (then the shared expert) in a fixed
// order, so the result is deterministic without atomics.
#include "device.hpp"
#include "launch.hpp"

namespace ecospec {

enum { FMT_BF16 = 0, FMT_FP8 = 1, FMT_MXFP4 = 2 };

constexpr int kMacroK = 128;   // K per macro step: 4 lane groups x 32 weights
constexpr int kMaxMB = 2;      // 16-token blocks per pass (register budget of 2 waves per SIMD)
constexpr int kWavesPerCU = 8; // persistent grid: wavefronts per compute unit

// ----------------------------------------------------------------------------- weight fragments

template <int FMT> struct WTraits;
template <> struct WTraits<FMT_BF16>  { static constexpr int kVecs = 4; static constexpr int kNum = 2, kDen = 1; };
template <> struct WTraits<FMT_FP8>   { static constexpr int kVecs = 2; static constexpr int kNum = 1, kDen = 1; };
template <> struct WTraits<FMT_MXFP4> { static constexpr int kVecs = 1; static constexpr int kNum = 1, kDen = 2; };

// 32 consecutive weights of one row held by one lane, plus its scale.
template <int FMT> struct WFrag {
    u32x4 v[WTraits<FMT>::kVecs];
    float scale;  // FP8: block scale (uniform over the wave); MXFP4: 2^(e8m0-127); bf16: unused
};

__device__ __forceinline__ float e8m0_to_f32(uint32_t code)
{
    // 2^(code-127); code 0 is the subnormal 2^-127, code 255 is NaN.
    return code == 0u ? __uint_as_float(0x00400000u) : code == 255u ? __uint_as_float(0x7fc00000u)
                                                                      : __uint_as_float(code << 23);
}

// Load the lane's 32 weights of row `row` starting at element k (k < K) of an N x K matrix.
template <int FMT>
__device__ __forceinline__ void load_wfrag(WFrag<FMT> &f, const uint8_t *__restrict__ mat, const void *__restrict__ sc,
                                           int K, int row, int k, bool valid, int scale_idx)
{
    if (valid) {
        const u32x4 *p = reinterpret_cast<const u32x4 *>(mat + ((size_t)row * K + k) * WTraits<FMT>::kNum /
                                                                   WTraits<FMT>::kDen);
#pragma unroll
        for (int i = 0; i < WTraits<FMT>::kVecs; ++i) f.v[i] = __builtin_nontemporal_load(p + i);
        if constexpr (FMT == FMT_MXFP4)
            f.scale = e8m0_to_f32(static_cast<const uint8_t *>(sc)[(size_t)row * (K / 32) + k / 32]);
    } else {
#pragma unroll
        for (int i = 0; i < WTraits<FMT>::kVecs; ++i) f.v[i] = u32x4{0u, 0u, 0u, 0u};
        if constexpr (FMT == FMT_MXFP4) f.scale = 0.f;
    }
    if constexpr (FMT == FMT_FP8) f.scale = static_cast<const float *>(sc)[scale_idx];
}

// bf16 A operand for sub-step s (weights 8s .. 8s+7 of the lane's 32).
template <int FMT>
__device__ __forceinline__ bf16x8 decode_a(const WFrag<FMT> &f, int s)
{
    if constexpr (FMT == FMT_BF16) {
        return __builtin_bit_cast(bf16x8, f.v[s]);
    } else if constexpr (FMT == FMT_FP8) {
        const uint32_t w0 = f.v[s >> 1][(s & 1) * 2], w1 = f.v[s >> 1][(s & 1) * 2 + 1];
        u32x4 o;
        o[0] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w0, 1.0f, false));
        o[1] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w0, 1.0f, true));
        o[2] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w1, 1.0f, false));
        o[3] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w1, 1.0f, true));
        return __builtin_bit_cast(bf16x8, o);
    } else {
        const uint32_t w = f.v[0][s];
        u32x4 o;
        o[0] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, f.scale, 0));
        o[1] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, f.scale, 1));
        o[2] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, f.scale, 2));
        o[3] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, f.scale, 3));
        return __builtin_bit_cast(bf16x8, o);
    }
}

// 32 consecutive bf16 activations of one token row (B operand for all 4 sub-steps).
struct BFrag {
    u32x4 v[4];
};

__device__ __forceinline__ void load_bfrag(BFrag &b, const uint16_t *__restrict__ rowp, int k, bool valid)
{
    if (valid) {
        const u32x4 *p = reinterpret_cast<const u32x4 *>(rowp + k);
#pragma unroll
        for (int i = 0; i < 4; ++i) b.v[i] = p[i];
    } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) b.v[i] = u32x4{0u, 0u, 0u, 0u};
    }
}

// ----------------------------------------------------------------------------- one expert band

// Which expert / rows / tokens a work item covers.
struct Item {
    const uint8_t *wa, *wb;  // weight matrices of the expert (gate/up: both; down: wa)
    const void *sa, *sb;     // their scales
    int p0;                  // first grouped position of the expert's tokens
    int M;                   // number of tokens routed to it
    bool shared;             // shared expert: positions T*k + t, gate weight 1
};

struct FfnParams {
    VerifyArgs a;
    int N, K;            // rows and reduction length of the streamed matrices
    int rows_per_item;   // 16 (gate/up) or 32 (down)
    int items_per_expert;
};

__device__ __forceinline__ Item make_item(const FfnParams &P, int u, int U, bool down)
{
    const VerifyArgs &a = P.a;
    Item it;
    const size_t mat_bytes = (size_t)P.N * P.K * (a.fmt == FMT_BF16 ? 2 : 1) / (a.fmt == FMT_MXFP4 ? 2 : 1);
    const size_t sc_elems = a.fmt == FMT_FP8 ? (size_t)(P.N / 128) * (P.K / 128)
                                             : a.fmt == FMT_MXFP4 ? (size_t)P.N * (P.K / 32) : 0;
    const size_t sc_bytes = sc_elems * (a.fmt == FMT_FP8 ? 4 : 1);
    if (u < U) {
        const int e = a.union_ids[u];
        it.p0 = a.offsets[u];
        it.M = a.offsets[u + 1] - it.p0;
        it.shared = false;
        if (!down) {
            it.wa = a.w_gate + (size_t)e * mat_bytes;
            it.wb = a.w_up + (size_t)e * mat_bytes;
            it.sa = a.s_gate ? static_cast<const uint8_t *>(a.s_gate) + (size_t)e * sc_bytes : nullptr;
            it.sb = a.s_up ? static_cast<const uint8_t *>(a.s_up) + (size_t)e * sc_bytes : nullptr;
        } else {
            it.wa = it.wb = a.w_down + (size_t)e * mat_bytes;
            it.sa = it.sb = a.s_down ? static_cast<const uint8_t *>(a.s_down) + (size_t)e * sc_bytes : nullptr;
        }
    } else {
        it.p0 = a.T * a.k;
        it.M = a.T;
        it.shared = true;
        if (!down) {
            it.wa = a.sh_gate;
            it.wb = a.sh_up;
            it.sa = a.sh_s_gate;
            it.sb = a.sh_s_up;
        } else {
            it.wa = it.wb = a.sh_down;
            it.sa = it.sb = a.sh_s_down;
        }
    }
    return it;
}

// Stream rows [n0, n0 + 16*NT) of the item's matrices over K for the tokens
// [mg, mg + 16*MB) of the expert; NT A-tiles per wave:
//   gate/up: tile 0 = gate rows, tile 1 = up rows (n0 .. n0+15);
//   down:    tiles 0, 1 = rows n0 .. n0+15, n0+16 .. n0+31.
template <int FMT, bool DOWN, int MB, int PD>
__device__ void run_band(const FfnParams &P, const Item &it, int n0, int mg)
{
    constexpr int NT = 2;
    const VerifyArgs &a = P.a;
    const int lane = lane_id(), col = lane & 15, grp = lane >> 4;
    const int K = P.K;
    const int nsteps = (K + kMacroK - 1) / kMacroK;

    // B rows: token block mb, column col.
    const uint16_t *brow[MB];
    bool bok[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
        const int r = mg + mb * 16 + col;
        bok[mb] = r < it.M;
        const int p = it.p0 + (bok[mb] ? r : 0);
        if (!DOWN) {
            const int tok = it.shared ? (p - a.T * a.k) : (a.perm[p] / a.k);
            brow[mb] = a.x + (size_t)tok * a.d;
        } else {
            brow[mb] = a.h + (size_t)p * a.d_ff;
        }
    }
    // A rows of each tile.
    int arow[NT];
    const uint8_t *amat[NT];
    const void *asc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        amat[t] = (!DOWN && t == 1) ? it.wb : it.wa;
        asc[t] = (!DOWN && t == 1) ? it.sb : it.sa;
        arow[t] = n0 + (DOWN ? t * 16 : 0) + col;
    }
    const int sc_row = (n0 / 128) * (K / 128);  // FP8: block row of the band (bands never straddle 128 rows)

    f32x4 acc[NT][MB];
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) acc[t][mb] = f32x4{0.f, 0.f, 0.f, 0.f};

    WFrag<FMT> wf[PD][NT];
    BFrag bf[2][MB];

    auto issue_a = [&](int slot, int step) {
        const int k = step * kMacroK + grp * 32;
        const bool ok = step < nsteps && k < K;
#pragma unroll
        for (int t = 0; t < NT; ++t) load_wfrag<FMT>(wf[slot][t], amat[t], asc[t], K, arow[t], ok ? k : 0, ok,
                                                     sc_row + (step < nsteps ? step : 0));
    };
    auto issue_b = [&](int slot, int step) {
        const int k = step * kMacroK + grp * 32;
        const bool ok = step < nsteps && k < K;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) load_bfrag(bf[slot][mb], brow[mb], ok ? k : 0, ok && bok[mb]);
    };

#pragma unroll
    for (int s = 0; s < PD - 1; ++s) issue_a(s, s);
    issue_b(0, 0);

    // Unrolled by a multiple of PD and 2 so every ring-buffer index is static.
    constexpr int UNR = (PD % 2 == 0) ? PD : 2 * PD;
    for (int step0 = 0; step0 < nsteps; step0 += UNR) {
#pragma unroll
        for (int j = 0; j < UNR; ++j) {
            const int step = step0 + j;
            if (step < nsteps) {
                // Prefetch: A for step + PD - 1, B for step + 1.
                issue_a((j + PD - 1) % PD, step + PD - 1);
                issue_b((j + 1) & 1, step + 1);
                const WFrag<FMT>(&w)[NT] = wf[j % PD];
                const BFrag(&b)[MB] = bf[j & 1];
                if constexpr (FMT == FMT_FP8) {
                    f32x4 part[NT][MB];
#pragma unroll
                    for (int s = 0; s < 4; ++s)
#pragma unroll
                        for (int t = 0; t < NT; ++t) {
                            const bf16x8 av = decode_a<FMT>(w[t], s);
#pragma unroll
                            for (int mb = 0; mb < MB; ++mb)
                                part[t][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                    av, __builtin_bit_cast(bf16x8, b[mb].v[s]),
                                    s == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : part[t][mb], 0, 0, 0);
                        }
#pragma unroll
                    for (int t = 0; t < NT; ++t)
#pragma unroll
                        for (int mb = 0; mb < MB; ++mb) acc[t][mb] += w[t].scale * part[t][mb];
                } else {
#pragma unroll
                    for (int s = 0; s < 4; ++s)
#pragma unroll
                        for (int t = 0; t < NT; ++t) {
                            const bf16x8 av = decode_a<FMT>(w[t], s);
#pragma unroll
                            for (int mb = 0; mb < MB; ++mb)
                                acc[t][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                    av, __builtin_bit_cast(bf16x8, b[mb].v[s]), acc[t][mb], 0, 0, 0);
                        }
                }
            }
        }
    }

    // Epilogue.  Lane (col, grp) holds rows 4*grp .. 4*grp+3 of each tile for token column col.
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
        if (!bok[mb]) continue;
        const int p = it.p0 + mg + mb * 16 + col;
        if (!DOWN) {
            const f32x4 g = acc[0][mb], v = acc[1][mb];
            uint32_t h2[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const float g0 = g[2 * i], g1 = g[2 * i + 1];
                const float h0 = g0 / (1.f + expf(-g0)) * v[2 * i];
                const float h1 = g1 / (1.f + expf(-g1)) * v[2 * i + 1];
                h2[i] = pack_bf16x2(h0, h1);
            }
            *reinterpret_cast<u32x2 *>(a.h + (size_t)p * a.d_ff + n0 + 4 * grp) = u32x2{h2[0], h2[1]};
        } else {
            const int slot = it.shared ? p : a.perm[p];
            const float gw = it.shared ? 1.f : a.topk_w[slot];
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const f32x4 o = gw * acc[t][mb];
                *reinterpret_cast<f32x4 *>(a.o + (size_t)slot * a.d + n0 + t * 16 + 4 * grp) = o;
            }
        }
    }
}

template <int FMT, bool DOWN, int PD>
__global__ __launch_bounds__(64) void expert_ffn_kernel(FfnParams P)
{
    const VerifyArgs &a = P.a;
    const int U = *a.n_unique;
    const int n_exp = U + (a.sh_gate != nullptr ? 1 : 0);
    const int n_items = n_exp * P.items_per_expert;
    for (int item = blockIdx.x; item < n_items; item += gridDim.x) {
        const int u = item / P.items_per_expert;
        const int n0 = (item - u * P.items_per_expert) * P.rows_per_item;
        const Item it = make_item(P, u, U, DOWN);
        for (int mg = 0; mg < it.M; mg += 16 * kMaxMB) {
            const int rem = it.M - mg;
            const int mb = rem > 16 ? 2 : 1;
            if (mb == 1)
                run_band<FMT, DOWN, 1, PD>(P, it, n0, mg);
            else
                run_band<FMT, DOWN, 2, PD>(P, it, n0, mg);
        }
    }
}

// y[t] = sum_j O[t*k + j] (+ O[T*k + t]) -> bf16; 4 columns per thread.
__global__ __launch_bounds__(256) void combine_kernel(const float *__restrict__ o, int T, int k, int d, int shared,
                                                      uint16_t *__restrict__ y)
{
    const int per_row = d / 4;
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= T * per_row) return;
    const int t = i / per_row, c = (i - t * per_row) * 4;
    f32x4 s = *reinterpret_cast<const f32x4 *>(o + (size_t)(t * k) * d + c);
    for (int j = 1; j < k; ++j) s += *reinterpret_cast<const f32x4 *>(o + (size_t)(t * k + j) * d + c);
    if (shared) s += *reinterpret_cast<const f32x4 *>(o + (size_t)(T * k + t) * d + c);
    *reinterpret_cast<u32x2 *>(y + (size_t)t * d + c) = u32x2{pack_bf16x2(s[0], s[1]), pack_bf16x2(s[2], s[3])};
}

// ----------------------------------------------------------------------------- host side

static int device_cus()
{
    static thread_local int cached_dev = -1, cached_cus = 0;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 256;
    if (dev != cached_dev) {
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
            cus = 256;
        cached_dev = dev;
        cached_cus = cus;
    }
    return cached_cus;
}

VerifyWorkspace verify_workspace(int d, int d_ff, int T, int k, bool shared)
{
    auto align = [](size_t v) { return (v + 255) & ~(size_t)255; };
    const size_t rows = (size_t)T * k + (shared ? (size_t)T : 0);
    VerifyWorkspace w;
    w.h_offset = 0;
    w.h_bytes = rows * d_ff * 2;
    w.o_offset = align(w.h_bytes);
    w.o_bytes = rows * d * 4;
    w.total = w.o_offset + align(w.o_bytes);
    return w;
}

template <int FMT>
static hipError_t launch_fmt(const VerifyArgs &a, hipStream_t stream)
{
    constexpr int PD = FMT == FMT_BF16 ? 2 : FMT == FMT_FP8 ? 3 : 4;
    const int n_exp_max = a.E + (a.sh_gate ? 1 : 0);
    const int grid_cap = device_cus() * kWavesPerCU;

    FfnParams g{};
    g.a = a;
    g.N = a.d_ff;
    g.K = a.d;
    g.rows_per_item = 16;
    g.items_per_expert = a.d_ff / 16;
    int grid = n_exp_max * g.items_per_expert;
    if (grid > grid_cap) grid = grid_cap;
    hipLaunchKernelGGL((expert_ffn_kernel<FMT, false, PD>), dim3(grid), dim3(64), 0, stream, g);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;

    FfnParams dn{};
    dn.a = a;
    dn.N = a.d;
    dn.K = a.d_ff;
    dn.rows_per_item = 32;
    dn.items_per_expert = a.d / 32;
    grid = n_exp_max * dn.items_per_expert;
    if (grid > grid_cap) grid = grid_cap;
    hipLaunchKernelGGL((expert_ffn_kernel<FMT, true, PD>), dim3(grid), dim3(64), 0, stream, dn);
    err = hipGetLastError();
    if (err != hipSuccess) return err;

    const int n = a.T * (a.d / 4);
    hipLaunchKernelGGL(combine_kernel, dim3((n + 255) / 256), dim3(256), 0, stream, a.o, a.T, a.k, a.d,
                       a.sh_gate ? 1 : 0, a.y);
    return hipGetLastError();
}

hipError_t launch_verify(const VerifyArgs &a, hipStream_t stream)
{
    switch (a.fmt) {
    case FMT_BF16: return launch_fmt<FMT_BF16>(a, stream);
    case FMT_FP8: return launch_fmt<FMT_FP8>(a, stream);
    case FMT_MXFP4: return launch_fmt<FMT_MXFP4>(a, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace ecospec
