// Grouped SwiGLU experts of the verification pass on gfx950 (CDNA4).
//
// The pass is bound by HBM bandwidth: every distinct expert routed to by the
// verified tokens must be read once, while each weight serves only the M_u
// tokens routed to its expert (at most 2*M_u flop per weight).  The kernels
// are weight streams with a small matrix-core contraction attached.
//
// Work decomposition ("stream-K").  An item is one expert, one band of rows
// and one group of up to 64 of the expert's tokens: gate/up bands are 16
// rows of W_gate together with the same 16 rows of W_up, down bands are 32
// rows of W_down.  An item is a sequence of K macro steps of 128 reduction
// elements.  All (item, step) units of a launch are laid end to end and cut
// into equal contiguous ranges, one per wavefront of a persistent grid (one
// wavefront per SIMD), so every wavefront streams the same number of bytes
// whatever the number of distinct experts.  A wavefront that covers a whole
// item finishes it in registers; an item cut between wavefronts leaves fp32
// partial sums in the workspace and a second, small kernel adds them in
// wavefront order and finishes it (the kernel boundary makes the partials
// visible across the chip's L2 slices; the fixed order makes the result
// deterministic).
//
// Streaming.  Weights are read in the packed layout (pack.hip): each macro
// step of a 16-row tile is 1-4 KiB of contiguous memory, fetched with 16-byte
// buffer loads that already form the A operand of v_mfma_f32_16x16x32_bf16
// (weights on the 16-row side, tokens on the 16-column side).  FP8 and MXFP4
// codes are decoded exactly to bf16 in registers (v_cvt_scalef32_pk_bf16_fp8
// with unit scale; v_cvt_scalef32_pk_bf16_fp4 with the e8m0 power of two); FP8
// 128x128 block scales multiply the fp32 partial sum of each macro step (one
// step lies inside one scale block).  Several macro steps are in flight per
// wavefront and the prefetch runs across item boundaries.  Loads that fall
// outside a buffer's range (padding tokens, K tails, the end of a range)
// return zeros, so the loop has no data-dependent branches around loads.
//
// Everything the streaming kernels index is either arithmetic on the grouped
// position p (rows of the expert's tokens are contiguous in grouped order) or
// a wave-uniform value read with scalar loads, so no vector load ever waits
// on metadata (a vector-memory wait is in order and would drain the weight
// prefetch).  A gather kernel first copies x into grouped order (xg) and
// records each slot's grouped position; the B operand is then xg rows for
// gate/up and rows of the bf16 SwiGLU output H for down.  Down writes one fp32
// row per grouped position; the combine kernel applies the gate weights and
// sums a token's k slots, then the shared expert, in a fixed order.
#include "device.hpp"
#include "launch.hpp"

// Compile-time tuning: macro steps in flight per wavefront (ring depth) for
// items of <= 16 tokens (PD1) and of up to 64 tokens (PD4), per format.
#ifndef ECOSPEC_PD1_BF16
#define ECOSPEC_PD1_BF16 4
#endif
#ifndef ECOSPEC_PD1_FP8
#define ECOSPEC_PD1_FP8 6
#endif
#ifndef ECOSPEC_PD1_FP4
#define ECOSPEC_PD1_FP4 8
#endif
#ifndef ECOSPEC_PD4_BF16
#define ECOSPEC_PD4_BF16 2
#endif
#ifndef ECOSPEC_PD4_FP8
#define ECOSPEC_PD4_FP8 3
#endif
#ifndef ECOSPEC_PD4_FP4
#define ECOSPEC_PD4_FP4 3
#endif

namespace ecospec {

enum { FMT_BF16 = 0, FMT_FP8 = 1, FMT_MXFP4 = 2 };

constexpr int kMacroK = 128;            // reduction elements per macro step
constexpr int kMB = 4;                  // 16-token blocks per item
constexpr int kTokGroup = 16 * kMB;     // tokens per item
constexpr int kWavesPerCU = 4;          // one wavefront per SIMD
constexpr uint32_t kOff = 0x80000000u;  // buffer offset beyond every range: the load returns zeros
constexpr int kAuxNT = 2;               // nontemporal: streamed weights should not displace activations
constexpr int kPartialFloats = 2 * kMB * 4 * kWave;  // one wavefront's accumulators

typedef __amdgpu_buffer_rsrc_t rsrc_t;

// Wave-uniform loads through the constant address space: scalar-memory loads
// (s_load), counted apart from the vector loads of the weight stream.
__device__ __forceinline__ int ld_s(const int32_t *p)
{
    return *reinterpret_cast<const __attribute__((address_space(4))) int32_t *>(reinterpret_cast<uintptr_t>(p));
}
__device__ __forceinline__ float ld_s(const float *p)
{
    return *reinterpret_cast<const __attribute__((address_space(4))) float *>(reinterpret_cast<uintptr_t>(p));
}

// Raw buffer descriptor over [p, p + bytes): loads at offsets >= bytes return 0.
__device__ __forceinline__ rsrc_t make_rsrc(const void *p, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), 0, (int)bytes, 0x00020000);
}

template <int AUX>
__device__ __forceinline__ u32x4 load16(rsrc_t r, uint32_t off)
{
    return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, AUX));
}

template <int FMT> struct Fmt;
template <> struct Fmt<FMT_BF16>  { static constexpr int kVecs = 4; };
template <> struct Fmt<FMT_FP8>   { static constexpr int kVecs = 2; };
template <> struct Fmt<FMT_MXFP4> { static constexpr int kVecs = 1; };

// One lane's 32 weights of one macro step of one tile (+ their scale).
template <int FMT> struct WFrag {
    u32x4 v[Fmt<FMT>::kVecs];
    float scale;  // FP8: the 128x128 block scale; MXFP4: 2^(e8m0 - 127)
};

__device__ __forceinline__ float e8m0_to_f32(uint32_t code)
{
    // 2^(code-127); code 0 is the subnormal 2^-127, code 255 is NaN.
    return code == 0u ? __uint_as_float(0x00400000u) : code == 255u ? __uint_as_float(0x7fc00000u)
                                                                      : __uint_as_float(code << 23);
}

// bf16 A operand of sub-step s (the lane's weights 8s .. 8s+7 of the step).
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

// 32 consecutive bf16 activations of one token row: B operand of the 4 sub-steps.
struct BFrag {
    u32x4 v[4];
};

// ----------------------------------------------------------------------------- launch geometry

struct FfnParams {
    VerifyArgs a;
    int N, K;          // rows and reduction length of one streamed matrix
    int nsteps;        // macro steps per item: ceil(K / 128)
    int nbands;        // bands per expert: N / 16 (gate/up) or N / 32 (down)
    int workers;       // wavefronts of the main kernel's grid
    float *partials;   // [workers][2][kPartialFloats]
    const int32_t *plan;  // token groups by class (see gather_kernel)
    int plan_cap;         // capacity of each group list
};

// Token groups of the call, written by the plan block of gather_kernel:
//   plan[0], plan[1]        number of groups of class 0 (<= 16 tokens) and 1 (17..64 tokens)
//   plan[8 + c*2*cap + i]   expert position u of group i of class c
//   plan[8 + c*2*cap + cap + i]  its group index tg within the expert (tokens 64*tg ...)
// Class-0 groups come first in the unit space, then class-1 groups; a group
// contributes nbands items of nsteps units each.
struct Plan {
    int U, n0, n1;
};

__device__ __forceinline__ Plan load_plan(const FfnParams &P)
{
    Plan pl;
    pl.U = ld_s(P.a.n_unique);
    pl.n0 = ld_s(P.plan);
    pl.n1 = ld_s(P.plan + 1);
    return pl;
}

__device__ __forceinline__ int expert_tokens(const VerifyArgs &a, int u, int U)
{
    return u < U ? ld_s(a.offsets + u + 1) - ld_s(a.offsets + u) : a.T;
}

// Unit range [x0, x1) of wavefront w: equal shares of n units.
__device__ __forceinline__ void worker_range(long n, int w, int workers, long &x0, long &x1)
{
    x0 = n * w / workers;
    x1 = n * (w + 1) / workers;
}

// Wavefront whose range holds unit x.
__device__ __forceinline__ int owner_of(long n, long x, int workers)
{
    return (int)(((x + 1) * workers - 1) / n);
}

// What a wavefront needs to know about one item.
struct ItemDesc {
    const uint8_t *wa, *wb;  // tile 0 / tile 1 matrices of the expert (packed)
    const void *sa, *sb;     // their scales
    int rb0, rb1;            // block rows of tile 0 / tile 1
    int p0;                  // grouped position of the group's first token
    int M;                   // tokens in the group (<= 64)
    bool shared;
};

template <bool DOWN>
__device__ __forceinline__ ItemDesc describe(const FfnParams &P, const Plan &pl, int item)
{
    const VerifyArgs &a = P.a;
    const int i0 = pl.n0 * P.nbands;
    const int cls = item >= i0 ? 1 : 0;
    const int local = item - cls * i0;
    const int gi = local / P.nbands, band = local - gi * P.nbands;
    const int32_t *lst = P.plan + 8 + cls * 2 * P.plan_cap;
    const int u = ld_s(lst + gi), tg = ld_s(lst + P.plan_cap + gi);
    const int fmt = a.fmt;
    const size_t kp = (size_t)P.nsteps * kMacroK;
    const size_t mat = (size_t)P.N * kp * (fmt == FMT_BF16 ? 2 : 1) / (fmt == FMT_MXFP4 ? 2 : 1);
    const size_t sc = fmt == FMT_FP8 ? (size_t)(P.N / 128) * (P.K / 128) * 4 : fmt == FMT_MXFP4 ? (size_t)P.N * kp / 32 : 0;
    ItemDesc d;
    d.shared = u >= pl.U;
    const int M = expert_tokens(a, u, pl.U);
    d.p0 = (d.shared ? a.T * a.k : ld_s(a.offsets + u)) + tg * kTokGroup;
    d.M = min(kTokGroup, M - tg * kTokGroup);
    const size_t e = d.shared ? 0 : (size_t)ld_s(a.union_ids + u);
    auto sptr = [&](const void *base) {
        return base ? static_cast<const void *>(static_cast<const uint8_t *>(base) + e * sc) : nullptr;
    };
    if (!DOWN) {
        d.wa = (d.shared ? a.sh_gate : a.w_gate) + e * mat;
        d.wb = (d.shared ? a.sh_up : a.w_up) + e * mat;
        d.sa = d.shared ? a.sh_s_gate : sptr(a.s_gate);
        d.sb = d.shared ? a.sh_s_up : sptr(a.s_up);
        d.rb0 = d.rb1 = band;
    } else {
        d.wa = d.wb = (d.shared ? a.sh_down : a.w_down) + e * mat;
        d.sa = d.sb = d.shared ? a.sh_s_down : sptr(a.s_down);
        d.rb0 = 2 * band;
        d.rb1 = 2 * band + 1;
    }
    return d;
}

// ----------------------------------------------------------------------------- epilogue

// Finishes the (tile 0, tile 1) accumulators of an item: gate/up -> bf16
// SwiGLU rows of H; down -> fp32 rows of O (both at grouped positions).
// Lane (col, grp) holds rows 4*grp .. 4*grp+3 of a tile for token column col.
template <bool DOWN, int MB>
__device__ __forceinline__ void finish_item(const FfnParams &P, const ItemDesc &d, int band,
                                            const f32x4 (&acc)[2][MB])
{
    const VerifyArgs &a = P.a;
    const int lane = lane_id(), col = lane & 15, grp = lane >> 4;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
        const int r = mb * 16 + col;
        if (r >= d.M) continue;
        const int p = d.p0 + r;
        if (!DOWN) {
            const f32x4 g = acc[0][mb], v = acc[1][mb];
            uint32_t h2[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const float g0 = g[2 * i], g1 = g[2 * i + 1];
                h2[i] = pack_bf16x2(g0 / (1.f + expf(-g0)) * v[2 * i], g1 / (1.f + expf(-g1)) * v[2 * i + 1]);
            }
            *reinterpret_cast<u32x2 *>(a.h + (size_t)p * a.d_ff + band * 16 + 4 * grp) = u32x2{h2[0], h2[1]};
        } else {
#pragma unroll
            for (int t = 0; t < 2; ++t)
                *reinterpret_cast<f32x4 *>(a.o + (size_t)p * a.d + band * 32 + t * 16 + 4 * grp) = acc[t][mb];
        }
    }
}

// ----------------------------------------------------------------------------- main kernel

// Streams units [xs, xe) (all in one token-group class, MB 16-token blocks)
// of wavefront w, whose whole range is [x0, x1).  A and B operands of a unit
// are issued together, PD-1 units ahead of the unit being computed: the
// vector-memory counter retires loads in issue order, so loads must be
// consumed in the order they were issued for the prefetch to stay deep.
template <int FMT, bool DOWN, int MB, int PD>
__device__ __forceinline__ void run_range(const FfnParams &P, const Plan &pl, long xs, long xe, long x0, long x1,
                                          int w)
{
    constexpr int NV = Fmt<FMT>::kVecs;
    constexpr uint32_t BLK = 1024u * NV;  // bytes of one 16 x 128 block
    const VerifyArgs &a = P.a;
    const int lane = lane_id(), col = lane & 15, grp = lane >> 4;
    const int K = P.K, nsteps = P.nsteps;

    // B rows at grouped positions: xg (gate/up) or H (down).
    const uint32_t brow_bytes = (uint32_t)(DOWN ? a.d_ff : a.d) * 2u;
    const uint32_t n_rows = (uint32_t)(a.T * a.k + (a.sh_gate ? a.T : 0));
    const rsrc_t rbuf = make_rsrc(DOWN ? (const void *)a.h : (const void *)a.xg, n_rows * brow_bytes);
    const uint32_t mat_bytes =
        (uint32_t)((size_t)P.N * nsteps * kMacroK * (FMT == FMT_BF16 ? 2 : 1) / (FMT == FMT_MXFP4 ? 2 : 1));
    const uint32_t msc_bytes = (uint32_t)((size_t)P.N * nsteps * 4);  // MXFP4 packed scales

    // Load cursor (PD-1 units ahead of the compute cursor).  The descriptor of
    // the item after the load cursor's is fetched one item early, so that its
    // scalar loads have long landed when the cursor gets there.
    long xl = xs;
    int il = (int)(xs / nsteps), sl = (int)(xs - (long)il * nsteps);
    const int i_last = (int)((xe - 1) / nsteps);
    ItemDesc dl = describe<DOWN>(P, pl, il);
    ItemDesc dn = il < i_last ? describe<DOWN>(P, pl, il + 1) : dl;
    ItemDesc dprev = dl;  // the load cursor's previous item (the compute cursor may still be in it)
    const uint32_t fsc_bytes = (uint32_t)((P.N / 128) * (K / 128) * 4);  // FP8 scales of one matrix
    rsrc_t ra0 = make_rsrc(dl.wa, mat_bytes), ra1 = make_rsrc(dl.wb, mat_bytes);
    rsrc_t rs0 = make_rsrc(dl.sa, FMT == FMT_FP8 ? fsc_bytes : msc_bytes);
    rsrc_t rs1 = make_rsrc(dl.sb, FMT == FMT_FP8 ? fsc_bytes : msc_bytes);
    uint32_t boff[MB];
    auto b_rows = [&]() {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
            const int r = mb * 16 + col;
            boff[mb] = r < dl.M ? (uint32_t)(dl.p0 + r) * brow_bytes + (uint32_t)grp * 64u : kOff;
        }
    };
    b_rows();
    // Compute cursor.
    int ic = il, sc = sl;
    ItemDesc dc = dl;

    WFrag<FMT> wf[PD][2];
    BFrag bf[PD][MB];
    f32x4 acc[2][MB];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) acc[t][mb] = f32x4{0.f, 0.f, 0.f, 0.f};

    // A, scale and B loads of the load cursor's unit into ring slot `slot`
    // (all vector-memory loads, retired in issue order); advance the cursor.
    auto issue = [&](int slot) {
        const bool ok = xl < xe;
        const uint32_t o0 = ok ? ((uint32_t)dl.rb0 * nsteps + sl) * BLK + lane * 16u : kOff;
        const uint32_t o1 = ok ? ((uint32_t)dl.rb1 * nsteps + sl) * BLK + lane * 16u : kOff;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            wf[slot][0].v[i] = load16<kAuxNT>(ra0, o0 + 1024u * i);
            wf[slot][1].v[i] = load16<kAuxNT>(ra1, o1 + 1024u * i);
        }
        if constexpr (FMT == FMT_FP8) {
            // One block scale per tile and step; every lane reads the same word.
            const uint32_t q0 = ok ? ((uint32_t)(dl.rb0 / 8) * (K / 128) + sl) * 4u : kOff;
            const uint32_t q1 = ok ? ((uint32_t)(dl.rb1 / 8) * (K / 128) + sl) * 4u : kOff;
            wf[slot][0].scale = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs0, (int)q0, 0, 0));
            wf[slot][1].scale = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs1, (int)q1, 0, 0));
        } else if constexpr (FMT == FMT_MXFP4) {
            const uint32_t q0 = ok ? ((uint32_t)dl.rb0 * nsteps + sl) * 64u + lane : kOff;
            const uint32_t q1 = ok ? ((uint32_t)dl.rb1 * nsteps + sl) * 64u + lane : kOff;
            wf[slot][0].scale = e8m0_to_f32(__builtin_amdgcn_raw_buffer_load_b8(rs0, (int)q0, 0, 0));
            wf[slot][1].scale = e8m0_to_f32(__builtin_amdgcn_raw_buffer_load_b8(rs1, (int)q1, 0, 0));
        }
        const int k = sl * kMacroK + grp * 32;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
            const uint32_t o = (ok && k < K && boff[mb] != kOff) ? boff[mb] + (uint32_t)sl * (kMacroK * 2) : kOff;
#pragma unroll
            for (int i = 0; i < 4; ++i) bf[slot][mb].v[i] = load16<0>(rbuf, o + 16u * i);
        }
        ++xl;
        if (++sl == nsteps && xl < xe) {  // entering the next item
            sl = 0;
            ++il;
            dprev = dl;
            dl = dn;
            if (il < i_last) dn = describe<DOWN>(P, pl, il + 1);
            ra0 = make_rsrc(dl.wa, mat_bytes);
            ra1 = make_rsrc(dl.wb, mat_bytes);
            rs0 = make_rsrc(dl.sa, FMT == FMT_FP8 ? fsc_bytes : msc_bytes);
            rs1 = make_rsrc(dl.sb, FMT == FMT_FP8 ? fsc_bytes : msc_bytes);
            b_rows();
        }
    };

#pragma unroll
    for (int s = 0; s < PD - 1; ++s) issue(s);

    for (long xc0 = xs; xc0 < xe; xc0 += PD) {
#pragma unroll
        for (int j = 0; j < PD; ++j) {
            const long xc = xc0 + j;
            if (xc < xe) {
                issue((j + PD - 1) % PD);
                const WFrag<FMT>(&wv)[2] = wf[j];
                const BFrag(&bv)[MB] = bf[j];
                const int nmb = (dc.M + 15) / 16;
                if constexpr (FMT == FMT_FP8) {
                    f32x4 part[2][MB];
#pragma unroll
                    for (int s = 0; s < 4; ++s)
#pragma unroll
                        for (int t = 0; t < 2; ++t) {
                            const bf16x8 av = decode_a<FMT>(wv[t], s);
#pragma unroll
                            for (int mb = 0; mb < MB; ++mb)
                                if (MB == 1 || mb < nmb)
                                    part[t][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                        av, __builtin_bit_cast(bf16x8, bv[mb].v[s]),
                                        s == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : part[t][mb], 0, 0, 0);
                        }
#pragma unroll
                    for (int t = 0; t < 2; ++t)
#pragma unroll
                        for (int mb = 0; mb < MB; ++mb)
                            if (MB == 1 || mb < nmb) acc[t][mb] += wv[t].scale * part[t][mb];
                } else {
#pragma unroll
                    for (int s = 0; s < 4; ++s)
#pragma unroll
                        for (int t = 0; t < 2; ++t) {
                            const bf16x8 av = decode_a<FMT>(wv[t], s);
#pragma unroll
                            for (int mb = 0; mb < MB; ++mb)
                                if (MB == 1 || mb < nmb)
                                    acc[t][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                        av, __builtin_bit_cast(bf16x8, bv[mb].v[s]), acc[t][mb], 0, 0, 0);
                        }
                }
                // Last unit of the item inside this range: finish it, or park the partial sums.
                if (sc == nsteps - 1 || xc == xe - 1) {
                    const long ib = (long)ic * nsteps;
                    if (ib >= x0 && ib + nsteps <= x1) {
                        finish_item<DOWN, MB>(P, dc, ic % P.nbands, acc);
                    } else {
                        float *dst = P.partials + ((size_t)w * 2 + (ib <= x0 ? 0 : 1)) * kPartialFloats;
#pragma unroll
                        for (int t = 0; t < 2; ++t)
#pragma unroll
                            for (int mb = 0; mb < MB; ++mb)
                                *reinterpret_cast<f32x4 *>(dst + ((t * kMB + mb) * kWave + lane) * 4) = acc[t][mb];
                    }
#pragma unroll
                    for (int t = 0; t < 2; ++t)
#pragma unroll
                        for (int mb = 0; mb < MB; ++mb) acc[t][mb] = f32x4{0.f, 0.f, 0.f, 0.f};
                    if (xc < xe - 1) {
                        ++ic;
                        sc = 0;
                        dc = ic == il ? dl : ic + 1 == il ? dprev : describe<DOWN>(P, pl, ic);
                    }
                } else {
                    ++sc;
                }
            }
        }
    }
}

template <int FMT, bool DOWN, int PD1, int PD4>
__global__ __launch_bounds__(kWave) __attribute__((amdgpu_waves_per_eu(1, 1))) void expert_ffn_kernel(FfnParams P)
{
    const int w = blockIdx.x;
    const Plan pl = load_plan(P);
    const long bound = (long)pl.n0 * P.nbands * P.nsteps;  // first unit of class 1
    const long n_units = (long)(pl.n0 + pl.n1) * P.nbands * P.nsteps;
    long x0, x1;
    worker_range(n_units, w, P.workers, x0, x1);
    if (x0 < x1 && x0 < bound) run_range<FMT, DOWN, 1, PD1>(P, pl, x0, x1 < bound ? x1 : bound, x0, x1, w);
    if (x0 < x1 && x1 > bound) run_range<FMT, DOWN, kMB, PD4>(P, pl, x0 > bound ? x0 : bound, x1, x0, x1, w);
}

// Finishes the items cut between wavefronts: the wavefront whose range holds
// an item's last unit (but not its first) sums the parked partial sums of
// every owner of the item, in wavefront order.
template <bool DOWN>
__global__ __launch_bounds__(kWave) void expert_ffn_fixup_kernel(FfnParams P)
{
    const int lane = lane_id();
    const int w = blockIdx.x;
    const Plan pl = load_plan(P);
    const long n_units = (long)(pl.n0 + pl.n1) * P.nbands * P.nsteps;
    long x0, x1;
    worker_range(n_units, w, P.workers, x0, x1);
    if (x0 >= x1) return;
    const int item = (int)(x0 / P.nsteps);
    const long ib = (long)item * P.nsteps, ie = ib + P.nsteps;
    if (ib >= x0 || ie > x1) return;  // not cut before this range, or its end lies beyond it
    const int w0 = owner_of(n_units, ib, P.workers);
    f32x4 acc[2][kMB];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int mb = 0; mb < kMB; ++mb) acc[t][mb] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int v = w0; v <= w; ++v) {
        long v0, v1;
        worker_range(n_units, v, P.workers, v0, v1);
        if (v0 >= v1) continue;
        const int slot = (ib <= v0 && v0 < ie) ? 0 : 1;  // the item holds v's first unit, or is v's last item
        const float *src = P.partials + ((size_t)v * 2 + slot) * kPartialFloats;
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int mb = 0; mb < kMB; ++mb)
                acc[t][mb] += *reinterpret_cast<const f32x4 *>(src + ((t * kMB + mb) * kWave + lane) * 4);
    }
    finish_item<DOWN, kMB>(P, describe<DOWN>(P, pl, item), item % P.nbands, acc);
}

// xg[p] = x[token of the slot at grouped position p] and ip[slot] = p for
// the routed rows; xg[T*k + t] = x[t] for the shared expert's rows.  One
// workgroup per row, 16 bytes per thread.  The extra last workgroup writes
// the token-group plan read by the expert kernels: every expert's tokens in
// groups of 64, the groups of <= 16 tokens (class 0) listed apart from the
// others (class 1), each list in expert order.
__global__ __launch_bounds__(256) void gather_kernel(VerifyArgs a, int32_t *plan, int cap)
{
    const int routed = a.T * a.k;
    const int U = ld_s(a.n_unique);
    if (blockIdx.x == gridDim.x - 1) {
        __shared__ int wave_tot[256 / kWave];
        const int n_exp = U + (a.sh_gate ? 1 : 0);
        int32_t *l0u = plan + 8, *l0t = l0u + cap, *l1u = l0t + cap, *l1t = l1u + cap;
        int run0 = 0, run1 = 0;
        for (int base = 0; base < n_exp; base += blockDim.x) {
            const int u = base + threadIdx.x;
            int c0 = 0, c1 = 0, ntg = 0;
            if (u < n_exp) {
                const int M = u < U ? a.offsets[u + 1] - a.offsets[u] : a.T;
                ntg = (M + kTokGroup - 1) / kTokGroup;
                const int last = M - kTokGroup * (ntg - 1);
                c0 = last <= 16 ? 1 : 0;
                c1 = ntg - c0;
            }
            int t0 = 0, t1 = 0;
            const int p0 = block_exclusive_scan(c0, wave_tot, &t0);
            const int p1 = block_exclusive_scan(c1, wave_tot, &t1);
            if (c0) {
                l0u[run0 + p0] = u;
                l0t[run0 + p0] = ntg - 1;
            }
            for (int g = 0; g < c1; ++g) {
                l1u[run1 + p1 + g] = u;
                l1t[run1 + p1 + g] = g;
            }
            run0 += t0;
            run1 += t1;
        }
        if (threadIdx.x == 0) {
            plan[0] = run0;
            plan[1] = run1;
        }
        return;
    }
    const int p = blockIdx.x;
    int t;
    if (p < routed) {
        if (p >= a.offsets[U]) return;  // unfilled position (out-of-range routing entries)
        const int slot = a.perm[p];
        t = slot / a.k;
        if (threadIdx.x == 0) a.ip[slot] = p;
    } else {
        t = p - routed;
    }
    const u32x4 *src = reinterpret_cast<const u32x4 *>(a.x + (size_t)t * a.d);
    u32x4 *dst = reinterpret_cast<u32x4 *>(a.xg + (size_t)p * a.d);
    for (int i = threadIdx.x; i < a.d / 8; i += blockDim.x) dst[i] = src[i];
}

// y[t] = sum_j w[t][j] * O[ip[t*k + j]] (+ O[T*k + t]) -> bf16; 4 columns per thread.
__global__ __launch_bounds__(256) void combine_kernel(VerifyArgs a)
{
    const int per_row = a.d / 4;
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= a.T * per_row) return;
    const int t = i / per_row, c = (i - t * per_row) * 4;
    const uint32_t rows = (uint32_t)(a.T * a.k + (a.sh_gate ? a.T : 0));
    f32x4 s = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int j = 0; j < a.k; ++j) {
        const int slot = t * a.k + j;
        const uint32_t p = (uint32_t)a.ip[slot];
        if (p < rows) s += a.topk_w[slot] * *reinterpret_cast<const f32x4 *>(a.o + (size_t)p * a.d + c);
    }
    if (a.sh_gate) s += *reinterpret_cast<const f32x4 *>(a.o + (size_t)(a.T * a.k + t) * a.d + c);
    *reinterpret_cast<u32x2 *>(a.y + (size_t)t * a.d + c) = u32x2{pack_bf16x2(s[0], s[1]), pack_bf16x2(s[2], s[3])};
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

static int workers()
{
    const int w = device_cus() * kWavesPerCU;
    return w < kMaxWorkers ? w : kMaxWorkers;
}

// Token groups an expert list can hold: one per expert (<= 1024 routed + 1
// shared) plus one per extra 64 tokens.
static int plan_capacity(int T, int k, bool shared)
{
    const long rows = (long)T * k + (shared ? T : 0);
    return (int)(1025 + (rows + kTokGroup - 1) / kTokGroup);
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
    w.p_offset = w.o_offset + align(w.o_bytes);
    w.p_bytes = (size_t)kMaxWorkers * 2 * kPartialFloats * 4;
    w.x_offset = w.p_offset + align(w.p_bytes);
    w.x_bytes = rows * d * 2;
    w.i_offset = w.x_offset + align(w.x_bytes);
    w.i_bytes = (size_t)T * k * 4;
    w.plan_cap = plan_capacity(T, k, shared);
    w.plan_offset = w.i_offset + align(w.i_bytes);
    w.plan_bytes = (8 + 4 * (size_t)w.plan_cap) * 4;
    w.total = w.plan_offset + align(w.plan_bytes);
    return w;
}

static hipError_t mark(hipEvent_t const *events, int i, hipStream_t stream)
{
    return (events && events[i]) ? hipEventRecord(events[i], stream) : hipSuccess;
}

template <int FMT>
static hipError_t launch_fmt(const VerifyArgs &a, float *partials, int32_t *plan, int plan_cap, hipStream_t stream,
                             hipEvent_t const *events)
{
    constexpr int PD1 = FMT == FMT_BF16 ? ECOSPEC_PD1_BF16 : FMT == FMT_FP8 ? ECOSPEC_PD1_FP8 : ECOSPEC_PD1_FP4;
    constexpr int PD4 = FMT == FMT_BF16 ? ECOSPEC_PD4_BF16 : FMT == FMT_FP8 ? ECOSPEC_PD4_FP8 : ECOSPEC_PD4_FP4;
    const int G = workers();
    hipError_t err;

    FfnParams g{};
    g.a = a;
    g.N = a.d_ff;
    g.K = a.d;
    g.nsteps = (a.d + kMacroK - 1) / kMacroK;
    g.nbands = a.d_ff / 16;
    g.workers = G;
    g.partials = partials;
    g.plan = plan;
    g.plan_cap = plan_cap;
    const int rows = a.T * a.k + (a.sh_gate ? a.T : 0);
    if ((err = mark(events, 0, stream)) != hipSuccess) return err;
    hipLaunchKernelGGL(gather_kernel, dim3(rows + 1), dim3(256), 0, stream, a, plan, plan_cap);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    hipLaunchKernelGGL((expert_ffn_kernel<FMT, false, PD1, PD4>), dim3(G), dim3(kWave), 0, stream, g);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    hipLaunchKernelGGL((expert_ffn_fixup_kernel<false>), dim3(G), dim3(kWave), 0, stream, g);
    if ((err = hipGetLastError()) != hipSuccess) return err;

    FfnParams dn = g;
    dn.N = a.d;
    dn.K = a.d_ff;
    dn.nsteps = (a.d_ff + kMacroK - 1) / kMacroK;
    dn.nbands = a.d / 32;
    if ((err = mark(events, 1, stream)) != hipSuccess) return err;
    hipLaunchKernelGGL((expert_ffn_kernel<FMT, true, PD1, PD4>), dim3(G), dim3(kWave), 0, stream, dn);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    hipLaunchKernelGGL((expert_ffn_fixup_kernel<true>), dim3(G), dim3(kWave), 0, stream, dn);
    if ((err = hipGetLastError()) != hipSuccess) return err;

    const int n = a.T * (a.d / 4);
    if ((err = mark(events, 2, stream)) != hipSuccess) return err;
    hipLaunchKernelGGL(combine_kernel, dim3((n + 255) / 256), dim3(256), 0, stream, a);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    return mark(events, 3, stream);
}

hipError_t launch_verify(const VerifyArgs &a, float *partials, int32_t *plan, int plan_cap, hipStream_t stream,
                         hipEvent_t const *events)
{
    switch (a.fmt) {
    case FMT_BF16: return launch_fmt<FMT_BF16>(a, partials, plan, plan_cap, stream, events);
    case FMT_FP8: return launch_fmt<FMT_FP8>(a, partials, plan, plan_cap, stream, events);
    case FMT_MXFP4: return launch_fmt<FMT_MXFP4>(a, partials, plan, plan_cap, stream, events);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace ecospec
