// Grouped SwiGLU experts of the verification pass on gfx950 (CDNA4).
//
// The pass is bound by HBM bandwidth: every distinct expert routed to by the
// verified tokens must be read once, while each weight serves only the M_u
// tokens routed to its expert (at most 2*M_u flop per weight).  The kernels
// are weight streams with a small matrix-core contraction attached.
//
// Workgroups.  One workgroup per compute unit, eight wavefronts (two per
// SIMD), all on one band of rows of one expert and one group of up to 64 of
// its tokens (an item): gate/up bands are 128 rows of W_gate with the same
// 128 rows of W_up (16 + 16 per wavefront), down bands are 256 rows of W_down
// (32 per wavefront).  All eight walk the reduction dimension together in
// macro steps of 128 elements, so the activation tile of a step (the item's
// tokens x 128 elements) is fetched from L2 once, by 16-byte loads that go
// straight into LDS (no registers, no LDS store instructions), and read there
// by every wavefront.  A single workgroup per CU keeps
// the CU's waves in lockstep: two workgroups sharing a CU drift apart (the
// older one wins instruction issue), which leaves the younger one's share of
// an equal split running alone at the end of the launch.
//
// Streaming.  Weights are read in the packed layout (pack.hip): each macro
// step of a 16-row tile is 1-4 KiB of contiguous memory, fetched with 16-byte
// buffer loads that are already the A operand of v_mfma_f32_16x16x32_bf16
// (weights on the 16-row side, tokens on the 16-column side).  In the paired
// layouts (gate with up, or a down wavefront's two tiles) a wavefront's two
// tiles of a step are one contiguous run.  FP8 and MXFP4
// codes are decoded exactly to bf16 in registers (v_cvt_scalef32_pk_bf16_fp8
// with unit scale; v_cvt_scalef32_pk_bf16_fp4 with the e8m0 power of two); FP8
// 128x128 block scales multiply the fp32 partial sum of each macro step (one
// step lies inside one scale block).  A step's weight and scale loads are
// issued PD-1 steps ahead of its use, its activation loads right after the
// barrier of the step PD-1 before it: the vector-memory counter retires loads
// in issue order, so consuming them in issue order is what keeps PD-1 steps
// in flight, and the barrier wait counts the loads still allowed in flight.
// Loads outside a buffer's range (padding tokens, K tails, rows past N)
// return zeros (into LDS too); the loop has no branches around loads.
//
// Work split ("stream-K").  All (item, step) units of a launch are laid end
// to end and cut into contiguous ranges of equal modelled cost (a step's
// weight bytes plus its contraction work, which grows with the item's token
// blocks), one per workgroup of a persistent grid, so the workgroups finish
// together whatever the number of distinct experts.  An item fully inside a
// range is finished in registers; an item cut between workgroups leaves fp32
// partial sums in the workspace, added in workgroup order by a small fix-up
// kernel (gate/up) or by the combine kernel as it reads O (down): the kernel
// boundary makes them visible across the XCDs' L2 caches, and the fixed order
// keeps the result deterministic.
//
// Outputs: gate/up writes the bf16 SwiGLU rows H at grouped positions; down
// writes one fp32 row per (token, slot); combine applies the gate weights and
// sums a token's k slots, then the shared expert, in a fixed order.
//
// MX activation mode (opt-in, MXFP4 weights): x and H are quantised to OCP MX
// FP8 (x by a small pre-pass, H in the gate/up epilogue) and both projections
// run on v_mfma_scale_f32_16x16x128_f8f6f4 (FP4 weights x FP8 activations,
// e8m0 scales of both applied by the instruction).  A lane of that
// instruction's FP4 operand holds 32 consecutive K of one row, exactly the
// packed MXFP4 fragment and its scale.  The scales of both operands apply to
// the same 32-wide K blocks (lane group g's scale to K 32g..32g+31 of the
// 128), the plain OCP MX blocks; the data of the FP8 operand's lane group g is
// K 16g..16g+15 and 64+16g..64+16g+15, so activation rows are stored in that
// order (each 128-element chunk as four 32-byte lane runs).
#include "device.hpp"
#include "launch.hpp"
#include "split.hpp"

// Compile-time tuning: macro steps in flight per wavefront, per format (each
// the fastest measured: bf16 and MXFP4 steps are 8 KiB per wavefront, MXFP4
// also with the decode's registers; FP8 steps 4 KiB).
#ifndef ECOSPEC_PD_BF16
#define ECOSPEC_PD_BF16 2
#endif
#ifndef ECOSPEC_PD_FP8
#define ECOSPEC_PD_FP8 3
#endif
#ifndef ECOSPEC_PD_FP4
#define ECOSPEC_PD_FP4 2
#endif
#ifndef ECOSPEC_PHYS_WAVES
#define ECOSPEC_PHYS_WAVES 8  // wavefronts of an expert workgroup (8: two per SIMD; 4: one per SIMD, measured slower)
#endif
#ifndef ECOSPEC_WG_PER_CU
#define ECOSPEC_WG_PER_CU 1
#endif

namespace ecospec {

enum { FMT_BF16 = 0, FMT_FP8 = 1, FMT_MXFP4 = 2 };

constexpr int kMacroK = 128;            // reduction elements per macro step
constexpr int kMB = 4;                  // 16-token blocks per item
constexpr int kTokGroup = 16 * kMB;     // tokens per item
// An item's rows are cut into kWG slots: 16 rows (gate/up, with the same
// rows of the up matrix) or 32 rows (down) each.  Slots are the unit of the
// partial-sum layout and of the fix-up kernel (one wavefront per slot); an
// expert workgroup has kPW wavefronts of kVPW slots each, i.e. kNT weight
// tiles of 16 rows per wavefront.
constexpr int kWG = 8;                               // slots per item
constexpr int kPW = ECOSPEC_PHYS_WAVES;              // wavefronts of an expert workgroup
constexpr int kVPW = kWG / kPW;                      // slots per wavefront
constexpr int kNT = 2 * kVPW;                        // 16-row weight tiles per wavefront
constexpr int kThreads = kWG * kWave;                // fix-up kernel
constexpr int kEThreads = kPW * kWave;               // expert kernels
constexpr int kBRowsPerPass = kEThreads / 16;        // activation rows staged per pass (16 threads per row)
constexpr int kBPass = kTokGroup / kBRowsPerPass;    // passes per step
static_assert(kWG % kPW == 0, "whole slots per wavefront");
constexpr int kAuxNT = 2;               // nontemporal: streamed weights should not displace activations
// Floats of one partial-sum slot: a workgroup's accumulators of the live token
// blocks (a token group holds at most min(T, 64) tokens).
constexpr int partial_floats(int T)
{
    return kWG * 2 * 4 * kWave * (((T < kTokGroup ? T : kTokGroup) + 15) / 16);
}

// Wave-uniform loads through the constant address space (scalar memory).
__device__ __forceinline__ int ld_s(const int32_t *p)
{
    return *reinterpret_cast<const __attribute__((address_space(4))) int32_t *>(reinterpret_cast<uintptr_t>(p));
}

__device__ __forceinline__ long long ld_s64(const long long *p)
{
    return *reinterpret_cast<const __attribute__((address_space(4))) long long *>(reinterpret_cast<uintptr_t>(p));
}

// kVecs: 16-byte vectors per lane in one 16 x 128 block of a tile; kBlocks:
// 128-wide K blocks per macro step.  MXFP4 takes two blocks a step, so that a
// step streams 2 KiB per tile like FP8 and pays its fixed per-step work (the
// activation staging, the barrier, the item bookkeeping) over as many bytes.
template <int FMT> struct Fmt;
template <> struct Fmt<FMT_BF16>  { static constexpr int kVecs = 4, kBlocks = 1; };
template <> struct Fmt<FMT_FP8>   { static constexpr int kVecs = 2, kBlocks = 1; };
template <> struct Fmt<FMT_MXFP4> { static constexpr int kVecs = 1, kBlocks = 2; };

// LDS geometry of one step's activation tile: 64 tokens x 128 * SB bf16
// elements, block-major.  Block b of token row r is 256 bytes at
// b * kBlk + r * 256, its 16-byte chunk c stored in position c ^ (r % 16): the
// tile is written by direct global-to-LDS loads, which put a wavefront's 64
// lanes on 1 KiB of consecutive LDS (no room for row padding), and the
// swizzle keeps the matrix-core operand reads free of bank conflicts (16
// consecutive token rows, same chunk: 16 different positions).
template <int SB> struct BTile {
    static constexpr int kBlk = kMB * 16 * 256;  // one 128-wide block of all 64 token rows
    static constexpr int kBuf = SB * kBlk;
};

// One lane's weights of one macro step of one tile (+ their scales).  The
// MXFP4 scales stay raw e8m0 codes until the step is decoded: converting one
// where it is loaded would wait for that load and drain the prefetch.
template <int FMT> struct WFrag {
    u32x4 v[Fmt<FMT>::kVecs * Fmt<FMT>::kBlocks];  // block b's vectors at [b * kVecs ...]
    float scale;                                   // FP8: the 128x128 block scale
    uint32_t code;                                 // MXFP4: the lane's e8m0 codes of a quad of blocks
    int shift;                                     // MXFP4: bit offset of the step's first block in `code`
};

// The scale operand of the scaled conversions (v_cvt_scalef32_*): the
// instruction takes the operand's exponent field as an e8m0 code, so field 0
// scales by 2^-127 and field 255 gives NaN, as the OCP MX definition of the
// code does (checked on the device against the exact scale value for all 256
// codes and all 256 FP4 code pairs: identical results).  The code shifted into
// the exponent field is therefore the operand for every code, with no special
// cases.
__device__ __forceinline__ float e8m0_scale_operand(uint32_t code) { return __uint_as_float((code & 0xffu) << 23); }

// MX FP8 activation quantisation.  A block's scale exponent from its largest
// magnitude: E = floor(log2(amax)) - 8 (448, the largest e4m3fn value, is
// 1.75 * 2^8), -127 for amax = 0 or below the fp32 normal range; E <= 119.
__device__ __forceinline__ int mx_exponent(float amax)
{
    const int ef = (int)((__float_as_uint(amax) >> 23) & 0xffu);
    return ef == 0 ? -127 : max(ef - 135, -127);
}

// 2^-E for a block exponent E in [-127, 119].
__device__ __forceinline__ float mx_inv_scale(int E) { return __uint_as_float((uint32_t)(127 - E) << 23); }

// e4m3fn code of v (already divided by the block scale): nearest value, ties
// to the even code, magnitudes of 448 and above saturating to 448 (code
// 0x7e), subnormals (multiples of 2^-9) kept, NaN to 0x7f.
__device__ __forceinline__ uint32_t e4m3_code(float v)
{
    const uint32_t bits = __float_as_uint(v), sign = (bits >> 24) & 0x80u;
    const float a = __uint_as_float(bits & 0x7fffffffu);
    uint32_t code;
    if (a != a) {
        code = 0x7fu;
    } else if (!(a < 448.f)) {
        code = 0x7eu;
    } else if (a < 0.015625f) {
        code = (uint32_t)__builtin_rintf(a * 512.f);  // 0 .. 8; 8 is 2^-6, the code of the first normal
    } else {
        const uint32_t b = __float_as_uint(a), mant = b & 0x7fffffu;
        const uint32_t r = (mant + 0x7ffffu + ((mant >> 20) & 1u)) >> 20;  // 3-bit mantissa, ties to even
        code = (((b >> 23) - 120u) << 3) + r;  // r = 8 carries into the exponent field
    }
    return sign | code;
}

// bf16 A operand of sub-step s (the lane's weights 8s .. 8s+7 of a block;
// MXFP4: sub-step s of block s / 4).
// Exact: FP8 codes as they are (the converter's scale operand only takes a
// power of two, so the 128x128 block scale multiplies the fp32 partial sum of
// the step instead); MXFP4 codes times their 2^e8m0 group scale.
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
        const uint32_t w = f.v[s >> 2][s & 3];
        const float sc = e8m0_scale_operand(f.code >> (f.shift + 8 * (s >> 2)));
        u32x4 o;
        o[0] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, sc, 0));
        o[1] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, sc, 1));
        o[2] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, sc, 2));
        o[3] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, sc, 3));
        return __builtin_bit_cast(bf16x8, o);
    }
}

// ----------------------------------------------------------------------------- launch geometry

struct FfnParams {
    VerifyArgs a;
    int N, K;             // rows and reduction length of one streamed matrix
    int nblocks;          // 128-wide K blocks of a matrix row tile: ceil(K / 128)
    int nsteps;           // macro steps per item: ceil(nblocks / kBlocks of the format)
    int band_rows;        // rows per item: 16 * kWG (gate/up) or 32 * kWG (down)
    int nbands;           // bands per expert: ceil(N / band_rows)
    int workers;          // workgroups of the main kernel's grid
    size_t mat_bytes;     // bytes of one packed matrix (W_gate, W_up or W_down) of an expert
    size_t sc_bytes;      // bytes of its scales (0 for bf16)
    float *partials;      // [workers][2][slot_floats]
    int slot_floats;      // floats per partial-sum slot: partial_floats(T)
    long long *ranges;    // [workers][2]: unit range [x0, x1) of each workgroup, written by the expert kernel
    long long *fix;       // gate/up only: [workers][4] fix-up record of each workgroup (see write_fix_record)
    const int32_t *plan;  // token groups when T > 64 (else null: one group per expert)
    void *dn_sched;       // T <= 64: the down launch's schedule (DownSched), written by the gate/up launch
    int dn_K;             // gate/up: the down launch's units per token group (bands x steps)
};

// Distinct experts of the call (+ the shared one) and the number of token groups.
struct Plan {
    int U, n_groups;
};

__device__ __forceinline__ Plan load_plan(const FfnParams &P)
{
    Plan pl;
    pl.U = ld_s(P.a.n_unique);
    pl.n_groups = P.plan ? ld_s(P.plan) : pl.U + (P.a.sh_gate ? 1 : 0);
    return pl;
}

// ----------------------------------------------------------------------------- cost-weighted split
//
// A unit is one macro step of one item.  Units of a token group with more
// 16-token blocks cost more (the contraction grows with the blocks, the weight
// bytes do not), so the units are split over the workgroups by cost: group g
// costs c_g per unit, unit x of g (offset r in the group) starts at cost
// P_x = CW_g * K + r * c_g, where CW_g is the exclusive prefix of c over the
// groups and K the units per group, and workgroup w of W takes the units with
// C * w <= P_x * W < C * (w + 1), C being the total cost.  The ranges are
// contiguous, cover every unit once and cut each group's items at most at
// the range ends, as an equal split does.

// Relative per-step cost of a token group: a weight part set by the bytes a
// step streams and a contraction part per 16-token block.  The weight parts
// are the fastest measured under uneven token counts per expert (clustered
// routing, T = 64 and 256) per format and activation mode.
#ifndef ECOSPEC_COST_BF16
#define ECOSPEC_COST_BF16 29
#endif
#ifndef ECOSPEC_COST_FP8
#define ECOSPEC_COST_FP8 12
#endif
#ifndef ECOSPEC_COST_FP4
#define ECOSPEC_COST_FP4 8
#endif
#ifndef ECOSPEC_COST_FP4_MX
#define ECOSPEC_COST_FP4_MX 16
#endif
#ifndef ECOSPEC_COST_BLOCK
#define ECOSPEC_COST_BLOCK 2  // per 16-token block
#endif
template <int FMT, bool MXA>
__device__ __forceinline__ int group_cost(int M)
{
    constexpr int A = FMT == FMT_BF16 ? ECOSPEC_COST_BF16
                    : FMT == FMT_FP8  ? ECOSPEC_COST_FP8
                    : MXA             ? ECOSPEC_COST_FP4_MX
                                      : ECOSPEC_COST_FP4;
    return A + ECOSPEC_COST_BLOCK * ((M + 15) / 16);
}

constexpr int kMaxTokLds = 4096;  // routed slots whose token rows are staged in LDS

// Per-launch schedule, built in LDS by every workgroup at start: the split,
// and the token groups' metadata so that moving to a new item reads LDS
// instead of waiting on global memory.
struct Split {
    int cw[kMaxGroups + 1];             // exclusive cost prefix over token groups; cw[n_groups] = total
    long long bound[kMaxWorkers + 1];   // bound[w] = first unit of workgroup w; bound[W] = all units
    int gp0[kMaxGroups];                // grouped position of each group's first token
    int gM[kMaxGroups];                 // tokens in each group (<= 64)
    int ge[kMaxGroups];                 // expert id of each group (-1: the shared expert)
    int tok[kMaxTokLds];                // gate/up: token of each grouped position, down: its routed slot
                                        // (if T*k <= kMaxTokLds)
    int wave_tot[2 * kWG];
};

// Fills sp.cw and the groups' metadata for the launch (whole workgroup) and
// returns the plan.  Without a token-group plan (one group per union member,
// then the shared expert) the union's offsets and ids are read for every
// possible member in the same round trip as the union size and the slots'
// tokens: the schedule waits for global memory once, not twice.
template <int FMT, bool MXA, bool DOWN>
__device__ __forceinline__ Plan build_costs(const FfnParams &P, Split &sp)
{
    constexpr int kPre = (1024 + kEThreads - 1) / kEThreads;  // groups per thread read ahead (E <= 1024: every union)
    const VerifyArgs &a = P.a;
    const int S = a.T * a.k;
    const int tid = threadIdx.x;
    int o0[kPre], o1[kPre], id[kPre];
#pragma unroll
    for (int j = 0; j < kPre; ++j) {
        const int g = j * kEThreads + tid;
        const bool ok = P.plan == nullptr && g < a.E;
        o0[j] = ok ? a.offsets[g] : 0;
        o1[j] = ok ? a.offsets[g + 1] : 0;
        id[j] = ok ? a.union_ids[g] : 0;
    }
    const Plan pl = load_plan(P);
    if (S <= kMaxTokLds)
        for (int p = tid; p < S; p += kEThreads) sp.tok[p] = DOWN ? a.perm[p] : a.perm[p] / a.k;
    int run = 0;
    for (int base = 0, j = 0; base < pl.n_groups; base += kEThreads, ++j) {
        const int g = base + tid;
        int c = 0;
        if (g < pl.n_groups) {
            const int u = P.plan ? P.plan[8 + 2 * g] : g, tg = P.plan ? P.plan[8 + 2 * g + 1] : 0;
            const bool shared = u >= pl.U;
            int lo = 0, hi = 0, e = -1;
            if (!shared) {
                if (P.plan == nullptr && j < kPre) {
#pragma unroll
                    for (int q = 0; q < kPre; ++q)
                        if (q == j) {
                            lo = o0[q];
                            hi = o1[q];
                            e = id[q];
                        }
                } else {
                    lo = a.offsets[u];
                    hi = a.offsets[u + 1];
                    e = a.union_ids[u];
                }
            }
            const int Mu = shared ? a.T : hi - lo;
            sp.gM[g] = min(kTokGroup, Mu - tg * kTokGroup);
            sp.gp0[g] = (shared ? S : lo) + tg * kTokGroup;
            sp.ge[g] = e;
            c = group_cost<FMT, MXA>(sp.gM[g]);
        }
        int tot = 0;
        const int ex = block_exclusive_scan(c, sp.wave_tot, &tot);
        if (g < pl.n_groups) sp.cw[g] = run + ex;
        run += tot;
    }
    if (threadIdx.x == 0) sp.cw[pl.n_groups] = run;
    __syncthreads();
    return pl;
}

// Gate/up launch without a token-group plan (T <= 64: every expert's tokens
// form one group).  The union of the routed experts and the grouping of the
// slots by expert (Eq. 1, the stable counting sort moe_expert_union computes)
// are built by each workgroup in LDS straight from topk_idx, with the groups'
// costs; workgroup 0 also writes them to the routing arrays for the later
// launches and the caller.  Per pass of one slot per thread: wavefront matches
// by ballot (rank among equal experts, count per wavefront), per-expert counts
// in wcnt[kPW][E] (scratch in the activation tiles, unused this early); one scan
// over the experts in id order (= union order) gives each member its union
// position and first grouped position, a second one the cost prefix; a second
// sweep places every slot.
template <int FMT, bool MXA>
__device__ __forceinline__ Plan union_and_costs(const FfnParams &P, Split &sp, int *wcnt)
{
    constexpr int kPass = 4096 / kEThreads;               // slots: T * k <= 64 * 64 = kPass * kEThreads
    constexpr int EPT = (1024 + kEThreads - 1) / kEThreads;  // experts per thread: E <= 1024
    const VerifyArgs &a = P.a;
    const int S = a.T * a.k, E = a.E, tid = threadIdx.x, wave = tid / kWave;
    const bool out = blockIdx.x == 0;
    int nbits = 0;
    while ((1 << nbits) < E) ++nbits;
    const int passes = (S + kEThreads - 1) / kEThreads;
    const int nj = (E + kEThreads - 1) / kEThreads;  // expert rounds actually needed (the code runs cold: skip the rest)
    int ex[kPass], rank[kPass], cnt[kPass];
    bool top[kPass];
#pragma unroll
    for (int ps = 0; ps < kPass; ++ps) {
        const int sl = ps * kEThreads + tid;
        ex[ps] = ps < passes && sl < S ? a.topk_idx[sl] : -1;
        rank[ps] = cnt[ps] = 0;
        top[ps] = false;
    }
    // Counts per expert over the passes.
    int tot[EPT];
#pragma unroll
    for (int j = 0; j < EPT; ++j) tot[j] = 0;
#pragma unroll
    for (int ps = 0; ps < kPass; ++ps) {
        if (ps >= passes) break;
        for (int i = tid; i < kPW * E; i += kEThreads) wcnt[i] = 0;
        __syncthreads();
        wave_match(ex[ps], (unsigned)ex[ps] < (unsigned)E, nbits, rank[ps], top[ps], cnt[ps]);
        if (top[ps]) wcnt[wave * E + ex[ps]] = cnt[ps];
        __syncthreads();
#pragma unroll
        for (int j = 0; j < EPT; ++j) {
            if (j >= nj) break;
            const int e = j * kEThreads + tid;
            if (e < E)
                for (int w = 0; w < kPW; ++w) tot[j] += wcnt[w * E + e];
        }
        if (ps + 1 < passes) __syncthreads();  // one pass: its counts stay in wcnt for the placement
    }
    // Union positions, first grouped positions and the cost prefix.  A group
    // keeps at most 64 tokens (more only with repeated experts within a token).
    int run_u = 0, run_p = 0, run_c = 0, start[EPT];
#pragma unroll
    for (int j = 0; j < EPT; ++j) start[j] = 0;
#pragma unroll
    for (int j = 0; j < EPT; ++j) {
        if (j >= nj) break;
        const int e = j * kEThreads + tid;
        const int c = e < E ? tot[j] : 0;
        const int M = min(kTokGroup, c);
        int up, cp, tup, tcost;
        block_exclusive_scan2((c << 11) | (c > 0 ? 1 : 0), c > 0 ? group_cost<FMT, MXA>(M) : 0, sp.wave_tot, up, cp,
                              tup, tcost);
        const int pos = run_u + (up & 2047);
        start[j] = run_p + (up >> 11);
        if (c > 0) {
            sp.ge[pos] = e;
            sp.gp0[pos] = start[j];
            sp.gM[pos] = M;
            sp.cw[pos] = run_c + cp;
        }
        if (out && e < E) a.counts[e] = c;
        run_u += tup & 2047;
        run_p += tup >> 11;
        run_c += tcost;
    }
    Plan pl;
    pl.U = run_u;
    pl.n_groups = run_u + (a.sh_gate ? 1 : 0);
    if (tid == 0) {
        int total = run_c;
        if (a.sh_gate) {  // the shared expert: all T tokens, after every routed slot
            sp.ge[run_u] = -1;
            sp.gp0[run_u] = S;
            sp.gM[run_u] = min(kTokGroup, a.T);
            sp.cw[run_u] = run_c;
            total += group_cost<FMT, MXA>(min(kTokGroup, a.T));
        }
        sp.cw[pl.n_groups] = total;
    }
    // Placement: first position of the expert + slots of earlier passes and wavefronts + rank.
    int run[EPT];
#pragma unroll
    for (int j = 0; j < EPT; ++j) run[j] = start[j];
#pragma unroll
    for (int ps = 0; ps < kPass; ++ps) {
        if (ps >= passes) break;
        if (passes > 1) {
            for (int i = tid; i < kPW * E; i += kEThreads) wcnt[i] = 0;
            __syncthreads();
            if (top[ps]) wcnt[wave * E + ex[ps]] = cnt[ps];
            __syncthreads();
        }
#pragma unroll
        for (int j = 0; j < EPT; ++j) {
            if (j >= nj) break;
            const int e = j * kEThreads + tid;
            if (e < E) {
                int nw[kPW];
#pragma unroll
                for (int w = 0; w < kPW; ++w) nw[w] = wcnt[w * E + e];
#pragma unroll
                for (int w = 0; w < kPW; ++w) {
                    wcnt[w * E + e] = run[j];
                    run[j] += nw[w];
                }
            }
        }
        __syncthreads();
        if ((unsigned)ex[ps] < (unsigned)E) {
            const int pos = wcnt[wave * E + ex[ps]] + rank[ps], sl = ps * kEThreads + tid;
            sp.tok[pos] = sl / a.k;
            if (out) a.perm[pos] = sl;
        }
        if (ps + 1 < passes) __syncthreads();
    }
    if (out) {
        for (int u = tid; u <= E; u += kEThreads) {
            if (u < E) a.union_ids[u] = u < run_u ? sp.ge[u] : -1;
            a.offsets[u] = u < run_u ? sp.gp0[u] : run_p;
        }
        if (tid == 0) *a.n_unique = run_u;
    }
    return pl;
}

// First unit x with P_x * W >= target (0 <= target <= C * W), by binary
// search over the groups' cost prefix.
__device__ __forceinline__ long first_unit(const Split &sp, int n_groups, long K, long W, long long target)
{
    return split::first_unit(sp.cw, n_groups, K, W, target);
}

// Every workgroup's first unit, into sp.bound (whole workgroup).
__device__ __forceinline__ void build_bounds(Split &sp, int n_groups, long K, int W)
{
    const long long C = (long long)sp.cw[n_groups] * K;
    for (int v = threadIdx.x; v <= W; v += kEThreads) sp.bound[v] = first_unit(sp, n_groups, K, W, C * v);
    __syncthreads();
}

// Workgroup whose range holds unit x.
__device__ __forceinline__ int owner_of(const Split &sp, int n_groups, long K, int W, long x)
{
    return split::owner_of(sp.cw, n_groups, K, W, x);
}

// The down launch's schedule when every expert's tokens form one group (T <= 64): its token
// groups are the gate/up launch's (the union members in order, then the shared expert) with the
// same costs, so only the unit ranges differ (K is the down launch's).  Workgroup 0 of the gate/up
// launch, which also writes the union, writes it before its first weight load; the down launch
// then reads it in one round trip instead of rebuilding it from the union.
constexpr int kSchedGroups = 1025;  // n_groups <= E + 1, E <= 1024
struct DownSched {
    long long bound[kMaxWorkers + 1];
    int cw[kSchedGroups + 1], ge[kSchedGroups], gp0[kSchedGroups], gM[kSchedGroups];
};

__device__ __forceinline__ void write_down_sched(const FfnParams &P, const Plan &pl, const Split &sp)
{
    DownSched *ds = static_cast<DownSched *>(P.dn_sched);
    const long K = P.dn_K;
    const long long C = (long long)sp.cw[pl.n_groups] * K;
    for (int v = threadIdx.x; v <= P.workers; v += kEThreads)
        ds->bound[v] = first_unit(sp, pl.n_groups, K, P.workers, C * v);
    for (int g = threadIdx.x; g <= pl.n_groups; g += kEThreads) {
        ds->cw[g] = sp.cw[g];
        if (g < pl.n_groups) {
            ds->ge[g] = sp.ge[g];
            ds->gp0[g] = sp.gp0[g];
            ds->gM[g] = sp.gM[g];
        }
    }
}

// The down launch's side (whole workgroup): the schedule, the union size and the slots of the
// grouped positions, every load issued before the first LDS store (one round trip; entries past
// the launch's groups are read but not used).
__device__ __forceinline__ Plan load_down_sched(const FfnParams &P, Split &sp)
{
    constexpr int kG = (kSchedGroups + 1 + kEThreads - 1) / kEThreads;
    constexpr int kB = (kMaxWorkers + 1 + kEThreads - 1) / kEThreads;
    const DownSched *ds = static_cast<const DownSched *>(P.dn_sched);
    const VerifyArgs &a = P.a;
    const int tid = threadIdx.x, S = a.T * a.k;
    long long b[kB];
    int cw[kG], ge[kG], gp0[kG], gM[kG];
#pragma unroll
    for (int j = 0; j < kB; ++j) {
        const int v = j * kEThreads + tid;
        b[j] = v <= P.workers ? ds->bound[v] : 0;
    }
#pragma unroll
    for (int j = 0; j < kG; ++j) {
        const int g = j * kEThreads + tid;
        const bool ok = g <= kSchedGroups;
        cw[j] = ok ? ds->cw[g] : 0;
        ge[j] = ok && g < kSchedGroups ? ds->ge[g] : 0;
        gp0[j] = ok && g < kSchedGroups ? ds->gp0[g] : 0;
        gM[j] = ok && g < kSchedGroups ? ds->gM[g] : 0;
    }
    const Plan pl = load_plan(P);
    if (S <= kMaxTokLds)
        for (int p = tid; p < S; p += kEThreads) sp.tok[p] = a.perm[p];
#pragma unroll
    for (int j = 0; j < kB; ++j) {
        const int v = j * kEThreads + tid;
        if (v <= P.workers) sp.bound[v] = b[j];
    }
#pragma unroll
    for (int j = 0; j < kG; ++j) {
        const int g = j * kEThreads + tid;
        if (g <= pl.n_groups) sp.cw[g] = cw[j];
        if (g < pl.n_groups) {
            sp.ge[g] = ge[j];
            sp.gp0[g] = gp0[j];
            sp.gM[g] = gM[j];
        }
    }
    __syncthreads();
    return pl;
}

// What a workgroup needs to know about one item.
struct ItemDesc {
    const uint8_t *wa, *wb;  // tile 0 / tile 1 matrices of the expert (packed)
    const void *sa, *sb;     // their scales
    int n0;                  // first row of the band
    int p0;                  // grouped position of the group's first token
    int M;                   // tokens in the group (<= 64)
    int e;                   // expert id (-1: the shared expert)
    bool shared;
    bool pair;               // gate/up: the two matrices packed as one pair at wa (wb == wa);
                             // down: the wavefront's two row tiles interleaved per block
};

// What a workgroup needs to know about an item, from the schedule in LDS.
template <bool DOWN>
__device__ __forceinline__ ItemDesc describe_lds(const FfnParams &P, const Split &sp, int item)
{
    const VerifyArgs &a = P.a;
    const int gi = item / P.nbands, band = item - gi * P.nbands;
    const size_t mat = P.mat_bytes, sc = P.sc_bytes;
    ItemDesc d;
    const int e0 = __builtin_amdgcn_readfirstlane(sp.ge[gi]);
    d.shared = e0 < 0;
    d.e = e0;
    d.p0 = __builtin_amdgcn_readfirstlane(sp.gp0[gi]);
    d.M = __builtin_amdgcn_readfirstlane(sp.gM[gi]);
    d.n0 = band * P.band_rows;
    const size_t e = d.shared ? 0 : (size_t)e0;
    auto sptr = [&](const void *base) {
        return base ? static_cast<const void *>(static_cast<const uint8_t *>(base) + e * sc) : nullptr;
    };
    d.pair = false;
    if (!DOWN) {
        d.pair = d.shared ? a.sh_gu_pair : a.gu_pair;
        d.wa = (d.shared ? a.sh_gate : a.w_gate) + e * mat * (d.pair ? 2 : 1);
        d.wb = d.pair ? d.wa : (d.shared ? a.sh_up : a.w_up) + e * mat;
        d.sa = d.shared ? a.sh_s_gate : sptr(a.s_gate);
        d.sb = d.shared ? a.sh_s_up : sptr(a.s_up);
    } else {
        d.wa = d.wb = (d.shared ? a.sh_down : a.w_down) + e * mat;
        d.sa = d.sb = d.shared ? a.sh_s_down : sptr(a.s_down);
        d.pair = a.down_pair;
    }
    return d;
}

// Rows of wavefront `wave`'s two tiles within an item (the same 16 rows of
// gate and up, or 32 consecutive rows of down).
template <bool DOWN>
__device__ __forceinline__ int tile_row(const ItemDesc &d, int wave, int t)
{
    return DOWN ? d.n0 + 32 * wave + 16 * t : d.n0 + 16 * wave;
}

// ----------------------------------------------------------------------------- epilogue

// Gate and up biases of a wavefront's rows of an item (zeros without biases,
// for the shared expert and for the down launch).  The expert kernel loads
// them when it starts an item and uses them when it finishes it, so the loads
// are long done by then.
struct ItemBias {
    f32x4 g, u;
};

template <bool DOWN>
__device__ __forceinline__ ItemBias load_bias(const FfnParams &P, const ItemDesc &d, int wave)
{
    const VerifyArgs &a = P.a;
    ItemBias b{f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
    if (DOWN || d.shared || (!a.b_gate && !a.b_up)) return b;
    const int row = d.n0 + 16 * wave + 4 * (lane_id() >> 4);  // gate/up rows row .. row + 3 of this lane
    if (row >= P.N) return b;
    if (a.b_gate) b.g = *reinterpret_cast<const f32x4 *>(a.b_gate + (size_t)d.e * a.d_ff + row);
    if (a.b_up) b.u = *reinterpret_cast<const f32x4 *>(a.b_up + (size_t)d.e * a.d_ff + row);
    return b;
}

// g * sigmoid(s * g) with the hardware exp2 and reciprocal (about 2 ulp in
// fp32, far below the bf16 rounding of H): g / (1 + e^(-s g)).  Large -s g
// gives 1 + inf, whose reciprocal is 0, and NaN stays NaN, as in the
// division form.
__device__ __forceinline__ float gated(float g, float s)
{
    return g * __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(-s * g * 1.44269504088896341f));
}

// h from the gate and up values of one row (biases already added):
// act 0 silu(g) * u; act 1 (GPT-OSS) with g capped at limit and u clamped to
// [-limit, limit], g * sigmoid(alpha * g) * (u + 1).  The comparisons keep NaN.
__device__ __forceinline__ float activate(const VerifyArgs &a, float g, float u)
{
    if (a.act == 0) return gated(g, 1.f) * u;
    if (g > a.limit) g = a.limit;
    if (u > a.limit) u = a.limit;
    if (u < -a.limit) u = -a.limit;
    return gated(g, a.alpha) * (u + 1.f);
}

// Finishes the accumulators of an item held by wavefront pw, which owns slots
// pw * VPW .. pw * VPW + VPW - 1 (tiles 2j, 2j + 1 of its slot j): gate/up ->
// bf16 SwiGLU rows of H at grouped positions, down -> fp32 rows of O at the
// rows' routed slots t * k + j (the shared expert's at T * k + t), so that the
// combine kernel finds a whole item's row without a lookup.  tok: the slot of
// each grouped position (down, T * k <= kMaxTokLds; else a.perm is read).
// Lane (col, grp) holds rows 4*grp .. 4*grp+3 of a tile for token column col
// of each 16-token block.
//
// MX activation mode, gate/up: the SwiGLU rows go to the down launch as MX
// FP8.  A band (128 rows) is one 128-element chunk of an H row; slot v's 16
// rows are half of the 32-row block v / 2, the other half being slot v ^ 1's,
// so the two exchange their per-token maxima through LDS (every wavefront of
// the workgroup takes part, also those past the last row, which write the
// zero padding the down launch reads).  Row 16v + j of the chunk is stored at
// byte 32 (v % 4) + 16 (v / 4) + j, the FP8 operand's lane order.
template <bool DOWN, bool MXA, int VPW>
__device__ __forceinline__ void finish_item(const FfnParams &P, const ItemDesc &d, int pw,
                                            const f32x4 (&acc)[2 * VPW][kMB], const ItemBias (&bias)[VPW],
                                            const int *tok = nullptr)
{
    const VerifyArgs &a = P.a;
    const int lane = lane_id(), col = lane & 15, grp = lane >> 4;
    if constexpr (!DOWN && MXA) {
        __shared__ float red[kWG][kMB][16];
        float h[VPW][kMB][4];
#pragma unroll
        for (int j = 0; j < VPW; ++j) {
            const int v = pw * VPW + j;
            const bool rows_ok = tile_row<false>(d, v, 0) < P.N;  // N % 32 == 0: a tile is all in or all out
#pragma unroll
            for (int mb = 0; mb < kMB; ++mb) {
                const f32x4 g = acc[2 * j][mb] + bias[j].g, u = acc[2 * j + 1][mb] + bias[j].u;
                const bool live = rows_ok && mb * 16 + col < d.M;
#pragma unroll
                for (int i = 0; i < 4; ++i) h[j][mb][i] = live ? activate(a, g[i], u[i]) : 0.f;
                float m = fmaxf(fmaxf(fabsf(h[j][mb][0]), fabsf(h[j][mb][1])), fmaxf(fabsf(h[j][mb][2]), fabsf(h[j][mb][3])));
                m = fmaxf(m, __shfl_xor(m, 16, kWave));
                m = fmaxf(m, __shfl_xor(m, 32, kWave));
                if (grp == 0) red[v][mb][col] = m;
            }
        }
        __syncthreads();
        const int kp = P.nbands * P.band_rows;  // padded d_ff
#pragma unroll
        for (int j = 0; j < VPW; ++j) {
            const int v = pw * VPW + j;
#pragma unroll
            for (int mb = 0; mb < kMB; ++mb) {
                const int r = mb * 16 + col;
                if (r >= d.M) continue;
                const int E = mx_exponent(fmaxf(red[v][mb][col], red[v ^ 1][mb][col]));
                const float inv = mx_inv_scale(E);
                const uint32_t q = e4m3_code(h[j][mb][0] * inv) | (e4m3_code(h[j][mb][1] * inv) << 8) |
                                   (e4m3_code(h[j][mb][2] * inv) << 16) | (e4m3_code(h[j][mb][3] * inv) << 24);
                const size_t p = (size_t)(d.p0 + r);
                *reinterpret_cast<uint32_t *>(a.hq + p * kp + d.n0 + 32 * (v & 3) + 16 * (v >> 2) + 4 * grp) = q;
                if ((v & 1) == 0 && grp == 0) a.hs[p * (kp / 32) + d.n0 / 32 + v / 2] = (uint8_t)(E + 127);
            }
        }
        return;
    }
#pragma unroll
    for (int j = 0; j < VPW; ++j) {
        const int v = pw * VPW + j;
        if (tile_row<DOWN>(d, v, 0) >= P.N) continue;  // rows past the last band
#pragma unroll
        for (int mb = 0; mb < kMB; ++mb) {
            const int r = mb * 16 + col;
            if (r >= d.M) continue;
            const int p = d.p0 + r;
            if (!DOWN) {
                f32x4 g = acc[2 * j][mb], u = acc[2 * j + 1][mb];
                uint32_t h2[2];
                if (a.act == 0 && !a.b_gate && !a.b_up) {
#pragma unroll
                    for (int i = 0; i < 2; ++i) {
                        const float g0 = g[2 * i], g1 = g[2 * i + 1];
                        h2[i] = pack_bf16x2(gated(g0, 1.f) * u[2 * i], gated(g1, 1.f) * u[2 * i + 1]);
                    }
                } else {
                    g += bias[j].g;
                    u += bias[j].u;
                    float h[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i) h[i] = activate(a, g[i], u[i]);
                    h2[0] = pack_bf16x2(h[0], h[1]);
                    h2[1] = pack_bf16x2(h[2], h[3]);
                }
                *reinterpret_cast<u32x2 *>(a.h + (size_t)p * a.d_ff + tile_row<DOWN>(d, v, 0) + 4 * grp) =
                    u32x2{h2[0], h2[1]};
            } else {
                const int S = a.T * a.k;
                const int row = p >= S ? p : S <= kMaxTokLds ? tok[p] : a.perm[p];
#pragma unroll
                for (int t = 0; t < 2; ++t)
                    *reinterpret_cast<f32x4 *>(a.o + (size_t)row * a.d + tile_row<DOWN>(d, v, t) + 4 * grp) =
                        acc[2 * j + t][mb];
            }
        }
    }
}

// ----------------------------------------------------------------------------- main kernel

// Where the loads of one item come from.  Wave-uniform except the lane offsets.
struct Source {
    rsrc_t ra0, ra1, rs0, rs1;  // matrices of each slot's tiles 0 / 1 (gate / up, or its two row tiles) and their scales
    uint32_t a[kNT];            // lane offsets of the wavefront's tiles at step 0 (tile 2j + t: slot j's tile t;
                                // kOff: rows past N)
    uint32_t kstride;           // bytes from one 128-wide block of a tile to the next
    uint32_t q[kNT];            // scale offsets at step 0
    uint32_t boff[kBPass];      // lane offsets of this thread's activation chunks at step 0 (kOff: no token)
    uint32_t soff[kBPass];      // MX activations: offsets of the rows' block scales at step 0
    int kc;                     // first element (within a 128-wide block) of the thread's activation chunk
    int ib, ie;                 // the item's units [ib, ie)
    int item;
};

template <int FMT, bool DOWN, bool MXA>
__device__ __forceinline__ void set_source(Source &src, const FfnParams &P, const Split &sp, int item)
{
    constexpr int NV = Fmt<FMT>::kVecs;
    constexpr uint32_t BLK = 1024u * NV;
    const VerifyArgs &a = P.a;
    const int lane = lane_id(), tid = threadIdx.x, bc = tid & 15;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int K = P.K, nsteps = P.nsteps;
    const ItemDesc d = describe_lds<DOWN>(P, sp, item);
    src.item = item;
    src.ib = item * nsteps;
    src.ie = src.ib + nsteps;

    const int nblocks = P.nblocks;
    const uint32_t mat_bytes = (uint32_t)P.mat_bytes;  // < 2^31 (checked at the boundary)
    // Paired layouts (pack.hip): a slot's two tiles of one block are one run (down: its two row tiles,
    // gate/up: the gate and up tiles of its rows), tile t at t * BLK in the run.
    if (d.pair) {
        src.ra0 = src.ra1 = make_rsrc(d.wa, DOWN ? mat_bytes : 2u * mat_bytes);
        src.kstride = 2u * BLK;
    } else {
        src.ra0 = make_rsrc(d.wa, mat_bytes);
        src.ra1 = make_rsrc(d.wb, mat_bytes);
        src.kstride = BLK;
    }
    const uint32_t sc_bytes = (uint32_t)P.sc_bytes;
    src.rs0 = make_rsrc(FMT == FMT_BF16 ? d.wa : d.sa, FMT == FMT_BF16 ? 0u : sc_bytes);
    src.rs1 = make_rsrc(FMT == FMT_BF16 ? d.wb : d.sb, FMT == FMT_BF16 ? 0u : sc_bytes);
#pragma unroll
    for (int tt = 0; tt < kNT; ++tt) {
        const int v = wave * kVPW + tt / 2, t = tt % 2;
        const int row0 = tile_row<DOWN>(d, v, 0), row = tile_row<DOWN>(d, v, t);
        const bool ok = row0 < P.N;  // a slot's rows are all in or all out
        if (d.pair)  // the slot's run (unit: 32 rows for down, 16 for gate/up) at block 0
            src.a[tt] = ok ? (uint32_t)(row0 / (DOWN ? 32 : 16)) * nblocks * 2u * BLK + (uint32_t)t * BLK + lane * 16u
                           : kOff;
        else
            src.a[tt] = ok ? (uint32_t)(row / 16) * nblocks * BLK + lane * 16u : kOff;
        src.q[tt] = 0;
        if constexpr (FMT == FMT_FP8)
            src.q[tt] = ok ? (uint32_t)(row / 128) * (K / 128) * 4u : kOff;
        else if constexpr (FMT == FMT_MXFP4)
            src.q[tt] = ok ? (uint32_t)(row / 16) * ((nblocks + 3) / 4) * 256u + lane * 4u : kOff;
    }

    // Activation rows: in pass i, lane l of this wavefront stages row
    // i*kBRowsPerPass + 4*wave + l/16 of the item's tokens (16 lanes per row)
    // into chunk position l % 16, i.e. the row's chunk (l % 16) ^ (row % 16)
    // (the tile's swizzle; MX activations: chunk l % 16).
    // Its source row (the token of a grouped position for gate/up, the grouped
    // position itself for down) is read by each lane for itself: no wave-wide
    // round trips.
    // MX activations: rows of nblocks * 128 e4m3fn codes and nblocks * 4 scales.
    const uint32_t brow_bytes = MXA ? (uint32_t)nblocks * kMacroK : (uint32_t)(DOWN ? a.d_ff : a.d) * 2u;
    const int q = lane >> 4;
    const int cq = MXA ? bc : bc ^ ((4 * wave + q) & 15);
    src.kc = cq * 8;
#pragma unroll
    for (int i = 0; i < kBPass; ++i) {
        const int r = i * kBRowsPerPass + 4 * wave + q;
        int row = -1;
        if (r < d.M) {
            const int p = d.p0 + r;
            row = DOWN ? p
                : d.shared ? p - a.T * a.k
                : a.T * a.k <= kMaxTokLds ? sp.tok[p]
                                          : (int)((uint32_t)a.perm[p] / (uint32_t)a.k);
        }
        src.boff[i] = row >= 0 ? (uint32_t)row * brow_bytes + (uint32_t)cq * 16u : kOff;
        src.soff[i] = row >= 0 ? (uint32_t)row * (uint32_t)nblocks * 4u + (uint32_t)(bc & 1) * 4u : kOff;
    }
}

// One macro step of a wavefront: its kNT 16 x 128 weight tiles against the
// nmb live 16-token blocks of the activation tile in LDS.  The tiles are
// decoded once for the step; then each token block reads its activation
// fragments and runs its chains.  Every accumulator is updated in place or
// skipped (a wave-uniform branch per token block), so the loop carries them in
// fixed registers whatever nmb is (a switch over nmb gave each arm its own
// registers and the loop copied the accumulators back every step).
template <int FMT>
__device__ __forceinline__ void contract(const WFrag<FMT> (&wv)[kNT], const uint8_t *buf, f32x4 (&acc)[kNT][kMB],
                                         int nmb)
{
    constexpr int SB = Fmt<FMT>::kBlocks, NS = 4 * SB;
    const int lane = lane_id(), col = lane & 15, grp = lane >> 4;
    // Sub-step s takes chunk 4 * grp + s % 4 of block s / 4 of token row 16 * mb + col, stored
    // at chunk position (4 * grp + s % 4) ^ col (the row's low four bits are col).
    const uint8_t *bp = buf + col * 256;
    const int xg = ((4 * grp) ^ col) * 16;
    auto boff = [&](int s) { return (s >> 2) * BTile<SB>::kBlk + (xg ^ ((s & 3) * 16)); };
    bf16x8 av[NS][kNT];
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
        for (int t = 0; t < kNT; ++t) av[s][t] = decode_a<FMT>(wv[t], s);
#pragma unroll
    for (int mb = 0; mb < kMB; ++mb) {
        if (mb > 0 && mb >= nmb) break;
        bf16x8 b[NS];
#pragma unroll
        for (int s = 0; s < NS; ++s)
            b[s] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(bp + mb * 16 * 256 + boff(s)));
        // FP8 accumulates the step in `part` and adds scale * part at the end; the other formats
        // accumulate in place.
        f32x4 part[kNT];
        if constexpr (FMT == FMT_FP8) {
#pragma unroll
            for (int t = 0; t < kNT; ++t) part[t] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int s = 0; s < NS; ++s)
#pragma unroll
            for (int t = 0; t < kNT; ++t) {
                f32x4 &c = FMT == FMT_FP8 ? part[t] : acc[t][mb];
                c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[s][t], b[s], c, 0, 0, 0);
            }
        if constexpr (FMT == FMT_FP8) {
#pragma unroll
            for (int t = 0; t < kNT; ++t)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[t][mb][j] = __builtin_fmaf(wv[t].scale, part[t][j], acc[t][mb][j]);
        }
    }
}

// MX activation mode: LDS geometry of one step's FP8 activation tile (64
// tokens x 256 codes, rows padded by 16 bytes) followed by its scales (8 per
// token: 4 blocks of each of the step's two 128-wide chunks).
// Activation tiles in LDS for a prefetch depth.  Direct loads: one per ring
// slot, the tile of step i + PD - 1 being loaded once every wavefront has
// passed step i's barrier, i.e. finished step i - 1, the tile's last reader.
// MX activations (staged through registers, written before the barrier): the
// slots and tiles cycle together, two tiles sufficing for correctness.
constexpr int kTiles(int PD, bool MXA) { return !MXA ? PD : PD % 2 ? PD : 2; }

constexpr int kRowQ = 256 + 16;
constexpr int kScaleQ = kMB * 16 * kRowQ;

typedef __attribute__((ext_vector_type(8))) int i32x8;

// One MXFP4 macro step of a wavefront with MX FP8 activations: per 128-wide
// block, one v_mfma_scale_f32_16x16x128_f8f6f4 per tile and token block.  The
// A operand is the lane's packed FP4 fragment (K 32grp..32grp+31 of its row)
// with its e8m0 code; the B operand is token col's codes of K 16grp..16grp+15
// and 64+16grp..64+16grp+15 (stored contiguously) with the scale of block grp
// (K 32grp..32grp+31), which the instruction applies to that K block.
__device__ __forceinline__ void contract_mx(const WFrag<FMT_MXFP4> (&wv)[kNT], const uint8_t *buf,
                                            f32x4 (&acc)[kNT][kMB], int nmb)
{
    const int lane = lane_id(), col = lane & 15, grp = lane >> 4;
    const uint8_t *bp = buf + col * kRowQ + grp * 32;
    const uint8_t *sp = buf + kScaleQ + col * 8 + grp;
    i32x8 av[2][kNT];
    int sa[2][kNT];
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int t = 0; t < kNT; ++t) {
            const u32x4 w = wv[t].v[b];
            av[b][t] = i32x8{(int)w[0], (int)w[1], (int)w[2], (int)w[3], 0, 0, 0, 0};
            sa[b][t] = (int)((wv[t].code >> (wv[t].shift + 8 * b)) & 0xffu);
        }
    // Token blocks past nmb are skipped with a wave-uniform branch; the accumulators stay in
    // place (see contract()).
#pragma unroll
    for (int mb = 0; mb < kMB; ++mb) {
        if (mb > 0 && mb >= nmb) break;
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            const u32x4 lo = *reinterpret_cast<const u32x4 *>(bp + mb * 16 * kRowQ + b * 128);
            const u32x4 hi = *reinterpret_cast<const u32x4 *>(bp + mb * 16 * kRowQ + b * 128 + 16);
            const i32x8 bv = i32x8{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3], (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
            const int sb = sp[mb * 16 * 8 + b * 4];
#pragma unroll
            for (int t = 0; t < kNT; ++t)
                acc[t][mb] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(av[b][t], bv, acc[t][mb], 4, 0, 0,
                                                                              sa[b][t], 0, sb);
        }
    }
}

// The contributors of a cut item (units [ib, ie)): the partial-sum slots
// (workgroup * 2 + slot) of the workgroups whose ranges overlap it, in
// workgroup order, 20 bits each, their count in bits 60..61 (bit 62 set); or,
// past 3 contributors, bits 62 and 63 clear and (w0 << 16 | w1), the first
// and last workgroup.
__device__ __forceinline__ long long contributors(const FfnParams &P, const Plan &pl, const Split &sp, long ib,
                                                  long ie)
{
    return split::contributors(sp.cw, sp.bound, pl.n_groups, (long)P.nbands * P.nsteps, P.workers, ib, ie);
}

// Down launch: for the combine kernel, the output descriptor (split.hpp) of
// every row of each item whose last unit lies in this range, so that every
// row of every item is described by exactly one range on every launch.  A
// whole item's row is its row of O (the row's slot); a cut item's row is the sum of its
// contributors' parked partial sums, in workgroup order.  Descriptors are
// indexed by the row's routed slot (the shared expert's rows by T*k + token).
__device__ __forceinline__ void record_outputs(const FfnParams &P, const Plan &pl, const Split &sp, int x0, int x1)
{
    const VerifyArgs &a = P.a;
    const int ns = P.nsteps, S = a.T * a.k;
    const long K = (long)P.nbands * ns;
    for (int item = x0 / ns; item * ns < x1; ++item) {
        const int ib = item * ns, ie = ib + ns;
        if (ie > x1) break;  // described by the range holding its last unit
        const int gi = item / P.nbands, band = item - gi * P.nbands;
        const int M = sp.gM[gi], p0 = sp.gp0[gi];
        const bool whole = ib >= x0;
        const uint64_t cut = whole ? 0ull : split::out_cut(sp.cw, sp.bound, pl.n_groups, K, P.workers, ib, ie);
        for (int r = threadIdx.x; r < M; r += kEThreads) {
            const int p = p0 + r;
            const int row = p >= S ? p : S <= kMaxTokLds ? sp.tok[p] : a.perm[p];
            a.desc[(size_t)row * P.nbands + band] = whole ? split::out_whole((uint32_t)row) : split::out_with_row(cut, r);
        }
    }
}

// Gate/up launch, thread 0 of workgroup w: the record its fix-up reads.  If
// the range starts inside an item that ends within it (w is the item's last
// contributor), {item, contributors(), first grouped position | (expert + 1)
// << 32, tokens} of that item; else item = -1.  Every workgroup writes its record on every launch.
__device__ __forceinline__ void write_fix_record(const FfnParams &P, const Plan &pl, const Split &sp, int w, long x0,
                                                 long x1)
{
    long long r[4] = {-1, 0, 0, 0};
    const long ns = P.nsteps;
    const long item = split::finished_item(x0, x1, ns);
    if (item >= 0) {
        const int gi = (int)(item / P.nbands);
        r[0] = item;
        r[1] = contributors(P, pl, sp, item * ns, item * ns + ns);
        r[2] = (long long)(uint32_t)sp.gp0[gi] | ((long long)(sp.ge[gi] + 1) << 32);
        r[3] = sp.gM[gi];
    }
    long long *dst = P.fix + 4 * (size_t)w;
    dst[0] = r[0];
    dst[1] = r[1];
    dst[2] = r[2];
    dst[3] = r[3];
}

// Where a wavefront's accumulator (tile t, token block mb) is parked in a
// partial-sum slot: gate/up in accumulator order (only its fix-up reads it);
// down as [64 tokens][band rows] fp32, the layout of O, so the combine
// kernel's reads are coalesced.
template <bool DOWN>
__device__ __forceinline__ int partial_offset(int wave, int t, int mb, int lane)
{
    if (!DOWN) return (((mb * kWG + wave) * 2 + t) * kWave + lane) * 4;
    const int col = lane & 15, grp = lane >> 4;
    return (mb * 16 + col) * (32 * kWG) + 32 * wave + 16 * t + 4 * grp;
}

// Persistent stream over the workgroup's unit range [x0, x1).  The loads of
// the unit PD - 1 places ahead are issued while a unit is contracted, across
// item boundaries: one pipeline for the whole range, never drained in between.
template <int FMT, bool DOWN, int PD, bool MXA>
__global__ __launch_bounds__(kEThreads) __attribute__((amdgpu_waves_per_eu(kVPW == 1 ? 2 : 1, kVPW == 1 ? 2 : 1)))
void expert_ffn_kernel(FfnParams P)
{
    static_assert(!MXA || FMT == FMT_MXFP4, "MX activations take MXFP4 weights");
    static_assert(!MXA || 2 * (kScaleQ + kMB * 16 * 8) <= 2 * BTile<Fmt<FMT>::kBlocks>::kBuf, "MX tile fits the LDS");
    constexpr int NV = Fmt<FMT>::kVecs, SB = Fmt<FMT>::kBlocks;
    constexpr int BBUF = BTile<SB>::kBuf, NT = kTiles(PD, MXA);
    constexpr uint32_t BLK = 1024u * NV;  // bytes of one 16 x 128 block of a tile
    __shared__ __attribute__((aligned(16))) uint8_t lds[NT * BBUF];
    const VerifyArgs &a = P.a;
    // Workgroups are dispatched round-robin over the 8 XCDs; taking the ranges
    // XCD-major gives each XCD one contiguous eighth of the units, so the
    // workgroups sharing an L2 work on neighbouring items (the same experts'
    // token rows) instead of the same band slice of every expert.
    const int w = P.workers % 8 == 0 ? (int)(blockIdx.x % 8) * (P.workers / 8) + (int)(blockIdx.x / 8) : (int)blockIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int lane = lane_id(), col = lane & 15, grp = lane >> 4;
    const int tid = threadIdx.x, br = tid >> 4, bc = tid & 15;
    const int nsteps = P.nsteps, K = P.K;
    __shared__ Split sp;
    static_assert(NT * BBUF >= kPW * 1024 * 4, "the union's scratch fits the activation tiles");
    const bool sched_in = DOWN && P.dn_sched != nullptr && P.plan == nullptr;
    const Plan pl = !DOWN && P.plan == nullptr ? union_and_costs<FMT, MXA>(P, sp, reinterpret_cast<int *>(lds))
                  : sched_in                   ? load_down_sched(P, sp)
                                               : build_costs<FMT, MXA, DOWN>(P, sp);
    if (!sched_in) build_bounds(sp, pl.n_groups, (long)P.nbands * nsteps, P.workers);
    if (!DOWN && P.dn_sched != nullptr && P.plan == nullptr && blockIdx.x == 0) write_down_sched(P, pl, sp);
    // Unit indices fit in 32 bits (fewer than 2^30 units: every matrix is below 2^31 bytes and a
    // launch has at most 4096 token groups), so the unit arithmetic below is 32-bit.
    const int x0 = (int)sp.bound[w], x1 = (int)sp.bound[w + 1];
    // For the fix-up (gate/up) and combine (down) kernels, written when the
    // range is done: the range, and the cut gate/up item it finishes.
    auto write_records = [&]() {
        if (threadIdx.x == 0) {
            P.ranges[2 * w] = x0;
            P.ranges[2 * w + 1] = x1;
            if (!DOWN) write_fix_record(P, pl, sp, w, x0, x1);
        }
    };
    if (x0 >= x1) {  // no units, no item
        write_records();
        return;
    }
    const uint32_t rows = (uint32_t)(DOWN ? a.T * a.k + (a.sh_gate ? a.T : 0) : a.T);
    // Activation rows: bf16 x or H, or (MX) e4m3fn codes of K padded to nblocks * 128 and their block scales.
    const uint32_t brow_bytes = MXA ? (uint32_t)P.nblocks * kMacroK : (uint32_t)(DOWN ? a.d_ff : a.d) * 2u;
    const rsrc_t rb = make_rsrc(MXA ? static_cast<const void *>(DOWN ? a.hq : a.xq)
                                    : static_cast<const void *>(DOWN ? a.h : a.x), rows * brow_bytes);
    const rsrc_t rsa = make_rsrc(DOWN ? a.hs : a.xs, MXA ? rows * (uint32_t)P.nblocks * 4u : 0u);
    const u32x4 rbw = rsrc_words(DOWN ? static_cast<const void *>(a.h) : static_cast<const void *>(a.x), rows * brow_bytes);

    // Processing order: from the range's first item boundary to its end, then
    // the head piece before that boundary.  All workgroups thus start their
    // whole items at step 0 and walk K in phase, which streams faster than
    // ranges at scattered K offsets (measured: gate/up -2% at 32 experts,
    // -1.2% at 128).  Each piece is still summed in K order, so the results do
    // not change.
    const uint32_t uns = (uint32_t)nsteps;
    auto item_of = [&](int u) { return (int)((uint32_t)u / uns); };
    const int n = x1 - x0;
    const int b0 = (int)(((uint32_t)x0 + uns - 1u) / uns * uns);  // first item boundary at or after x0
    const int rot = b0 < x1 ? b0 - x0 : 0;
    auto unit_of = [&](int i) { return i < n - rot ? x0 + rot + i : x0 + i - (n - rot); };

    Source src;
    set_source<FMT, DOWN, MXA>(src, P, sp, item_of(unit_of(0)));

    WFrag<FMT> wf[PD][kNT];
    u32x4 bst[MXA ? PD : 1][kBPass][SB];      // MX: the activation codes of a step
    uint32_t sst[MXA ? PD : 1][kBPass];       // MX: the rows' block scales of a step (threads bc < 2)
    // Vector-memory instructions per unit: weight side (weights and scales, plus MX activations)
    // and direct activation loads.  Every unit issues exactly these, past the range too (loads
    // of zeros: offsets beyond every buffer), so that the counted wait below is exact.
    constexpr int kLdW = kNT * NV * SB + (FMT == FMT_FP8 ? kNT * SB : FMT == FMT_MXFP4 ? kNT : 0) + (MXA ? 2 * kBPass : 0);
    constexpr int kLdA = MXA ? 0 : kBPass * SB;
    // Weight-side loads of the i-th unit of the sequence into ring slot `slot`.
    auto issue_w = [&](int slot, int i) {
        const bool ok = i < n;
        const int v = ok ? unit_of(i) : src.ib;
        if (ok && (v < src.ib || v >= src.ie)) set_source<FMT, DOWN, MXA>(src, P, sp, item_of(v));
        const uint32_t step = (uint32_t)(v - src.ib);
#pragma unroll
        for (int b = 0; b < SB; ++b) {
            // Block kb of the tile; a step's second block can lie past the last one.
            const uint32_t kb = step * SB + b;
            const bool okb = ok && (SB == 1 || (int)kb < P.nblocks);
            const uint32_t so = kb * src.kstride;
#pragma unroll
            for (int tt = 0; tt < kNT; ++tt)
#pragma unroll
                for (int i = 0; i < NV; ++i)
                    wf[slot][tt].v[b * NV + i] = load16<kAuxNT>(tt % 2 ? src.ra1 : src.ra0, okb ? src.a[tt] + so + 1024u * i : kOff);
            if constexpr (FMT == FMT_FP8) {
                const uint32_t sso = kb * 4u;
#pragma unroll
                for (int tt = 0; tt < kNT; ++tt)
                    wf[slot][tt].scale = __builtin_bit_cast(
                        float, __builtin_amdgcn_raw_buffer_load_b32(tt % 2 ? src.rs1 : src.rs0, (int)(okb ? src.q[tt] + sso : kOff),
                                                                    0, 0));
            } else if constexpr (FMT == FMT_MXFP4) {
                // The quad holding the step's blocks (kb0 = step * SB is even, so both lie in it).
                if (b == 0) {
                    const uint32_t sso = (kb >> 2) * 256u;
#pragma unroll
                    for (int tt = 0; tt < kNT; ++tt) {
                        wf[slot][tt].code = __builtin_amdgcn_raw_buffer_load_b32(tt % 2 ? src.rs1 : src.rs0,
                                                                                 (int)(okb ? src.q[tt] + sso : kOff), 0, 0);
                        wf[slot][tt].shift = (int)(kb & 3u) * 8;
                    }
                }
            }
        }
        if constexpr (MXA) {
            // A step's 2 x 128 codes of a row are 256 contiguous bytes (16 per thread),
            // its 8 block scales two dwords (threads bc = 0, 1).
            const bool aok = ok && (int)(step * SB + (bc >> 3)) < P.nblocks;
            const bool sok = ok && bc < 2 && (int)(step * SB + (bc & 1)) < P.nblocks;
#pragma unroll
            for (int i = 0; i < kBPass; ++i) {
                // A row's kOff plus the in-range step offset stays beyond the buffer: zeros.
                bst[slot][i][0] = load16<0>(rb, aok ? src.boff[i] + step * 256u : kOff);
                sst[slot][i] = __builtin_amdgcn_raw_buffer_load_b32(rsa, (int)(sok ? src.soff[i] + step * 8u : kOff), 0, 0);
            }
        }
    };
    // Activation tile of the i-th unit straight into LDS tile i % PD (bf16 activations): pass p,
    // block b of this wavefront covers token rows kBRowsPerPass p + 4 wave .. + 3, 1 KiB of the tile.  Rows
    // past the item's tokens and elements past K read zeros.  Uses the sources issue_w(i) set.
    auto issue_a = [&](int i) {
        if constexpr (!MXA) {
            const bool ok = i < n;
            const int v = ok ? unit_of(i) : src.ib;
            const uint32_t step = (uint32_t)(v - src.ib);
            const uint32_t tile = lds_addr(lds) + (uint32_t)((i % PD) * BBUF + 4 * wave * 256);
#pragma unroll
            for (int b = 0; b < SB; ++b) {
                const uint32_t kb = step * SB + b;
                const bool kok = ok && (SB == 1 || (int)kb < P.nblocks) && (int)kb * kMacroK + src.kc < K;
#pragma unroll
                for (int p = 0; p < kBPass; ++p)  // a row's kOff plus kb * 256 stays beyond the buffer: zeros
                    load16_lds(rbw, kok ? src.boff[p] + kb * 256u : kOff,
                               tile + (uint32_t)(b * BTile<SB>::kBlk + p * kBRowsPerPass * 256));
            }
        }
    };

    // The item being contracted.
    int citem = item_of(unit_of(0));
    ItemDesc cd = describe_lds<DOWN>(P, sp, citem);
    ItemBias cbias[kVPW];
#pragma unroll
    for (int j = 0; j < kVPW; ++j) cbias[j] = load_bias<DOWN>(P, cd, wave * kVPW + j);
    int cib = citem * nsteps;
    f32x4 acc[kNT][kMB];
#pragma unroll
    for (int t = 0; t < kNT; ++t)
#pragma unroll
        for (int mb = 0; mb < kMB; ++mb) acc[t][mb] = f32x4{0.f, 0.f, 0.f, 0.f};

    // One step: the weight loads of the unit PD - 1 places ahead, the wait
    // for unit i's activation tile and the barrier, the direct activation
    // loads of the unit PD - 1 places ahead (into the tile unit i - 1 used),
    // then unit i's contraction.  Only this part depends on the ring slot, so
    // only it is replicated per unrolled step.  MX activations are staged
    // through registers and stored to LDS before the barrier instead.
    auto step = [&](int slot, int par, int i) {
        issue_w((slot + PD - 1) % PD, i + PD - 1);
        if (i >= n) return;  // the last round of the unrolled loop runs past the range
        const int nmb = (cd.M + 15) / 16;
        uint8_t *buf = lds + par * BBUF;
        if constexpr (MXA) {
            // After the previous step's barrier no wavefront still reads this buffer.
#pragma unroll
            for (int i = 0; i < kBPass; ++i) {
                *reinterpret_cast<u32x4 *>(buf + (i * kBRowsPerPass + br) * kRowQ + bc * 16) = bst[slot][i][0];
                if (bc < 2)
                    *reinterpret_cast<uint32_t *>(buf + kScaleQ + (i * kBRowsPerPass + br) * 8 + bc * 4) = sst[slot][i];
            }
            __syncthreads();
        } else {
            // This wavefront's direct loads of unit i have landed once at most the loads issued
            // after them are outstanding: PD - 2 whole units and the weight side of unit
            // i + PD - 1.  (A workgroup barrier with a fence would wait for every direct load,
            // the prefetched ones too.)  The barrier then publishes all wavefronts' parts.
            asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"((PD - 2) * (kLdW + kLdA) + kLdW) : "memory");
            issue_a(i + PD - 1);
        }
        if constexpr (MXA) {
            contract_mx(wf[slot], buf, acc, nmb);
        } else {
            contract<FMT>(wf[slot], buf, acc, nmb);
        }
    };

    // End of a piece (an item boundary, the range's end or the end of the
    // sequence): finish the item, or park its partial sums if it is cut at
    // either end of the range, and move on to the next piece.  It runs a few
    // times per range: every copy of it is cold in the instruction cache, so
    // the loop keeps as few copies as it can (one per unrolled step).
    auto end_of_piece = [&](int i) {
        const int u = unit_of(i);
        const int nmb = (cd.M + 15) / 16;
        const int un = i + 1 < n ? unit_of(i + 1) : -1;
        if (u + 1 == cib + nsteps || un != u + 1) {
            if (cib >= x0 && cib + nsteps <= x1) {
                finish_item<DOWN, MXA, kVPW>(P, cd, wave, acc, cbias, sp.tok);
            } else {
                float *dst = P.partials + ((size_t)w * 2 + (cib <= x0 ? 0 : 1)) * P.slot_floats;
#pragma unroll
                for (int tt = 0; tt < kNT; ++tt)
#pragma unroll
                    for (int mb = 0; mb < kMB; ++mb)
                        if (mb < nmb)
                            *reinterpret_cast<f32x4 *>(dst + partial_offset<DOWN>(wave * kVPW + tt / 2, tt % 2, mb, lane)) =
                                acc[tt][mb];
            }
#pragma unroll
            for (int t = 0; t < kNT; ++t)
#pragma unroll
                for (int mb = 0; mb < kMB; ++mb) acc[t][mb] = f32x4{0.f, 0.f, 0.f, 0.f};
            if (un >= 0) {
                citem = item_of(un);
                cib = citem * nsteps;
                cd = describe_lds<DOWN>(P, sp, citem);
#pragma unroll
                for (int j = 0; j < kVPW; ++j) cbias[j] = load_bias<DOWN>(P, cd, wave * kVPW + j);
            }
        }
    };

#pragma unroll
    for (int j = 0; j < PD - 1; ++j) {
        issue_w(j, j);
        issue_a(j);
    }
    // The loop unrolls PD steps (ring slot j); the NT activation tiles (PD,
    // or 2 for MX activations at even PD) cycle with the slot, so PD steps
    // suffice, not 2 * PD: half the code, half the cold copies.
    for (int i0 = 0; i0 < n; i0 += PD) {
#pragma unroll
        for (int j = 0; j < PD; ++j) {
            step(j, j % NT, i0 + j);  // the last round may run past the range: loads of zeros only
            if (i0 + j < n) end_of_piece(i0 + j);
        }
    }
    // No direct load may still be writing this workgroup's LDS when it ends.
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    write_records();
    if (DOWN) record_outputs(P, pl, sp, x0, x1);
}

// Finishes the gate/up items cut between workgroups.  Block w handles the
// record of workgroup w (an item whose last unit, but not its first, lies in
// w's range): it adds the parked partial sums of the item's contributors, in
// workgroup order, and finishes the item.  The kernel boundary makes the
// expert kernel's records and partial sums visible here.
template <bool DOWN, bool MXA>
__global__ __launch_bounds__(kThreads) void expert_ffn_fixup_kernel(FfnParams P)
{
    const int lane = lane_id();
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int w = blockIdx.x;
    const long long *rec = P.fix + 4 * (size_t)w;
    const long long item = ld_s64(rec);
    if (item < 0) return;
    const long long cut = ld_s64(rec + 1);
    ItemDesc d{};
    const long long pe = ld_s64(rec + 2);
    d.p0 = (int)(uint32_t)pe;
    d.e = (int)(pe >> 32) - 1;
    d.shared = d.e < 0;
    d.M = (int)ld_s64(rec + 3);
    d.n0 = (int)(item % P.nbands) * P.band_rows;
    const int nmb = (d.M + 15) / 16;  // only the live token blocks were parked
    const ItemBias bias[1] = {load_bias<DOWN>(P, d, wave)};  // in flight with the partial sums
    f32x4 acc[2][kMB];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int mb = 0; mb < kMB; ++mb) acc[t][mb] = f32x4{0.f, 0.f, 0.f, 0.f};
    auto add = [&](const float *src) {
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int mb = 0; mb < kMB; ++mb)
                if (mb < nmb) acc[t][mb] += *reinterpret_cast<const f32x4 *>(src + partial_offset<DOWN>(wave, t, mb, lane));
    };
    if (split::packed_contributors(cut)) {
        // Up to three contributors: every load is issued before the first sum (one round trip;
        // absent contributors and dead token blocks read zeros), then added in workgroup order.
        const int cnt = split::packed_count(cut);
        const rsrc_t rp = make_rsrc(P.partials, (uint32_t)((size_t)P.workers * 2 * P.slot_floats * 4));
        f32x4 v[3][2][kMB];
#pragma unroll
        for (int i = 0; i < 3; ++i) {
            const uint32_t slot = (uint32_t)split::packed_slot(cut, i);
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int mb = 0; mb < kMB; ++mb)
                    v[i][t][mb] = __builtin_bit_cast(
                        f32x4, load16<0>(rp, (i < cnt && mb < nmb)
                                                 ? (slot * (uint32_t)P.slot_floats + (uint32_t)partial_offset<DOWN>(wave, t, mb, lane)) * 4u
                                                 : kOff));
        }
#pragma unroll
        for (int i = 0; i < 3; ++i)
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int mb = 0; mb < kMB; ++mb)
                    if (i < cnt && mb < nmb) acc[t][mb] += v[i][t][mb];
    } else {
        // More than three contributors: each one's slot follows from its range.
        const long ib = (long)item * P.nsteps, ie = ib + P.nsteps;
        for (int v = split::first_worker(cut), w1 = split::last_worker(cut); v <= w1; ++v) {
            const int slot = split::piece_slot(v, (long)ld_s64(P.ranges + 2 * v), (long)ld_s64(P.ranges + 2 * v + 1),
                                               ib, ie);
            if (slot >= 0) add(P.partials + (size_t)slot * P.slot_floats);
        }
    }
    finish_item<DOWN, MXA, 1>(P, d, wave, acc, bias);
}

// MX activation mode: x [T][K] bf16 -> e4m3fn codes [T][kp] in the FP8
// operand's lane order and e8m0 scales [T][kp / 32] (kp = K padded to a
// multiple of 128, zeros beyond K), one thread per block of 32 consecutive
// elements.  Block g of a chunk is K 32g..32g+31; its first 16 codes go to
// chunk byte 64 (g % 2) + 16 (g / 2), its last 16 to 32 bytes further.
__global__ __launch_bounds__(256) void mx_quant_x_kernel(const uint16_t *__restrict__ x, int T, int K, int kp,
                                                         uint8_t *__restrict__ xq, uint8_t *__restrict__ xs)
{
    const int nb = kp / 32;
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= T * nb) return;
    const int row = i / nb, blk = i - row * nb, c = blk >> 2, g = blk & 3;
    float v[32];
    u32x4 w[4] = {u32x4{0u, 0u, 0u, 0u}, u32x4{0u, 0u, 0u, 0u}, u32x4{0u, 0u, 0u, 0u}, u32x4{0u, 0u, 0u, 0u}};
    if (32 * blk < K) {  // K % 32 == 0: a block is all in range or all out
        const u32x4 *src = reinterpret_cast<const u32x4 *>(x + (size_t)row * K + 32 * blk);
#pragma unroll
        for (int j = 0; j < 4; ++j) w[j] = src[j];
    }
#pragma unroll
    for (int j = 0; j < 32; ++j) {
        const uint32_t word = w[j >> 3][(j >> 1) & 3];
        v[j] = bf16_bits_to_f32((uint16_t)(j & 1 ? word >> 16 : word & 0xffffu));
    }
    float amax = 0.f;
#pragma unroll
    for (int j = 0; j < 32; ++j) amax = fmaxf(amax, fabsf(v[j]));
    const int E = mx_exponent(amax);
    const float inv = mx_inv_scale(E);
    u32x4 q[2];
#pragma unroll
    for (int j = 0; j < 8; ++j)
        q[j >> 2][j & 3] = e4m3_code(v[4 * j] * inv) | (e4m3_code(v[4 * j + 1] * inv) << 8) |
                           (e4m3_code(v[4 * j + 2] * inv) << 16) | (e4m3_code(v[4 * j + 3] * inv) << 24);
    uint8_t *dst = xq + (size_t)row * kp + c * 128 + 64 * (g & 1) + 16 * (g >> 1);
    *reinterpret_cast<u32x4 *>(dst) = q[0];
    *reinterpret_cast<u32x4 *>(dst + 32) = q[1];
    xs[(size_t)row * nb + blk] = (uint8_t)(E + 127);
}

// Token groups when some expert may have more than 64 tokens (T > 64):
// plan[0] = number of groups; plan[8 + 2i], plan[8 + 2i + 1] = (expert
// position, group index within the expert) of group i, in expert order;
// plan[8 + 2 * kMaxGroups + u] = first group of expert position u.
__global__ __launch_bounds__(256) void plan_kernel(VerifyArgs a, int32_t *plan)
{
    __shared__ int wave_tot[256 / kWave];
    const int U = *a.n_unique;
    const int n_exp = U + (a.sh_gate ? 1 : 0);
    int run = 0;
    for (int base = 0; base < n_exp; base += blockDim.x) {
        const int u = base + threadIdx.x;
        int n = 0;
        if (u < n_exp) {
            const int M = u < U ? a.offsets[u + 1] - a.offsets[u] : a.T;
            n = (M + kTokGroup - 1) / kTokGroup;
        }
        int tot = 0;
        const int pos = block_exclusive_scan(n, wave_tot, &tot);
        if (u < n_exp) plan[8 + 2 * kMaxGroups + u] = run + pos;  // first group of expert position u
        for (int g = 0; g < n; ++g) {
            plan[8 + 2 * (run + pos + g)] = u;
            plan[8 + 2 * (run + pos + g) + 1] = g;
        }
        run += tot;
    }
    if (threadIdx.x == 0) plan[0] = run;
}

// A row of a down item cut over two or three ranges (descriptor kind 1): its
// parked partial sums, all loads issued at once (absent ones read zeros) and
// added in workgroup order.
__device__ __forceinline__ f32x4 parked_sum(const FfnParams &D, uint64_t ds, int c)
{
    const int off = split::out_row(ds) * D.band_rows + c % D.band_rows;  // partial_offset<true>
    const int cnt = split::out_count(ds);
    const rsrc_t rp = make_rsrc(D.partials, (uint32_t)((size_t)D.workers * 2 * D.slot_floats * 4));
    const uint32_t sf = (uint32_t)D.slot_floats;
    const f32x4 v0 = __builtin_bit_cast(f32x4, load16<0>(rp, ((uint32_t)split::out_slot(ds, 0) * sf + (uint32_t)off) * 4u));
    const f32x4 v1 = __builtin_bit_cast(
        f32x4, load16<0>(rp, cnt > 1 ? ((uint32_t)split::out_slot(ds, 1) * sf + (uint32_t)off) * 4u : kOff));
    const f32x4 v2 = __builtin_bit_cast(
        f32x4, load16<0>(rp, cnt > 2 ? ((uint32_t)split::out_slot(ds, 2) * sf + (uint32_t)off) * 4u : kOff));
    return cnt > 2 ? v0 + v1 + v2 : cnt > 1 ? v0 + v1 : v0;
}

// The same for a row of an item cut over more than three ranges w0..w1, eight
// contributors at a time: their partial sums in one round trip (kind 2: slot
// 2*w0 + tail0, then each later range's head piece), or, if some range in
// between is empty (kind 3), the ranges first to skip the empty ones.
__device__ __forceinline__ f32x4 expert_out_walk(const FfnParams &D, uint64_t ds, int c)
{
    constexpr int CW = 8;
    const int off = split::out_row(ds) * D.band_rows + c % D.band_rows;
    const int w0 = split::out_w0(ds), w1 = split::out_w1(ds);
    const bool check = split::out_kind(ds) == 3;
    f32x4 s = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int v0 = w0; v0 <= w1; v0 += CW) {
        bool live[CW];
#pragma unroll
        for (int q = 0; q < CW; ++q) live[q] = v0 + q <= w1;
        if (check) {
            long long rg[CW][2];
#pragma unroll
            for (int q = 0; q < CW; ++q) {
                const int v = min(v0 + q, w1);
                rg[q][0] = D.ranges[2 * v];
                rg[q][1] = D.ranges[2 * v + 1];
            }
#pragma unroll
            for (int q = 0; q < CW; ++q) live[q] = live[q] && rg[q][0] < rg[q][1];
        }
        f32x4 pv[CW];
#pragma unroll
        for (int q = 0; q < CW; ++q) {
            const int v = v0 + q;
            const int slot = v == w0 ? 2 * w0 + split::out_tail0(ds) : 2 * v;
            pv[q] = live[q] ? *reinterpret_cast<const f32x4 *>(D.partials + (size_t)slot * D.slot_floats + off)
                            : f32x4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int q = 0; q < CW; ++q)
            if (live[q]) s += pv[q];
    }
    return s;
}

// y[t] = sum_j w[t][j] * (O[slot t*k + j] + b_down[expert of the slot]) (+ shared) -> bf16, summed in the
// order j = 0..k-1, then the shared expert; 4 columns per thread.  D is the
// down launch's geometry.  The k slots are handled 8 at a time: each stage
// loads its slots' experts, gate weights and output descriptors together, the
// shared expert's descriptor going with the first stage's, then every output
// row the descriptors name, so the kernel waits on global memory twice per
// stage.  Rows of items cut over more than three ranges (small batches spread
// thin over the workgroups) are walked afterwards, one at a time, so that the
// common path stays short.
__global__ __launch_bounds__(256) void combine_kernel(FfnParams D)
{
    constexpr int CH = 8;
    const VerifyArgs &a = D.a;
    const int per_row = a.d / 4;
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= a.T * per_row) return;
    const int t = i / per_row, c = (i - t * per_row) * 4;
    const int band = c / D.band_rows;
    const int S = a.T * a.k;
    const bool sh = a.sh_gate != nullptr;
    const rsrc_t ro = make_rsrc(a.o, (uint32_t)((size_t)(S + (sh ? a.T : 0)) * a.d * 4));
    f32x4 s = f32x4{0.f, 0.f, 0.f, 0.f}, vsh = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int j0 = 0; j0 < a.k; j0 += CH) {
        const bool with_sh = sh && j0 == 0;
        int ej[CH];
        float wj[CH];
        uint64_t dj[CH];
        f32x4 oj[CH], vj[CH];
        bool ok[CH];
        // One round trip: the slots' experts, gate weights and descriptors, and their rows of O
        // (a whole item's output; unused for a cut item's row).
#pragma unroll
        for (int q = 0; q < CH; ++q) {
            const int slot = t * a.k + min(j0 + q, a.k - 1);
            ej[q] = a.topk_idx[slot];
            wj[q] = a.topk_w[slot];
            dj[q] = a.desc[(size_t)slot * D.nbands + band];
            oj[q] = __builtin_bit_cast(f32x4, load16<0>(ro, (uint32_t)((size_t)slot * a.d + c) * 4u));
        }
        const uint64_t dsh = with_sh ? a.desc[(size_t)(S + t) * D.nbands + band] : 0ull;
        const f32x4 osh = with_sh ? __builtin_bit_cast(f32x4, load16<0>(ro, (uint32_t)((size_t)(S + t) * a.d + c) * 4u))
                                  : f32x4{0.f, 0.f, 0.f, 0.f};
        // vj[q] = O + b_down of slot q.  A slot whose expert lies outside [0, E) was never placed:
        // it adds nothing and its (unwritten) descriptor is not used.  A cut item's row is the sum
        // of its parked partial sums (kind 1), or needs the walk (kinds 2, 3): it holds b_down for
        // now (its walk sum w is added as w + b below, the same operation as O + b).
        uint32_t walk = 0;  // bit q: slot q's row needs the walk; bit CH: the shared expert's
#pragma unroll
        for (int q = 0; q < CH; ++q) {
            ok[q] = j0 + q < a.k && (unsigned)ej[q] < (unsigned)a.E;
            const int kind = ok[q] ? split::out_kind(dj[q]) : 0;
            const f32x4 b = a.b_down && ok[q] ? *reinterpret_cast<const f32x4 *>(a.b_down + (size_t)ej[q] * a.d + c)
                                              : f32x4{0.f, 0.f, 0.f, 0.f};
            const f32x4 v = kind == 0 ? oj[q] : kind == 1 ? parked_sum(D, dj[q], c) : f32x4{0.f, 0.f, 0.f, 0.f};
            const bool wk = kind >= 2;
            vj[q] = a.b_down ? (wk ? b : v + b) : v;
            if (wk) walk |= 1u << q;
        }
        if (with_sh) {
            const int kind = split::out_kind(dsh);
            vsh = kind == 0 ? osh : kind == 1 ? parked_sum(D, dsh, c) : f32x4{0.f, 0.f, 0.f, 0.f};
            if (kind >= 2) walk |= 1u << CH;
        }
        while (walk) {
            const int q = __builtin_ctz(walk);
            walk &= walk - 1;
            uint64_t dq = dsh;
#pragma unroll
            for (int qq = 0; qq < CH; ++qq)
                if (qq == q) dq = dj[qq];
            const f32x4 v = expert_out_walk(D, dq, c);
#pragma unroll
            for (int qq = 0; qq < CH; ++qq)
                if (qq == q) vj[qq] = a.b_down ? v + vj[qq] : v;
            if (q == CH) vsh = v;
        }
#pragma unroll
        for (int q = 0; q < CH; ++q)
            if (ok[q]) s += wj[q] * vj[q];
    }
    if (sh) s += vsh;
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

int verify_workers()
{
    const int w = device_cus() * ECOSPEC_WG_PER_CU;
    return w < kMaxWorkers ? w : kMaxWorkers;
}

// Token groups a plan can hold: one per expert (<= 1024 routed + 1 shared)
// plus one per extra 64 tokens.
static int plan_capacity(int T, int k, bool shared)
{
    const long rows = (long)T * k + (shared ? T : 0);
    return (int)(1025 + (rows + kTokGroup - 1) / kTokGroup);
}

VerifyWorkspace verify_workspace(int d, int d_ff, int T, int k, bool shared, bool mx, int workers)
{
    auto align = [](size_t v) { return (v + 255) & ~(size_t)255; };
    const size_t rows = (size_t)T * k + (shared ? (size_t)T : 0);
    VerifyWorkspace w;
    w.h_offset = 0;
    w.h_bytes = rows * d_ff * 2;
    w.o_offset = align(w.h_bytes);
    w.o_bytes = rows * d * 4;
    w.p_offset = w.o_offset + align(w.o_bytes);
    // partial sums, unit ranges, fix-up records
    w.workers = workers;
    w.slot_floats = partial_floats(T);
    w.p_bytes = (size_t)workers * 2 * w.slot_floats * 4 + (size_t)workers * 2 * 8 + (size_t)workers * 4 * 8;
    w.plan_cap = plan_capacity(T, k, shared);
    w.plan_offset = w.p_offset + align(w.p_bytes);
    w.plan_bytes = (8 + 2 * (size_t)kMaxGroups + 1026) * 4;  // groups, then first group per expert
    w.desc_offset = w.plan_offset + align(w.plan_bytes);
    w.desc_bytes = rows * ((d + 32 * kWG - 1) / (32 * kWG)) * 8;  // one output descriptor per row and down band
    // MX activations: x codes + scales, then H codes + scales (rows padded to multiples of 128).
    const size_t kpd = (size_t)(d + kMacroK - 1) / kMacroK * kMacroK, kpf = (size_t)(d_ff + kMacroK - 1) / kMacroK * kMacroK;
    w.mx_offset = w.desc_offset + align(w.desc_bytes);
    w.mx_bytes = mx ? align((size_t)T * kpd) + align((size_t)T * kpd / 32) + align(rows * kpf) + align(rows * kpf / 32) : 0;
    w.total = w.mx_offset + align(w.mx_bytes);
    return w;
}

static hipError_t mark(hipEvent_t const *events, int i, hipStream_t stream)
{
    return (events && events[i]) ? hipEventRecord(events[i], stream) : hipSuccess;
}

template <int FMT, bool MXA>
static hipError_t launch_fmt(const VerifyArgs &args, uint8_t *ws_base, const VerifyWorkspace &ws, hipStream_t stream,
                             hipEvent_t const *events)
{
    constexpr int PD = FMT == FMT_BF16 ? ECOSPEC_PD_BF16 : FMT == FMT_FP8 ? ECOSPEC_PD_FP8 : ECOSPEC_PD_FP4;
    const int G = ws.workers;
    const bool grouped = args.T > kTokGroup;  // some expert may need several token groups
    VerifyArgs a = args;
    a.h = reinterpret_cast<uint16_t *>(ws_base + ws.h_offset);
    a.o = reinterpret_cast<float *>(ws_base + ws.o_offset);
    a.desc = reinterpret_cast<uint64_t *>(ws_base + ws.desc_offset);
    float *partials = reinterpret_cast<float *>(ws_base + ws.p_offset);
    int32_t *plan = reinterpret_cast<int32_t *>(ws_base + ws.plan_offset);
    hipError_t err;

    if (grouped) {
        // The token-group plan needs the union first; without it the gate/up kernel builds the union itself.
        if ((err = launch_expert_union(a.topk_idx, a.T, a.k, a.E, a.counts, a.union_ids, a.n_unique, a.offsets,
                                       a.perm, stream)) != hipSuccess)
            return err;
        hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(256), 0, stream, a, plan);
        if ((err = hipGetLastError()) != hipSuccess) return err;
    }
    if ((err = mark(events, 0, stream)) != hipSuccess) return err;
    if constexpr (MXA) {
        auto align = [](size_t v) { return (v + 255) & ~(size_t)255; };
        const size_t rows = (size_t)a.T * a.k + (a.sh_gate ? (size_t)a.T : 0);
        const int kpd = (a.d + kMacroK - 1) / kMacroK * kMacroK, kpf = (a.d_ff + kMacroK - 1) / kMacroK * kMacroK;
        a.xq = ws_base + ws.mx_offset;
        a.xs = a.xq + align((size_t)a.T * kpd);
        a.hq = a.xs + align((size_t)a.T * kpd / 32);
        a.hs = a.hq + align(rows * kpf);
        const int n = a.T * (kpd / 32);
        hipLaunchKernelGGL(mx_quant_x_kernel, dim3((n + 255) / 256), dim3(256), 0, stream, a.x, a.T, a.d, kpd, a.xq,
                           a.xs);
        if ((err = hipGetLastError()) != hipSuccess) return err;
    }
    FfnParams g{};
    g.a = a;
    g.N = a.d_ff;
    g.K = a.d;
    constexpr int SB = Fmt<FMT>::kBlocks;
    g.nblocks = (a.d + kMacroK - 1) / kMacroK;
    g.nsteps = (g.nblocks + SB - 1) / SB;
    g.band_rows = 16 * kWG;
    g.nbands = (a.d_ff + g.band_rows - 1) / g.band_rows;
    g.workers = G;
    g.mat_bytes = packed_matrix_bytes(FMT, a.d_ff, a.d);
    g.sc_bytes = packed_scale_bytes(FMT, a.d_ff, a.d);
    g.partials = partials;
    g.slot_floats = ws.slot_floats;
    g.ranges = reinterpret_cast<long long *>(partials + (size_t)G * 2 * ws.slot_floats);
    g.fix = g.ranges + (size_t)G * 2;
    g.plan = grouped ? plan : nullptr;
    // Without a plan the (unused) plan region holds the down launch's schedule.
    static_assert(sizeof(DownSched) <= (8 + 2 * (size_t)kMaxGroups + 1026) * 4, "the down schedule fits the plan region");
    g.dn_sched = grouped ? nullptr : static_cast<void *>(plan);
    {
        const int dn_nsteps = ((a.d_ff + kMacroK - 1) / kMacroK + SB - 1) / SB;
        const int dn_nbands = (a.d + 32 * kWG - 1) / (32 * kWG);
        g.dn_K = dn_nbands * dn_nsteps;
    }
    hipLaunchKernelGGL((expert_ffn_kernel<FMT, false, PD, MXA>), dim3(G), dim3(kEThreads), 0, stream, g);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    if ((err = mark(events, 1, stream)) != hipSuccess) return err;
    hipLaunchKernelGGL((expert_ffn_fixup_kernel<false, MXA>), dim3(G), dim3(kThreads), 0, stream, g);
    if ((err = hipGetLastError()) != hipSuccess) return err;

    FfnParams dn = g;
    dn.N = a.d;
    dn.K = a.d_ff;
    dn.nblocks = (a.d_ff + kMacroK - 1) / kMacroK;
    dn.nsteps = (dn.nblocks + SB - 1) / SB;
    dn.band_rows = 32 * kWG;
    dn.nbands = (a.d + dn.band_rows - 1) / dn.band_rows;
    dn.mat_bytes = packed_matrix_bytes(FMT, a.d, a.d_ff);
    dn.sc_bytes = packed_scale_bytes(FMT, a.d, a.d_ff);
    if ((err = mark(events, 2, stream)) != hipSuccess) return err;
    hipLaunchKernelGGL((expert_ffn_kernel<FMT, true, PD, MXA>), dim3(G), dim3(kEThreads), 0, stream, dn);
    if ((err = hipGetLastError()) != hipSuccess) return err;

    // Combine also adds up the down items cut between workgroups.
    const int n = a.T * (a.d / 4);
    if ((err = mark(events, 3, stream)) != hipSuccess) return err;
    hipLaunchKernelGGL(combine_kernel, dim3((n + 255) / 256), dim3(256), 0, stream, dn);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    return mark(events, 4, stream);
}

hipError_t launch_verify(const VerifyArgs &a, void *workspace, const VerifyWorkspace &ws, hipStream_t stream,
                         hipEvent_t const *events)
{
    uint8_t *base = static_cast<uint8_t *>(workspace);
    switch (a.fmt) {
    case FMT_BF16: return launch_fmt<FMT_BF16, false>(a, base, ws, stream, events);
    case FMT_FP8: return launch_fmt<FMT_FP8, false>(a, base, ws, stream, events);
    case FMT_MXFP4:
        return a.act_fmt == 1 ? launch_fmt<FMT_MXFP4, true>(a, base, ws, stream, events)
                              : launch_fmt<FMT_MXFP4, false>(a, base, ws, stream, events);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace ecospec
