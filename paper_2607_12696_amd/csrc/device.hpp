// Device-side helpers shared by the gfx950 kernels of the verification pass.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ecospec {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;

constexpr int kWave = 64;

typedef __amdgpu_buffer_rsrc_t rsrc_t;

// Buffer offset beyond every range used here (all ranges are below 2 GiB):
// a load at it returns zeros.
constexpr uint32_t kOff = 0x80000000u;

// Raw buffer descriptor over [p, p + bytes): loads at offsets >= bytes return 0.
// The base goes through readfirstlane: descriptors must live in scalar
// registers, and a descriptor the compiler cannot prove wave-uniform would
// turn every load into a loop over the distinct values in the wave.
__device__ __forceinline__ rsrc_t make_rsrc(const void *p, uint32_t bytes)
{
    const uint64_t v = reinterpret_cast<uintptr_t>(p);
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
    void *u = reinterpret_cast<void *>(((uint64_t)hi << 32) | lo);
    return __builtin_amdgcn_make_buffer_rsrc(u, 0, (int)__builtin_amdgcn_readfirstlane(bytes), 0x00020000);
}

template <int AUX>
__device__ __forceinline__ u32x4 load16(rsrc_t r, uint32_t off)
{
    return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, AUX));
}

// The descriptor of make_rsrc as its four dwords (base, stride 0, range,
// format word), for the direct-to-LDS load below.
__device__ __forceinline__ u32x4 rsrc_words(const void *p, uint32_t bytes)
{
    const uint64_t v = reinterpret_cast<uintptr_t>(p);
    return u32x4{(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)v),
                 (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(v >> 32)) & 0xffffu,
                 (uint32_t)__builtin_amdgcn_readfirstlane(bytes), 0x00020000u};
}

// LDS address of a pointer into a __shared__ array.
__device__ __forceinline__ uint32_t lds_addr(const void *p)
{
    return (uint32_t)reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) void *)p);
}

// 16 bytes per lane from a raw buffer straight into LDS: lane l's bytes land
// at lds + 16 l (lds wave-uniform, passed to the hardware in M0, which needs
// one wait state before the load reads it); offsets beyond the buffer's range
// write zeros.  The load counts in vmcnt like any other; it is written as
// assembly because the compiler, seeing an LDS write it cannot place, would
// make every later LDS read wait for all outstanding loads.  Callers
// therefore wait for it themselves (s_waitcnt vmcnt); the compiler's own waits
// for other loads only grow stricter from loads it does not know about.
__device__ __forceinline__ void load16_lds(const u32x4 &rsrc, uint32_t off, uint32_t lds)
{
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %2, 0 offen lds" ::"v"(off), "s"(lds), "s"(rsrc)
                 : "memory", "m0");
}

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

// Butterfly reductions over the 64 lanes of a wavefront; every lane gets the result.
__device__ __forceinline__ float wave_sum(float v)
{
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
    return v;
}

// Maximum of a 64-bit value over the wavefront, with DPP lane moves (row
// shifts within each row of 16 lanes, then row broadcasts): lane 63 ends with
// the maximum, which is then read back as a uniform value.  Lanes a move does
// not reach see 0, the identity of an unsigned maximum.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint64_t dpp_max_step(uint64_t v)
{
    const uint32_t lo = __builtin_amdgcn_update_dpp(0u, (uint32_t)v, CTRL, ROW_MASK, 0xf, false);
    const uint32_t hi = __builtin_amdgcn_update_dpp(0u, (uint32_t)(v >> 32), CTRL, ROW_MASK, 0xf, false);
    const uint64_t o = ((uint64_t)hi << 32) | lo;
    return o > v ? o : v;
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v)
{
    v = dpp_max_step<0x111, 0xf>(v);  // row_shr:1
    v = dpp_max_step<0x112, 0xf>(v);  // row_shr:2
    v = dpp_max_step<0x114, 0xf>(v);  // row_shr:4
    v = dpp_max_step<0x118, 0xf>(v);  // row_shr:8: lane 15 of each row holds the row's maximum
    v = dpp_max_step<0x142, 0xa>(v);  // row_bcast:15 into rows 1 and 3
    v = dpp_max_step<0x143, 0xc>(v);  // row_bcast:31 into rows 2 and 3: lane 63 holds the maximum
    const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)v, 63);
    const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(v >> 32), 63);
    return ((uint64_t)hi << 32) | lo;
}

// Inclusive sum over lanes 0..lane of a wavefront: the same DPP steps as the
// maximum above (an inclusive scan within each row of 16 lanes, then the row
// totals carried into the later rows), a few cycles each, where a ds_bpermute
// shuffle waits on the LDS crossbar at every step.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ int dpp_add_step(int v)
{
    return v + __builtin_amdgcn_update_dpp(0, v, CTRL, ROW_MASK, 0xf, false);
}

__device__ __forceinline__ int wave_inclusive_sum(int v)
{
    v = dpp_add_step<0x111, 0xf>(v);  // row_shr:1
    v = dpp_add_step<0x112, 0xf>(v);  // row_shr:2
    v = dpp_add_step<0x114, 0xf>(v);  // row_shr:4
    v = dpp_add_step<0x118, 0xf>(v);  // row_shr:8: each row scanned
    v = dpp_add_step<0x142, 0xa>(v);  // row_bcast:15: row 0's total into row 1, row 2's into row 3
    v = dpp_add_step<0x143, 0xc>(v);  // row_bcast:31: lanes 0..31's total into rows 2 and 3
    return v;
}

// fp32 -> bf16 bits, round to nearest even (NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f)
{
    return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi)
{
    return (uint32_t)f32_to_bf16_bits(lo) | ((uint32_t)f32_to_bf16_bits(hi) << 16);
}

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b)
{
    return __uint_as_float((uint32_t)b << 16);
}

// Exclusive scan of one int per thread over the block; returns the total in *total.
__device__ __forceinline__ int block_exclusive_scan(int v, int *wave_tot, int *total)
{
    const int lane = lane_id(), wave = threadIdx.x / kWave, nwaves = blockDim.x / kWave;
    const int incl = wave_inclusive_sum(v);
    if (lane == kWave - 1) wave_tot[wave] = incl;
    __syncthreads();
    if (wave == 0) {
        const int w = wave_inclusive_sum(lane < nwaves ? wave_tot[lane] : 0);
        if (lane < nwaves) wave_tot[lane] = w;  // inclusive wave prefix
    }
    __syncthreads();
    const int before = wave > 0 ? wave_tot[wave - 1] : 0;
    *total = wave_tot[nwaves - 1];
    __syncthreads();  // wave_tot is reused by the next scan
    return before + incl - v;
}

// Two block-wide exclusive scans in one pass (three barriers for both).
// wave_tot: 2 * (blockDim.x / kWave) ints of LDS.
__device__ __forceinline__ void block_exclusive_scan2(int v0, int v1, int *wave_tot, int &ex0, int &ex1, int &tot0,
                                                      int &tot1)
{
    const int lane = lane_id(), wave = threadIdx.x / kWave, nwaves = blockDim.x / kWave;
    const int a = wave_inclusive_sum(v0), b = wave_inclusive_sum(v1);
    if (lane == kWave - 1) {
        wave_tot[wave] = a;
        wave_tot[nwaves + wave] = b;
    }
    __syncthreads();
    if (wave == 0) {
        const int wa = wave_inclusive_sum(lane < nwaves ? wave_tot[lane] : 0);
        const int wb = wave_inclusive_sum(lane < nwaves ? wave_tot[nwaves + lane] : 0);
        if (lane < nwaves) {
            wave_tot[lane] = wa;  // inclusive wave prefixes
            wave_tot[nwaves + lane] = wb;
        }
    }
    __syncthreads();
    ex0 = (wave > 0 ? wave_tot[wave - 1] : 0) + a - v0;
    ex1 = (wave > 0 ? wave_tot[nwaves + wave - 1] : 0) + b - v1;
    tot0 = wave_tot[nwaves - 1];
    tot1 = wave_tot[2 * nwaves - 1];
    __syncthreads();  // wave_tot is reused by the next scan
}

// Rank of this lane's expert e among the lower lanes holding e, and whether
// this lane is the highest lane holding e (ok: the lane holds a valid expert).
__device__ __forceinline__ void wave_match(int e, bool ok, int nbits, int &rank, bool &top, int &count)
{
    const int lane = lane_id();
    uint64_t peers = __ballot(ok);
    for (int b = 0; b < nbits; ++b) {
        const bool bit = ok && ((e >> b) & 1);
        const uint64_t m = __ballot(bit);
        peers &= bit ? m : ~m;
    }
    rank = __popcll(peers & ((1ull << lane) - 1ull));
    count = __popcll(peers);
    top = ok && lane == 63 - __clzll(peers);
}

}  // namespace ecospec
