// Conversion of expert weights from the interchange layout ([E][N][K], K
// contiguous) to the streaming layout the verify kernels read.
//
// Streaming layout of one N x K matrix (N % 16 == 0; K padded to Kp, the next
// multiple of 128, with zero codes): blocks of 16 rows x 128 reduction
// elements, block (rb, kb) at byte offset (rb * Kp/128 + kb) * B where B is
// 4096 (bf16), 2048 (FP8) or 1024 (MXFP4) bytes.  A block is B/1024 vectors
// of 1 KiB; in vector i, the 16 bytes at offset 16*l (l = c + 16*g, c < 16,
// g < 4) hold the weights of row rb*16 + c starting at element
// kb*128 + 32*g + i*(32*1024/B).  So lane l of a wavefront reading vector i
// with one 16-byte load gets exactly the A-operand fragment of the matrix-core
// instruction, and a wavefront reads each vector as 1 KiB of contiguous memory.
//
// W_gate and W_up can also be packed as one pair (moe_pack_gate_up): block
// (rb, kb) of the pair is the gate block followed by the up block, so a
// wavefront reads both tiles of a step as one contiguous run (one stream
// instead of two, measured 4% more bandwidth in the kernel's geometry).
// W_down likewise (moe_pack_down): row tiles 2p and 2p + 1 (the two tiles of
// one down wavefront) are interleaved block by block, block (2p + j, kb) at
// ((p * Kp/128 + kb) * 2 + j) * B.
//
// MXFP4 scales move to the same blocking, four blocks to a 256-byte quad: in
// quad q of row tile rb, the 4 bytes at offset 4*l (l = c + 16*g) are the
// e8m0 codes of row rb*16 + c for the 32-element chunks (4q + j)*4 + g,
// j = 0..3 (127, i.e. 1.0, in the padding), so one dword load per lane
// brings a lane's codes for four blocks.  FP8 block scales keep their
// [N/128][K/128] layout.
#include "device.hpp"
#include "launch.hpp"

namespace ecospec {

// One thread writes one 16-byte lane vector of the packed matrix.  pair = 2
// packs W_gate and W_up together: block (rb, kb) of the pair holds the gate
// block and then the up block (`which` = 0 / 1), so the verify kernel reads
// both tiles of a step as one contiguous run.  tile_pairs = 1 interleaves row
// tiles 2p and 2p + 1 of one matrix the same way (pair = 1).
__global__ __launch_bounds__(256) void pack_weights_kernel(const uint8_t *__restrict__ src, uint8_t *__restrict__ dst,
                                                           int E, int N, int K, int num, int den, int vecs, int pair,
                                                           int which, int tile_pairs)
{
    const int nkb = (K + 127) / 128;
    const size_t per_block = (size_t)vecs * 64;  // lane vectors per block
    const size_t total = (size_t)E * (N / 16) * nkb * per_block;
    const size_t src_row = (size_t)K * num / den, src_mat = (size_t)N * src_row;
    const size_t dst_mat = (size_t)(N / 16) * nkb * per_block * 16 * pair;
    for (size_t q = blockIdx.x * (size_t)blockDim.x + threadIdx.x; q < total; q += (size_t)gridDim.x * blockDim.x) {
        const size_t e = q / ((size_t)(N / 16) * nkb * per_block);
        size_t r = q - e * ((size_t)(N / 16) * nkb * per_block);
        const int rb = (int)(r / ((size_t)nkb * per_block));
        r -= (size_t)rb * nkb * per_block;
        const int kb = (int)(r / per_block);
        r -= (size_t)kb * per_block;
        const int i = (int)(r / 64), l = (int)(r % 64);
        const int c = l & 15, g = l >> 4;
        const int k0 = kb * 128 + 32 * g + i * (32 / vecs);  // first element of this 16-byte vector
        u32x4 v = u32x4{0u, 0u, 0u, 0u};
        if (k0 < K) {
            const uint8_t *p = src + e * src_mat + (size_t)(rb * 16 + c) * src_row + (size_t)k0 * num / den;
            v = *reinterpret_cast<const u32x4 *>(p);
        }
        const size_t blk = tile_pairs ? ((size_t)(rb >> 1) * nkb + kb) * 2 + (rb & 1)
                                      : ((size_t)rb * nkb + kb) * pair + which;
        uint8_t *o = dst + e * dst_mat + blk * ((size_t)vecs * 1024) + (size_t)i * 1024 + (size_t)l * 16;
        *reinterpret_cast<u32x4 *>(o) = v;
    }
}

// MXFP4 scales: [E][N][K/32] -> [E][N/16][ceil(Kp/512)][64][4], one byte per thread.
__global__ __launch_bounds__(256) void pack_mx_scales_kernel(const uint8_t *__restrict__ src, uint8_t *__restrict__ dst,
                                                             int E, int N, int K)
{
    const int nq = ((K + 127) / 128 + 3) / 4;
    const size_t per_e = (size_t)(N / 16) * nq * 256;
    const size_t total = (size_t)E * per_e;
    for (size_t q = blockIdx.x * (size_t)blockDim.x + threadIdx.x; q < total; q += (size_t)gridDim.x * blockDim.x) {
        const size_t e = q / per_e;
        size_t r = q - e * per_e;
        const int rb = (int)(r / ((size_t)nq * 256));
        r -= (size_t)rb * nq * 256;
        const int qd = (int)(r / 256), l = (int)(r % 256) / 4, j = (int)(r % 4);
        const int c = l & 15, g = l >> 4;
        const int chunk = (qd * 4 + j) * 4 + g;
        dst[q] = chunk < K / 32 ? src[e * (size_t)N * (K / 32) + (size_t)(rb * 16 + c) * (K / 32) + chunk] : 127;
    }
}

size_t packed_matrix_bytes(int fmt, int N, int K)
{
    const size_t kp = (size_t)((K + 127) / 128) * 128;
    return fmt == 0 ? (size_t)N * kp * 2 : fmt == 1 ? (size_t)N * kp : (size_t)N * kp / 2;
}

size_t packed_scale_bytes(int fmt, int N, int K)
{
    if (fmt == 1) return (size_t)(N / 128) * (K / 128) * 4;
    if (fmt == 2) return (size_t)N * (((K + 127) / 128 + 3) / 4) * 16;
    return 0;
}

static hipError_t pack_matrix(int fmt, int E, int N, int K, const void *w, void *wp, int pair, int which,
                              hipStream_t stream, int tile_pairs = 0)
{
    const int num = fmt == 0 ? 2 : 1, den = fmt == 2 ? 2 : 1, vecs = fmt == 0 ? 4 : fmt == 1 ? 2 : 1;
    const size_t vec_total = (size_t)E * (N / 16) * ((K + 127) / 128) * vecs * 64;
    const int grid = (int)((vec_total + 255) / 256 < 65536 ? (vec_total + 255) / 256 : 65536);
    hipLaunchKernelGGL(pack_weights_kernel, dim3(grid), dim3(256), 0, stream, static_cast<const uint8_t *>(w),
                       static_cast<uint8_t *>(wp), E, N, K, num, den, vecs, pair, which, tile_pairs);
    return hipGetLastError();
}

static hipError_t pack_scales(int fmt, int E, int N, int K, const void *s, void *sp, hipStream_t stream)
{
    if (fmt == 1)
        return hipMemcpyAsync(sp, s, (size_t)E * packed_scale_bytes(1, N, K), hipMemcpyDeviceToDevice, stream);
    if (fmt == 2) {
        const size_t total = (size_t)E * packed_scale_bytes(2, N, K);
        const int g2 = (int)((total + 255) / 256 < 65536 ? (total + 255) / 256 : 65536);
        hipLaunchKernelGGL(pack_mx_scales_kernel, dim3(g2), dim3(256), 0, stream, static_cast<const uint8_t *>(s),
                           static_cast<uint8_t *>(sp), E, N, K);
        return hipGetLastError();
    }
    return hipSuccess;
}

hipError_t launch_pack(int fmt, int E, int N, int K, const void *w, const void *s, void *wp, void *sp,
                       hipStream_t stream)
{
    hipError_t err = pack_matrix(fmt, E, N, K, w, wp, 1, 0, stream);
    if (err != hipSuccess) return err;
    return pack_scales(fmt, E, N, K, s, sp, stream);
}

hipError_t launch_pack_down(int fmt, int E, int N, int K, const void *w, const void *s, void *wp, void *sp,
                            hipStream_t stream)
{
    hipError_t err = pack_matrix(fmt, E, N, K, w, wp, 1, 0, stream, 1);
    if (err == hipSuccess) err = pack_scales(fmt, E, N, K, s, sp, stream);
    return err;
}

hipError_t launch_pack_gate_up(int fmt, int E, int N, int K, const void *wg, const void *sg, const void *wu,
                               const void *su, void *wp, void *sgp, void *sup, hipStream_t stream)
{
    hipError_t err = pack_matrix(fmt, E, N, K, wg, wp, 2, 0, stream);
    if (err == hipSuccess) err = pack_matrix(fmt, E, N, K, wu, wp, 2, 1, stream);
    if (err == hipSuccess) err = pack_scales(fmt, E, N, K, sg, sgp, stream);
    if (err == hipSuccess) err = pack_scales(fmt, E, N, K, su, sup, stream);
    return err;
}

}  // namespace ecospec
