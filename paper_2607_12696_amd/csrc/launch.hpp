// Internal launchers of the gfx950 kernels; the C ABI in abi.cpp validates
// arguments and then calls these.  All enqueue on `stream` and return the
// hipError_t of the launch.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

namespace ecospec {

// slices == 0: logits [T][E]; slices > 0: router partial sums [slices][T][E]
// (summed in slice order, and stored to logits_out if it is not null).
hipError_t launch_route_topk(const float *logits, int slices, int T, int E, int k, int score, int32_t *idx, float *w,
                             float *logits_out, hipStream_t stream);

// Group-limited sigmoid routing with correction bias (may be null) and scaling.
hipError_t launch_route_grouped(const float *logits, const float *bias, int T, int E, int k, int G, int TG,
                                float scale, int32_t *idx, float *w, hipStream_t stream);

// Router K-slice partial sums of x [T][d] . W_router [E][d]^T -> [router_slices(d)][T][E] fp32.
int router_slices(int d);
hipError_t launch_router_gemm(const uint16_t *x, const uint16_t *w, int T, int d, int E, float *partial,
                              hipStream_t stream);

hipError_t launch_expert_union(const int32_t *idx, int T, int k, int E, int32_t *counts, int32_t *union_ids,
                               int32_t *n_unique, int32_t *offsets, int32_t *perm, hipStream_t stream);

struct VerifyArgs {
    int fmt, d, d_ff, E, T, k;
    const uint8_t *w_gate, *w_up, *w_down;  // routed experts, stacked [E]
    bool gu_pair, sh_gu_pair;               // W_gate and W_up packed as one pair in w_gate / sh_gate
    bool down_pair;                         // W_down (and sh_down) packed with row tiles 2p, 2p+1 interleaved
    const void *s_gate, *s_up, *s_down;
    const uint8_t *sh_gate, *sh_up, *sh_down;  // shared expert or null
    const void *sh_s_gate, *sh_s_up, *sh_s_down;
    const float *topk_w;
    const int32_t *topk_idx;
    int act;             // 0: SwiGLU, 1: GPT-OSS clamped SwiGLU
    float alpha, limit;
    const float *b_gate, *b_up, *b_down;  // routed experts' biases or null
    // The union and grouping of the slots (Eq. 1): written by the call itself (by the gate/up kernel, or by
    // the union kernel when T > 64), read by its later kernels.
    int32_t *counts, *union_ids, *n_unique, *offsets, *perm;
    const uint16_t *x;  // [T][d] bf16
    uint16_t *y;        // [T][d] bf16
    uint16_t *h;        // workspace: [T*k (+T)][d_ff] bf16 SwiGLU rows at grouped positions
    float *o;           // workspace: [T*k (+T)][d] fp32 expert outputs at grouped positions (shared: T*k + t)
    // workspace: [T*k + T][bands of the down launch] where the combine kernel reads each row of the down
    // launch's output (routed slot s at row s, the shared expert's row of token t at T*k + t): an output
    // descriptor of split.hpp, written by the down launch.
    uint64_t *desc;
    // MX activation mode (act_fmt 1, MXFP4 weights only): x and the SwiGLU rows
    // are the projections' inputs as OCP MX FP8 (one e8m0 code per 32
    // consecutive elements), rows padded to the next multiple of 128 elements
    // and each 128-element chunk stored in the FP8 operand's lane order (lane
    // group g: elements 16g..16g+15, then 64+16g..64+16g+15).
    int act_fmt;
    uint8_t *xq, *xs;  // workspace: [T][Kp(d)] e4m3fn codes, [T][Kp(d)/32] e8m0 codes
    uint8_t *hq, *hs;  // workspace: [T*k (+T)][Kp(d_ff)], [T*k (+T)][Kp(d_ff)/32]
};

// Upper bound on the workgroups of a verify grid (sizes the partial-sum slots).
constexpr int kMaxWorkers = 512;
constexpr int kMaxGroups = 4096;  // token groups of one launch (one per expert and 64 of its tokens)
constexpr int kTimingMarks = 5;  // events recorded by the timed entry point

// Workspace layout shared by the size query and the launcher: H (bf16 SwiGLU
// rows) and O (fp32 expert outputs), both at grouped positions; partial sums
// and unit ranges of work items cut between workgroups; the token-group plan;
// the down launch's output descriptors for the combine kernel.
struct VerifyWorkspace {
    size_t h_offset, h_bytes, o_offset, o_bytes, p_offset, p_bytes, plan_offset, plan_bytes, desc_offset, desc_bytes,
        mx_offset, mx_bytes;
    int plan_cap;
    int workers;      // workgroups of the expert kernels' grid (one per compute unit)
    int slot_floats;  // floats per partial-sum slot (two slots per workgroup)
    size_t total;
};
// Workgroups of the expert kernels' grid on the current device.
int verify_workers();
// mx: room for the MX activation mode's quantised x and SwiGLU rows; workers:
// the grid the call will launch (the partial-sum slots are sized by it).
VerifyWorkspace verify_workspace(int d, int d_ff, int T, int k, bool shared, bool mx, int workers);

// events: kTimingMarks optional marks (before gate/up, before its fix-up, before
// down, before combine, after combine).
hipError_t launch_verify(const VerifyArgs &a, void *workspace, const VerifyWorkspace &ws, hipStream_t stream,
                         hipEvent_t const *events = nullptr);

// Packed (streaming) weight layout; see pack.hip.
size_t packed_matrix_bytes(int fmt, int N, int K);
size_t packed_scale_bytes(int fmt, int N, int K);
hipError_t launch_pack_gate_up(int fmt, int E, int N, int K, const void *wg, const void *sg, const void *wu,
                               const void *su, void *wp, void *sgp, void *sup, hipStream_t stream);
hipError_t launch_pack(int fmt, int E, int N, int K, const void *w, const void *s, void *wp, void *sp,
                       hipStream_t stream);
hipError_t launch_pack_down(int fmt, int E, int N, int K, const void *w, const void *s, void *wp, void *sp,
                            hipStream_t stream);

}  // namespace ecospec
