// Internal declarations shared by the host API and the HIP kernels of libkvq.
// Nothing here is part of the public C ABI (include/kvq.h).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/kvq.h"

// Host handle behind the opaque kvq_cache.
struct kvq_cache {
    kvq_format fmt;
    int B, H, D, T_max, T_alloc;
    uint8_t* base;
    size_t bytes;
    size_t off[10], len[10];
    int n;
};

namespace kvq {

// Launch timing requested by kvq_time_launches on this host thread: while
// stop is set, every kernel the library launches records stop when it
// completes and the first one records start when it begins, from the
// kernel's own dispatch timestamps.
struct LaunchTiming {
    hipEvent_t start = nullptr, stop = nullptr;
};
LaunchTiming& launch_timing();

// Every kernel launch of the library (hipExtLaunchKernelGGL with the
// requested events, null when none are).
template <typename F, typename... Args>
inline void launch_kernel(F kernel, dim3 grid, dim3 block, size_t lds, hipStream_t stream, Args... args)
{
    LaunchTiming& t = launch_timing();
    hipExtLaunchKernelGGL(kernel, grid, block, (uint32_t)lds, stream, t.stop ? t.start : nullptr, t.stop, 0u, args...);
    if (t.stop)
        t.start = nullptr;
}

// Tail tokens (past the sink) at length n.
int num_tail(const kvq_format& f, int n);
// Tokens held as codes at length n: the tail count m, or floor(max(0, m -
// R)/F) * F with a window.
int num_coded(const kvq_format& f, int n);

// ---------------------------------------------------------------- append
struct AppendParams {
    uint32_t* kc;
    float* ks;
    float* kz;
    uint32_t* vc;
    float* vs;
    float* vz;
    uint16_t* kr;
    uint16_t* vr;
    const uint16_t* kin;  // bf16 [B][n_new][H][D]
    const uint16_t* vin;
    int B, H, T;          // T = T_alloc
    int n0, n_new;        // length before the call, tokens appended
    int q0, q1;           // coded-token range written by this call
    int ring;             // R + F (0 = no window)
    int ring_lo;          // first token written to the ring by this call
    int k_bits, v_bits, k_mode, v_mode, k_axis, k_group, v_group;
    int rotate;           // 0 or D
    float rot_c;          // binary32 value nearest D^(-1/2)
    int meta16;           // scales and offsets stored as fp16 (ks..vz then point at halves)
};
hipError_t launch_append(const AppendParams& p, int D, hipStream_t stream);
// fp16 rows [p.ring_lo, hi) of kr/vr with row stride p.ring and slot t mod
// p.ring, from input token t - p.n0 (the sink tokens: ring = sink).
hipError_t launch_append_rows(const AppendParams& p, int D, int hi, hipStream_t stream);

// ------------------------------------------------------------- projection
struct ProjParams {
    const uint16_t* x;    // bf16 [M][K]  (hidden states)
    const uint16_t* w;    // bf16 [N][K]  (weight rows)
    const uint16_t* bm;   // bf16 [N][rank] adapter up-projection rows (rank > 0)
    const float* t;       // rank > 0: fp32 [M][3 rank] scaled adapter activations (M > 32), or for
                          // M <= 32 the workspace of [ks][M][3 rank] unscaled partial sums over K slices
    const uint16_t* a;    // bf16 [3 rank][K] adapter down-projections (rank > 0, fused decode path)
    uint16_t* y0;         // bf16 outputs: columns [0, n1) -> y0, [n1, n2) -> y1, [n2, N) -> y2
    uint16_t* y1;
    uint16_t* y2;
    float* yf;            // fp32 output [M][N] (activation pass), else null
    int M, K, N;
    int n1, n2;           // column split points (d_q, d_q + d_kv)
    int rank;
    float scale;          // multiplies the fp32 output (activation pass); the adapter scale (fused path)
    int nxcd;             // XCDs the large-M tile order spreads over (set at launch)
    int tslices;          // K slices of the partial adapter activations (M <= 32, set at launch)
    int t_hilo;           // activations as bf16 hi and lo, [M][3][2 rank] (written by the activation pass
                          // through yf, read by the large-M pass as extra K stages; see project_adapter_stages)
    // Fused append (large-M path only): with fuse set, the K and V tiles are
    // coded into the cache instead of stored.  Rows are (sequence, token)
    // pairs, cn_new tokens per sequence starting at cache position cn0 (a
    // multiple of 32); per-token groups, no window, rotation or sink.
    int fuse;
    uint32_t* kc;
    float* ks;
    float* kz;
    uint32_t* vc;
    float* vs;
    float* vz;
    int cH, cD, cT, cn0, cn_new;  // KV heads, head size, T_alloc, first position, tokens per sequence
    int k_bits, v_bits, k_mode, v_mode, k_group, v_group, meta16;
    // Fused window append (decode path, M <= 32): with kr set, row m's K and
    // V go to slot rslot of sequence m's fp16 window ([B][cH][rslots][cD]
    // halves, the bf16-rounded values converted to fp16) instead of y1 / y2.
    uint16_t* kr;
    uint16_t* vr;
    int rslots, rslot;
};
hipError_t launch_project(const ProjParams& p, hipStream_t stream);
// The decode path (M <= 32) of launch_project.
hipError_t launch_project_decode(const ProjParams& p, hipStream_t stream);
// Whether the large-M pass of an M x d_in x (d_q + 2 d_kv) projection with
// adapter rank `rank` streams the adapter as extra K stages (its activation
// pass then writes t_hilo activations): 256x256 tiles that never straddle
// Q, K and V, and a rank that is a multiple of 16.
bool project_adapter_stages(int M, int d_in, int d_q, int d_kv, int rank);
// Upper bound on the K slices of the decode path's partial adapter activations.
constexpr int kProjTSlices = 16;
// Workspace bytes of the projection for M rows and adapter rank r.
inline size_t project_workspace_bytes(int M, int rank)
{
    return (size_t)(M <= 32 ? kProjTSlices : 1) * M * 3 * rank * sizeof(float);
}

// ---------------------------------------------------------------- merge
struct MergeParams {
    const uint16_t* w;    // bf16 [d_q + 2 d_kv][d_in] base weights
    const uint16_t* a;    // bf16 [3 rank][d_in] adapter down-projections
    const uint16_t* bm;   // bf16 [d_q + 2 d_kv][rank] adapter up-projections
    uint16_t* out;        // bf16 [d_q + 2 d_kv][d_in] merged weights (may equal w)
    int d_in, d_q, d_kv, rank;
    float scale;          // lora_scale
};
hipError_t launch_merge(const MergeParams& p, hipStream_t stream);

// ---------------------------------------------------------------- decode
struct AttnParams {
    const uint32_t* kc;
    const float* ks;
    const float* kz;
    const uint32_t* vc;
    const float* vs;
    const float* vz;
    const uint16_t* kr;
    const uint16_t* vr;
    const uint16_t* kq;   // fp16 sink rows [B][H][sink][D]
    const uint16_t* vq;
    const uint16_t* q;    // bf16 [B][H_q][D]
    float* part_o;        // fp32 [B*H_q][S_tot][D]  unnormalized partial outputs
    float* part_ml;       // fp32 [B*H_q][S_tot][2]  (running max in log2 units, sum)
    float* out;           // fp32 [B][H_q][D]
    int B, H, H_q, G, T;  // T = T_alloc
    int n, nq;            // tail tokens (past the sink; prefill: n - sink, negative inside the sink), coded tokens
    int ring;
    int sink, n_sink;     // sink rows per (b, h), and those holding tokens (min(length, sink))
    int S_q;              // splits over coded tokens (fp16 sink and window blocks are spread over them)
    int S_tot;            // splits in the grid (= S_q)
    int bps;              // 32-token blocks per split
    int k_bits, v_bits, k_mode, v_mode, k_axis, k_group, v_group;
    int rotate;
    float sm_log2;        // softmax scale * log2(e)
    float rot_c;
    size_t lds_bytes;     // dynamic LDS of the split kernel
    int C;                // chunked prefill: query tokens (the newest C of the cache); q is [B][C][H_q][D]
    int meta16;           // scales and offsets stored as fp16 (ks..vz then point at halves)
    // chunked prefill: workspace of block images [units of a group][pf_nvb][192 D bytes]
    uint8_t* pf_ws;
    int pf_u0;            // first unit (b H + h) of the group
    int pf_nvb;           // images per unit: pf_nsb sink blocks, then the tail blocks
    int pf_nsb;
    int pf_tiles;         // query tiles per unit
};
// Workgroups of the split kernel that fit the device at once (all fields of p
// that select the kernel instance and its LDS must be set).
int decode_target_groups(const AttnParams& p, int D);
// Waves per workgroup of the split kernel for head size D and format f.
int decode_waves(int D, const kvq_format& f);
// Split count (at least 1) and 32-token blocks per split (a multiple of
// `waves`) over nq coded tokens for a target number of workgroups.
void decode_plan(int B, int H, int waves, int groups, int nq, int* S_q, int* bps);
// Upper bound of S_q for any coded-token count and target.
int decode_split_bound(int B, int H);
// Dynamic LDS of the split kernel.
size_t decode_lds_bytes(int D, const kvq_format& f, int G);
hipError_t launch_decode(const AttnParams& p, int D, hipStream_t stream);
// Bytes of one reconstructed 32-token block (prefill workspace unit).
size_t prefill_image_bytes(int D);
// Chunked prefill over units in groups that fit ws_bytes (at least one unit).
hipError_t launch_prefill(const AttnParams& p, int D, size_t ws_bytes, hipStream_t stream);

}  // namespace kvq
