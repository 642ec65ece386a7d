// Dense-merge deployment of the adapter (Sec. 3.4 "Deployment overhead"):
// the dense-base update folded into the base weights,
//     W'[n][i] = W[n][i] + lora_scale * sum_k B[n][k] A_p[k][i],
// p the projection of row n, so that the plain projection with W' equals the
// explicit-adapter one and the adapter branch disappears at inference.
//
// HBM-bound (read W, write W'); the update B_p A_p is a rank-r contraction,
// done on the matrix cores: v_mfma_f32_32x32x16_bf16 with B's rows as the A
// operand and A_p's columns as the B operand (bf16 x bf16 products are exact
// in fp32), the rank padded to a multiple of 16 with zeros.
//
// Workgroup: 128 rows x 128 input channels, four waves of 32 rows each (a
// 32-row block never straddles projections: d_q and d_kv are multiples of
// 32).  A_p's 128 columns of every projection the tile touches are staged in
// LDS transposed ([channel][k], rows padded by 16 bytes), so that a lane's
// eight consecutive k of one channel are one 16-byte read.  The accumulators
// go through LDS once more to be combined with W in 16-byte pieces.

#include "kvq_internal.h"
#include "kvq_device.h"

namespace kvq {
namespace {

constexpr int kMT = 128;       // rows (output features) per workgroup
constexpr int kMC = 128;       // input channels per workgroup
constexpr int kMaxRank = 64;

typedef float floatx16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ int proj_row(const MergeParams& p, int n)
{
    return n < p.d_q ? 0 : (n < p.d_q + p.d_kv ? 1 : 2);
}

__global__ __launch_bounds__(256) void merge_kernel(MergeParams p)
{
    extern __shared__ __attribute__((aligned(16))) uint16_t mlds[];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int N = p.d_q + 2 * p.d_kv;
    const int c0 = blockIdx.x * kMC, n0 = blockIdx.y * kMT;
    const int RP = (p.rank + 15) & ~15;  // rank padded to the MFMA depth
    const int pitch = RP + 8;            // LDS row of one channel, bf16 units
    const int p_lo = proj_row(p, n0), p_hi = proj_row(p, min(n0 + kMT, N) - 1);

    // This lane's W pieces (rows nw + lane / 16 + 4 j, eight channels from
    // c0 + 8 (lane % 16)) are loaded first, so that their HBM latency
    // overlaps the staging and the MFMAs.
    const int nw = n0 + 32 * wave;  // this wave's 32 rows
    const int c8 = 8 * (lane & 15);
    const int c = c0 + c8;
    u32x4 wv[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int n = nw + (lane >> 4) + 4 * j;
        wv[j] = (n < N && c < p.d_in) ? *(const u32x4*)(p.w + (size_t)n * p.d_in + c) : u32x4{0u, 0u, 0u, 0u};
    }

    // stage A_p[0..RP)[c0..c0+128) transposed for the projections of this tile
    for (int pp = p_lo; pp <= p_hi; ++pp) {
        uint16_t* at = mlds + (pp - p_lo) * kMC * pitch;
        for (int idx = threadIdx.x; idx < RP * (kMC / 8); idx += 256) {
            const int k = idx / (kMC / 8), c8 = 8 * (idx % (kMC / 8));
            u32x4 v = {0u, 0u, 0u, 0u};
            if (k < p.rank && c0 + c8 < p.d_in)
                v = *(const u32x4*)(p.a + ((size_t)pp * p.rank + k) * p.d_in + c0 + c8);
            const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int e = 0; e < 8; ++e)
                at[(c8 + e) * pitch + k] = (uint16_t)(w[e >> 1] >> (16 * (e & 1)));
        }
    }
    __syncthreads();

    const bool live = nw < N;
    floatx16 acc[kMC / 32];
#pragma unroll
    for (int j = 0; j < kMC / 32; ++j)
        acc[j] = floatx16{};
    if (live) {
        const int pw = proj_row(p, nw);
        const uint16_t* at = mlds + (pw - p_lo) * kMC * pitch;
        const int fr = lane & 31, fk = lane >> 5;
        const bool vec = (p.rank & 7) == 0;
        for (int kc = 0; kc < RP; kc += 16) {
            // A operand: row nw + fr of B, k = kc + 8 fk .. + 7
            const int k0 = kc + 8 * fk;
            u32x4 bo = {0u, 0u, 0u, 0u};
            const uint16_t* brow = p.bm + (size_t)(nw + fr) * p.rank;
            if (vec) {
                if (k0 < p.rank)
                    bo = *(const u32x4*)(brow + k0);
            } else {
                uint16_t e8[8];
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    e8[e] = k0 + e < p.rank ? brow[k0 + e] : (uint16_t)0;
                bo.x = e8[0] | ((uint32_t)e8[1] << 16);
                bo.y = e8[2] | ((uint32_t)e8[3] << 16);
                bo.z = e8[4] | ((uint32_t)e8[5] << 16);
                bo.w = e8[6] | ((uint32_t)e8[7] << 16);
            }
            const bf16x8 av = __builtin_bit_cast(bf16x8, bo);
#pragma unroll
            for (int j = 0; j < kMC / 32; ++j) {
                // B operand: channel c0 + 32 j + fr, the same eight k
                const bf16x8 bv = __builtin_bit_cast(bf16x8, *(const u32x4*)(at + (32 * j + fr) * pitch + k0));
                acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bv, acc[j], 0, 0, 0);
            }
        }
    }
    __syncthreads();  // the staged A_p is no longer read

    // accumulator element e of lane l: row 8 (e / 4) + 4 (l / 32) + e % 4,
    // channel l % 32 of its 32x32 block -> fp32 rows of 128 channels in LDS
    float* xo = (float*)mlds + wave * (32 * kMC);
    if (live) {
#pragma unroll
        for (int j = 0; j < kMC / 32; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e)
                xo[(8 * (e >> 2) + 4 * (lane >> 5) + (e & 3)) * kMC + 32 * j + (lane & 31)] = acc[j][e];
    }
    __syncthreads();
    if (!live)
        return;
    // 16 lanes per row, eight channels each; four rows per pass
    if (c >= p.d_in)
        return;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int r = (lane >> 4) + 4 * j;
        const int n = nw + r;
        if (n >= N)
            break;
        const float* u = xo + r * kMC + c8;
        const uint32_t win[4] = {wv[j].x, wv[j].y, wv[j].z, wv[j].w};
        uint32_t wout[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float lo = __uint_as_float(win[q] << 16) + p.scale * u[2 * q];
            const float hi = __uint_as_float(win[q] & 0xFFFF0000u) + p.scale * u[2 * q + 1];
            wout[q] = (uint32_t)f32_to_bf16(lo) | ((uint32_t)f32_to_bf16(hi) << 16);
        }
        *(u32x4*)(p.out + (size_t)n * p.d_in + c) = u32x4{wout[0], wout[1], wout[2], wout[3]};
    }
}

}  // namespace

size_t merge_lds_bytes(const MergeParams& p)
{
    const int RP = (p.rank + 15) & ~15;
    const int nproj = 3;  // upper bound on the projections one tile touches
    const size_t stage = (size_t)nproj * kMC * (RP + 8) * sizeof(uint16_t);
    const size_t epi = (size_t)4 * 32 * kMC * sizeof(float);
    return stage > epi ? stage : epi;
}

hipError_t launch_merge(const MergeParams& p, hipStream_t stream)
{
    const int N = p.d_q + 2 * p.d_kv;
    if (p.rank < 1 || p.rank > kMaxRank)
        return hipErrorInvalidValue;
    dim3 grid((p.d_in + kMC - 1) / kMC, (N + kMT - 1) / kMT);
    launch_kernel(merge_kernel, grid, dim3(256), merge_lds_bytes(p), stream, p);
    return hipGetLastError();
}

}  // namespace kvq
