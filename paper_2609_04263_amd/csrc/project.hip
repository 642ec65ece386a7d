// Adapted Q/K/V projection (Sec. 3, Eq. (1)-(2); explicit adapter branch of
// Sec. 3.4):  y_p = W_p h + (alpha/r) B_p (A_p h)  for p in {Q, K, V}.
//
// Two passes, both on bf16 MFMA (v_mfma_f32_16x16x32_bf16, fp32 accumulate):
//   1. activation pass: t = (alpha/r) H A^T, fp32 [M][3r], into the workspace;
//   2. main pass: Y = H W^T, with the adapter branch fused as a K-extension
//      of the same accumulators: t_p (split into bf16 hi + lo parts) times
//      B_p^T, then one rounding to bf16 and routing of the columns to Q/K/V.
//
// M <= 32 (decode: one token per sequence) streams the weights from HBM with
// a skinny kernel: a workgroup owns 16 weight rows and its four waves split
// the reduction dimension, keeping many 16-byte loads in flight.  Larger M
// (prefill) uses a 128x128 tiled GEMM staged through LDS.

#include "kvq_device.h"
#include "kvq_internal.h"

namespace kvq {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ bf16x8 load_bf16x8(const uint16_t* p)
{
    return __builtin_bit_cast(bf16x8, *(const u32x4*)p);
}

__device__ __forceinline__ bf16x8 zero_bf16x8()
{
    return __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
}

// Eight fp32 values -> bf16 hi part (nearest) and lo part (remainder, nearest).
__device__ __forceinline__ void split_bf16x8(const float* v, bf16x8* hi, bf16x8* lo)
{
    uint16_t h[8], l[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        h[e] = f32_to_bf16(v[e]);
        l[e] = f32_to_bf16(v[e] - bf16_to_f32(h[e]));
    }
    u32x4 a, b;
    a.x = h[0] | ((uint32_t)h[1] << 16);
    a.y = h[2] | ((uint32_t)h[3] << 16);
    a.z = h[4] | ((uint32_t)h[5] << 16);
    a.w = h[6] | ((uint32_t)h[7] << 16);
    b.x = l[0] | ((uint32_t)l[1] << 16);
    b.y = l[2] | ((uint32_t)l[3] << 16);
    b.z = l[4] | ((uint32_t)l[5] << 16);
    b.w = l[6] | ((uint32_t)l[7] << 16);
    *hi = __builtin_bit_cast(bf16x8, a);
    *lo = __builtin_bit_cast(bf16x8, b);
}

__device__ __forceinline__ int proj_of(const ProjParams& p, int n)
{
    return n < p.n1 ? 0 : (n < p.n2 ? 1 : 2);
}

__device__ __forceinline__ void store_out(const ProjParams& p, int m, int n, float v)
{
    if (m >= p.M || n >= p.N)
        return;
    if (p.yf) {
        p.yf[(size_t)m * p.N + n] = v * p.scale;
        return;
    }
    uint16_t o = f32_to_bf16(v);
    if (n < p.n1)
        p.y0[(size_t)m * p.n1 + n] = o;
    else if (n < p.n2)
        p.y1[(size_t)m * (p.n2 - p.n1) + (n - p.n1)] = o;
    else
        p.y2[(size_t)m * (p.N - p.n2) + (n - p.n2)] = o;
}

// Adapter operands for one 32-wide chunk kk of the rank dimension:
//   rows side: token m's activations t[m][p r + k] (fp32 -> bf16 hi/lo),
//   cols side: weight row n's up-projection B[n][k], zero unless n is in p.
__device__ __forceinline__ void lora_token_operand(const ProjParams& p, int m, int proj, int kk, int qg,
                                                   bf16x8* hi, bf16x8* lo)
{
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        int k = 32 * kk + 8 * qg + e;
        v[e] = (m < p.M && k < p.rank) ? p.t[(size_t)m * 3 * p.rank + proj * p.rank + k] : 0.0f;
    }
    split_bf16x8(v, hi, lo);
}

__device__ __forceinline__ bf16x8 lora_weight_operand(const ProjParams& p, int n, int proj, int kk, int qg)
{
    uint16_t v[8];
    const bool ok = n < p.N && proj_of(p, n) == proj;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        int k = 32 * kk + 8 * qg + e;
        v[e] = (ok && k < p.rank) ? p.bm[(size_t)n * p.rank + k] : (uint16_t)0;
    }
    u32x4 a;
    a.x = v[0] | ((uint32_t)v[1] << 16);
    a.y = v[2] | ((uint32_t)v[3] << 16);
    a.z = v[4] | ((uint32_t)v[5] << 16);
    a.w = v[6] | ((uint32_t)v[7] << 16);
    return __builtin_bit_cast(bf16x8, a);
}

// ------------------------------------------------------------------ skinny
// Workgroup: weight rows [n0, n0 + 16) x all M (<= 32) tokens.
// MFMA roles: A = W rows (M-dim = 16 weight rows), B = H^T (N-dim = 16 tokens).
// Output lane layout: token = 16 nt + (lane % 16), row n0 + 4 qg + i.
constexpr int kSkinnyUnroll = 8;

__global__ __launch_bounds__(kThreads) void proj_skinny_kernel(ProjParams p)
{
    __shared__ floatx4 red[4][2][64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r = lane & 15, qg = lane >> 4;
    const int n0 = blockIdx.x * 16;
    const int nt_count = p.M > 16 ? 2 : 1;
    const int steps = p.K / 32;
    const int per = (steps + 3) / 4;
    const int s_begin = wave * per, s_end = min(steps, s_begin + per);

    const int wrow = n0 + r;
    const uint16_t* wp = p.w + (size_t)min(wrow, p.N - 1) * p.K + 8 * qg;
    const bool wok = wrow < p.N;
    const uint16_t* xp0 = p.x + (size_t)min(r, p.M - 1) * p.K + 8 * qg;
    const uint16_t* xp1 = p.x + (size_t)min(16 + r, p.M - 1) * p.K + 8 * qg;
    const bool x0ok = r < p.M, x1ok = 16 + r < p.M;

    floatx4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
    for (int s = s_begin; s < s_end; s += kSkinnyUnroll) {
        bf16x8 a[kSkinnyUnroll], b0[kSkinnyUnroll], b1[kSkinnyUnroll];
#pragma unroll
        for (int u = 0; u < kSkinnyUnroll; ++u) {
            int ss = s + u;
            bool in = ss < s_end;
            a[u] = (in && wok) ? load_bf16x8(wp + 32 * ss) : zero_bf16x8();
            b0[u] = (in && x0ok) ? load_bf16x8(xp0 + 32 * ss) : zero_bf16x8();
            b1[u] = (in && x1ok && nt_count > 1) ? load_bf16x8(xp1 + 32 * ss) : zero_bf16x8();
        }
#pragma unroll
        for (int u = 0; u < kSkinnyUnroll; ++u) {
            acc0 = mfma16_bf16(a[u], b0[u], acc0);
            if (nt_count > 1)
                acc1 = mfma16_bf16(a[u], b1[u], acc1);
        }
    }
    red[wave][0][lane] = acc0;
    red[wave][1][lane] = acc1;
    __syncthreads();
    if (wave != 0)
        return;
    acc0 = red[0][0][lane] + red[1][0][lane] + red[2][0][lane] + red[3][0][lane];
    acc1 = red[0][1][lane] + red[1][1][lane] + red[2][1][lane] + red[3][1][lane];

    if (p.rank > 0) {
        // Tiles never straddle projections (d_q, d_kv are multiples of 16).
        const int proj = proj_of(p, n0);
        const int nk = (p.rank + 31) / 32;
        for (int kk = 0; kk < nk; ++kk) {
            bf16x8 wa = lora_weight_operand(p, wrow, proj, kk, qg);
            bf16x8 hi, lo;
            lora_token_operand(p, r, proj, kk, qg, &hi, &lo);
            acc0 = mfma16_bf16(wa, hi, acc0);
            acc0 = mfma16_bf16(wa, lo, acc0);
            if (nt_count > 1) {
                lora_token_operand(p, 16 + r, proj, kk, qg, &hi, &lo);
                acc1 = mfma16_bf16(wa, hi, acc1);
                acc1 = mfma16_bf16(wa, lo, acc1);
            }
        }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        store_out(p, r, n0 + 4 * qg + i, acc0[i]);
        if (nt_count > 1)
            store_out(p, 16 + r, n0 + 4 * qg + i, acc1[i]);
    }
}

// --------------------------------------------------------------------- big
// 128x128 output tile, four waves in a 2x2 grid of 64x64 sub-tiles, K step
// 64 through double-buffered LDS (rows padded by 16 bytes).
// MFMA roles: A = H rows (M-dim = tokens), B = W^T (N-dim = weight rows).
// Output lane layout: token m = row base + 4 qg + i, column n = base + lane % 16.
constexpr int kBM = 128, kBN = 128, kBK = 64, kLdsRow = kBK + 8;

__global__ __launch_bounds__(kThreads) void proj_big_kernel(ProjParams p)
{
    __shared__ uint16_t As[2][kBM * kLdsRow];
    __shared__ uint16_t Bs[2][kBN * kLdsRow];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int r = lane & 15, qg = lane >> 4;
    const int wm = wave >> 1, wn = wave & 1;
    const int m0 = blockIdx.y * kBM, n0 = blockIdx.x * kBN;

    // Global -> register staging: 4 x 16 bytes per thread per operand.
    u32x4 ra[4], rb[4];
    auto gload = [&](int k0) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            int idx = tid + kThreads * i;      // 0..1023
            int row = idx >> 3, c8 = (idx & 7) * 8;
            int m = m0 + row, n = n0 + row;
            ra[i] = m < p.M ? *(const u32x4*)(p.x + (size_t)m * p.K + k0 + c8) : u32x4{0u, 0u, 0u, 0u};
            rb[i] = n < p.N ? *(const u32x4*)(p.w + (size_t)n * p.K + k0 + c8) : u32x4{0u, 0u, 0u, 0u};
        }
    };
    auto lstore = [&](int buf) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            int idx = tid + kThreads * i;
            int row = idx >> 3, c8 = (idx & 7) * 8;
            *(u32x4*)(&As[buf][row * kLdsRow + c8]) = ra[i];
            *(u32x4*)(&Bs[buf][row * kLdsRow + c8]) = rb[i];
        }
    };

    floatx4 acc[4][4];
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
        for (int ni = 0; ni < 4; ++ni)
            acc[mi][ni] = floatx4{0.f, 0.f, 0.f, 0.f};

    const int ksteps = p.K / kBK;
    gload(0);
    lstore(0);
    __syncthreads();
    for (int ks = 0; ks < ksteps; ++ks) {
        const int buf = ks & 1;
        if (ks + 1 < ksteps)
            gload((ks + 1) * kBK);
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            bf16x8 af[4], bfr[4];
#pragma unroll
            for (int mi = 0; mi < 4; ++mi)
                af[mi] = __builtin_bit_cast(
                    bf16x8, *(const u32x4*)(&As[buf][(wm * 64 + 16 * mi + r) * kLdsRow + 32 * kk + 8 * qg]));
#pragma unroll
            for (int ni = 0; ni < 4; ++ni)
                bfr[ni] = __builtin_bit_cast(
                    bf16x8, *(const u32x4*)(&Bs[buf][(wn * 64 + 16 * ni + r) * kLdsRow + 32 * kk + 8 * qg]));
#pragma unroll
            for (int mi = 0; mi < 4; ++mi)
#pragma unroll
                for (int ni = 0; ni < 4; ++ni)
                    acc[mi][ni] = mfma16_bf16(af[mi], bfr[ni], acc[mi][ni]);
        }
        if (ks + 1 < ksteps) {
            lstore(buf ^ 1);
            __syncthreads();
        }
    }

    if (p.rank > 0) {
        const int nk = (p.rank + 31) / 32;
        const int p_lo = proj_of(p, n0), p_hi = proj_of(p, min(n0 + kBN, p.N) - 1);
        for (int proj = p_lo; proj <= p_hi; ++proj) {
            for (int kk = 0; kk < nk; ++kk) {
                bf16x8 wop[4];
#pragma unroll
                for (int ni = 0; ni < 4; ++ni)
                    wop[ni] = lora_weight_operand(p, n0 + wn * 64 + 16 * ni + r, proj, kk, qg);
#pragma unroll
                for (int mi = 0; mi < 4; ++mi) {
                    bf16x8 hi, lo;
                    lora_token_operand(p, m0 + wm * 64 + 16 * mi + r, proj, kk, qg, &hi, &lo);
#pragma unroll
                    for (int ni = 0; ni < 4; ++ni) {
                        acc[mi][ni] = mfma16_bf16(hi, wop[ni], acc[mi][ni]);
                        acc[mi][ni] = mfma16_bf16(lo, wop[ni], acc[mi][ni]);
                    }
                }
            }
        }
    }
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
        for (int ni = 0; ni < 4; ++ni)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                store_out(p, m0 + wm * 64 + 16 * mi + 4 * qg + i, n0 + wn * 64 + 16 * ni + r, acc[mi][ni][i]);
}

}  // namespace

hipError_t launch_project(const ProjParams& p, hipStream_t stream)
{
    if (p.M <= 0)
        return hipSuccess;
    if (p.M <= 32) {
        hipLaunchKernelGGL(proj_skinny_kernel, dim3((p.N + 15) / 16), dim3(kThreads), 0, stream, p);
    } else {
        dim3 grid((p.N + kBN - 1) / kBN, (p.M + kBM - 1) / kBM);
        hipLaunchKernelGGL(proj_big_kernel, grid, dim3(kThreads), 0, stream, p);
    }
    return hipGetLastError();
}

}  // namespace kvq
