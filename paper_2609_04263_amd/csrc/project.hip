// Adapted Q/K/V projection (Sec. 3, Eq. (1)-(2); explicit adapter branch of
// Sec. 3.4):  y_p = W_p h + (alpha/r) B_p (A_p h)  for p in {Q, K, V}.
//
// Two passes, both on bf16 MFMA (v_mfma_f32_16x16x32_bf16, fp32 accumulate):
//   1. activation pass: t = (alpha/r) H A^T, fp32 [M][3r], into the workspace;
//   2. main pass: Y = H W^T, with the adapter branch fused as a K-extension
//      of the same accumulators: t_p (split into bf16 hi + lo parts) times
//      B_p^T, then one rounding to bf16 and routing of the columns to Q/K/V.
//
// M <= 32 (decode: one token per sequence) runs as one fused kernel that
// streams the weights from HBM: a workgroup owns 16 weight rows and its
// eight waves split the reduction dimension, each issuing its 16-byte loads
// of W, H and the adapter rows A_p in one batch.  The same H fragments feed
// both Y = H W^T and the adapter activations t = H A_p^T (its own copy per
// workgroup: the adapter rows are small and stay in L2), which are reduced
// across waves in LDS and applied as the K-extension.  Larger M (prefill)
// uses the two passes with a 128x128 tiled GEMM staged through LDS.

#include <atomic>

#include "coder.h"
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
    const bool ok = n < p.N && proj_of(p, n) == proj;
    const int k0 = 32 * kk + 8 * qg;
    if ((p.rank & 7) == 0 && ((uintptr_t)p.bm & 15) == 0)  // eight whole elements or none, 16-byte aligned
        return (ok && k0 < p.rank) ? load_bf16x8(p.bm + (size_t)n * p.rank + k0) : zero_bf16x8();
    uint16_t v[8];
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

// ----------------------------------------------------------- fused decode
// Workgroup: weight rows [n0, n0 + 16 R) x all M (<= 16 MT) tokens, 8 waves.
// Each wave owns one eighth of the reduction dimension for all R row tiles,
// so one H fragment (and one adapter fragment) serves R weight tiles: the
// rows of H and A_p, which every workgroup reads, cost 1/R of the weight
// traffic instead of as much as it.  Workgroups start their waves at
// different eighths so that concurrent workgroups read different lines.
// MFMA roles: Y: A = W rows (16 weight rows), B = H^T (16 tokens);
//             t: A = H rows (16 tokens), B = A_p^T (16 adapter rows).
// Output lane layout: token = 16 mt + (lane % 16), row n0 + 16 rt + 4 qg + i.
constexpr int kDecWaves = 8;

template <int R, int MT, int NKT, bool TLOAD>
struct DecShape {
    static constexpr int NV = R * MT + MT * NKT;       // floatx4 partials per lane
    static constexpr int NKK = (16 * NKT + 31) / 32;   // 32-wide rank chunks of the fused K-extension
    static constexpr int PER_STEP = R + MT + NKT;      // 16-byte loads per K-step
    static constexpr int U = PER_STEP <= 3 ? 8 : PER_STEP <= 6 ? 4 : 2;  // K-steps per load batch
    static constexpr size_t LDS = sizeof(floatx4) * kDecWaves * NV * 64 + sizeof(float) * 16 * MT * 16 * NKT;
};

template <int R, int MT, int NKT, bool TLOAD>
__global__ __launch_bounds__(kDecWaves * 64) void proj_decode_kernel(ProjParams p)
{
    using S = DecShape<R, MT, NKT, TLOAD>;
    constexpr int NV = S::NV, NKK = S::NKK, U = S::U;
    extern __shared__ floatx4 red[];  // [kDecWaves][NV][64], then t [16 MT][16 NKT]
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r = lane & 15, qg = lane >> 4;
    const int n0 = blockIdx.x * 16 * R;
    const int proj = proj_of(p, n0);  // tiles never straddle projections (see launch_project)
    const int steps = p.K / 32;
    const int per = (steps + kDecWaves - 1) / kDecWaves;
    const int chunk = (wave + (int)blockIdx.x) % kDecWaves;
    const int s_begin = chunk * per, s_end = min(steps, s_begin + per);

    const uint16_t* wp[R];
    bool wok[R];
#pragma unroll
    for (int rt = 0; rt < R; ++rt) {
        wp[rt] = p.w + (size_t)min(n0 + 16 * rt + r, p.N - 1) * p.K + 8 * qg;
        wok[rt] = n0 + 16 * rt + r < p.N;
    }
    const uint16_t* xp[MT];
    bool xok[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        xp[mt] = p.x + (size_t)min(16 * mt + r, p.M - 1) * p.K + 8 * qg;
        xok[mt] = 16 * mt + r < p.M;
    }
    const uint16_t* ap[NKT > 0 ? NKT : 1];
    bool aok[NKT > 0 ? NKT : 1];
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt) {
        ap[kt] = p.a + (size_t)(proj * p.rank + min(16 * kt + r, p.rank - 1)) * p.K + 8 * qg;
        aok[kt] = 16 * kt + r < p.rank;
    }

    // the adapter up-projection operands of this wave's row tile (used after
    // the reduction) are loaded now, so that their latency overlaps the loop
    bf16x8 bop[NKK > 0 ? NKK : 1];
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk)
        bop[kk] = wave < R ? lora_weight_operand(p, n0 + 16 * (wave < R ? wave : 0) + r, proj, kk, qg) : zero_bf16x8();

    floatx4 acc[R][MT], tacc[MT][NKT > 0 ? NKT : 1];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
        for (int rt = 0; rt < R; ++rt)
            acc[rt][mt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kt = 0; kt < NKT; ++kt)
            tacc[mt][kt] = floatx4{0.f, 0.f, 0.f, 0.f};
    }
    for (int s = s_begin; s < s_end; s += U) {
        bf16x8 wv[R][U], xv[MT][U], av[NKT > 0 ? NKT : 1][U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const bool in = s + u < s_end;
#pragma unroll
            for (int rt = 0; rt < R; ++rt)
                wv[rt][u] = (in && wok[rt]) ? load_bf16x8(wp[rt] + 32 * (s + u)) : zero_bf16x8();
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
                xv[mt][u] = (in && xok[mt]) ? load_bf16x8(xp[mt] + 32 * (s + u)) : zero_bf16x8();
#pragma unroll
            for (int kt = 0; kt < NKT; ++kt)
                av[kt][u] = (in && aok[kt]) ? load_bf16x8(ap[kt] + 32 * (s + u)) : zero_bf16x8();
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
                for (int rt = 0; rt < R; ++rt)
                    acc[rt][mt] = mfma16_bf16(wv[rt][u], xv[mt][u], acc[rt][mt]);
#pragma unroll
                for (int kt = 0; kt < NKT; ++kt)
                    tacc[mt][kt] = mfma16_bf16(xv[mt][u], av[kt][u], tacc[mt][kt]);
            }
    }
    // reduce the eight waves' partials: slot v of every wave -> wave v % 8 sums it
#pragma unroll
    for (int rt = 0; rt < R; ++rt)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
            red[(wave * NV + rt * MT + mt) * 64 + lane] = acc[rt][mt];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int kt = 0; kt < NKT; ++kt)
            red[(wave * NV + R * MT + mt * NKT + kt) * 64 + lane] = tacc[mt][kt];
    __syncthreads();
    for (int v = wave; v < NV; v += kDecWaves) {
        floatx4 sum = red[v * 64 + lane];
#pragma unroll
        for (int w = 1; w < kDecWaves; ++w)
            sum += red[(w * NV + v) * 64 + lane];
        red[v * 64 + lane] = sum;  // wave 0's slots hold the totals
    }
    if constexpr (NKT > 0) {
        __syncthreads();
        // t[m][k] = scale * total, from the accumulator layout (lane: k = 16 kt + r,
        // m = 16 mt + 4 qg + i) to rows of m after the partial slots
        float* tl = (float*)(red + kDecWaves * NV * 64);
        constexpr int TK = 16 * NKT;
        if (wave == 0) {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int kt = 0; kt < NKT; ++kt) {
                    const floatx4 tv = red[(R * MT + mt * NKT + kt) * 64 + lane];
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        tl[(16 * mt + 4 * qg + i) * TK + 16 * kt + r] = tv[i] * p.scale;
                }
        }
        __syncthreads();
        if (wave >= R)
            return;
        // wave rt applies the K-extension to row tile rt
        const int rt = wave;
        floatx4 out[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
            out[mt] = red[(rt * MT + mt) * 64 + lane];
#pragma unroll
        for (int kk = 0; kk < NKK; ++kk) {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                float v[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int k = 32 * kk + 8 * qg + e;
                    v[e] = k < TK ? tl[(16 * mt + r) * TK + k] : 0.0f;
                }
                bf16x8 hi, lo;
                split_bf16x8(v, &hi, &lo);
                out[mt] = mfma16_bf16(bop[kk], hi, out[mt]);
                out[mt] = mfma16_bf16(bop[kk], lo, out[mt]);
            }
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                store_out(p, 16 * mt + r, n0 + 16 * rt + 4 * qg + i, out[mt][i]);
    } else {
        __syncthreads();
        if (wave >= R)
            return;
        const int rt = wave;
        floatx4 out[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
            out[mt] = red[(rt * MT + mt) * 64 + lane];
        if (TLOAD && p.rank > 0) {
            // K-extension with the activations of a separate pass (fp32 in p.t)
            const int nk = (p.rank + 31) / 32;
            for (int kk = 0; kk < nk; ++kk) {
                const bf16x8 bop = lora_weight_operand(p, n0 + 16 * rt + r, proj, kk, qg);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    bf16x8 hi, lo;
                    lora_token_operand(p, 16 * mt + r, proj, kk, qg, &hi, &lo);
                    out[mt] = mfma16_bf16(bop, hi, out[mt]);
                    out[mt] = mfma16_bf16(bop, lo, out[mt]);
                }
            }
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
                store_out(p, 16 * mt + r, n0 + 16 * rt + 4 * qg + i, out[mt][i]);
        }
    }
}

template <int R, int MT, int NKT, bool TLOAD>
hipError_t launch_decode_proj(const ProjParams& p, hipStream_t stream)
{
    constexpr size_t lds = DecShape<R, MT, NKT, TLOAD>::LDS;
    hipLaunchKernelGGL((proj_decode_kernel<R, MT, NKT, TLOAD>), dim3((p.N + 16 * R - 1) / (16 * R)),
                       dim3(kDecWaves * 64), lds, stream, p);
    return hipGetLastError();
}

// Decode-path dispatch.  Adapters of rank <= 16 are fused (each workgroup
// computes its projection's activations: one adapter row tile per row tile
// of weights); larger ranks read activations from a separate pass, since
// recomputing them per workgroup would read the adapter rows more often
// than the weights.  Workgroups take two row tiles when the output is wide
// enough to keep all compute units busy with half as many workgroups.
template <int MT>
hipError_t launch_decode_proj_m(const ProjParams& p, hipStream_t stream)
{
    const int dq = p.n1, dkv = p.n2 - p.n1;
    const bool two = p.N >= 4096 && dq % 32 == 0 && dkv % 32 == 0;
    if (p.yf || p.rank == 0)
        return two ? launch_decode_proj<2, MT, 0, false>(p, stream) : launch_decode_proj<1, MT, 0, false>(p, stream);
    if (p.a && p.rank <= 16)
        return two ? launch_decode_proj<2, MT, 1, false>(p, stream) : launch_decode_proj<1, MT, 1, false>(p, stream);
    return two ? launch_decode_proj<2, MT, 0, true>(p, stream) : launch_decode_proj<1, MT, 0, true>(p, stream);
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


// -------------------------------------------------------------------- gemm
// Large-M main pass: 256x256 output tile per workgroup, four waves in a 2x2
// grid of 128x128 sub-tiles, v_mfma_f32_32x32x16_bf16 (16 accumulators of
// 32x32 per wave).  A 128x128 sub-tile reads 64 bytes of LDS per 4096 MACs,
// half of what 64x64 sub-tiles need, which keeps the compute units' LDS
// bandwidth below what the matrix cores consume.
// Operands reach LDS through registers in two stages of K = 64: a copy moves
// 8 rows x 128 bytes (16 bytes per lane), so every cache line is fetched
// whole by one instruction (a 64-byte half-line per load doubles the requests
// the L2 serves).  Each stage's copies are loaded two stages before they are
// written to LDS (two register sets of 16 x 16 bytes per lane), which hides
// the latency of the L2 misses that the first touch of every row incurs.
// Chunk c (16 bytes) of row r sits at chunk position c ^ sw(r),
// sw(r) = (r & 7) ^ bit3(r): the 8 rows (32 banks) or 16 rows (64 banks)
// that one phase of a 16-byte fragment read serves fall on distinct banks.
// Workgroups take tiles so that the ones running together on an XCD form a
// patch of 4 row blocks x 8 column blocks, whose operands its L2 shares.
// The adapter branch is applied as a K-extension of the same accumulators
// (activation hi + lo times B_p), then outputs are rounded once to bf16.
constexpr int kGM = 256, kGN = 256, kGK = 64;
constexpr int kGStageBytes = (kGM + kGN) * kGK * 2;  // A then B rows of one stage
constexpr size_t kGLds = 2 * (size_t)kGStageBytes;

typedef float floatx16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ floatx16 mfma32_bf16(bf16x8 a, bf16x8 b, floatx16 c)
{
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ int gemm_swz(int row)
{
    return (row & 7) ^ ((row >> 3) & 1);
}

// Fused append of one 32-row slice pair of a K or V tile (the tile's two
// row halves, rows m0 + 128 h + 32 mi .. + 31, 256 columns, fp32 in the four
// waves' LDS regions): the outputs are rounded to bf16 as the unfused path
// stores them and coded as the append kernel codes them (per-token groups:
// statistics reduced over the group's lanes, one piece per thread).  A
// slice is 32 tokens of one sequence starting on a cache block, so each
// (row half, KV head) pair is one whole cache block: its pieces and
// metadata are assembled in LDS and written with contiguous 16-byte stores
// (value codes pass through LDS as bytes to be packed along tokens).
__device__ void fused_code_slices(const ProjParams& p, uint8_t* glds, int m0, int n0, int mi, int tid)
{
    const bool isv = n0 >= p.n2;
    const int col0 = n0 - (isv ? p.n2 : p.n1);
    const int D = p.cD, NB = p.cT / 32, hpt = 256 / D;  // KV heads per tile
    const int bits = isv ? p.v_bits : p.k_bits, mode = isv ? p.v_mode : p.k_mode;
    const int g = isv ? p.v_group : p.k_group, lanes = g / 8, ng = D / g;
    const int msz = p.meta16 ? 2 : 4;
    const int cbytes = 4 * D * bits, mcount = ng * 32;          // a block's code bytes, metadata elements
    uint8_t* vcode = glds + 4 * 32 * 128 * sizeof(float);       // [2][32][256] value codes
    uint8_t* stg = vcode + 2 * 32 * 256;                         // [2 hpt] blocks of pieces
    float* mss = (float*)(stg + 2 * 256 * 32 * bits / 8 * 1);    // [2 hpt][mcount] scales (fp32 or fp16)
    float* mzs = mss + 2 * 256;                                  // offsets
    for (int step = 0; step < 8; ++step) {
        const int idx = tid + kThreads * step;
        const int hh = idx >> 10, i = (idx >> 5) & 31, P = idx & 31;
        const float* src = (const float*)glds + (2 * hh + (P >> 4)) * (32 * 128) + i * 128 + 8 * (P & 15);
        float x[8];
#pragma unroll
        for (int e = 0; e < 8; ++e)
            x[e] = bf16_to_f32(f32_to_bf16(src[e]));
        float s, z;
        piece_group_stats(x, lanes, mode, bits, &s, &z);
        round_meta(p.meta16, &s, &z);
        const int hl = (8 * P) / D, Ph = ((8 * P) % D) / 8, q = hh * hpt + hl;
        if (Ph % lanes == 0) {
            const int mi_ = (Ph / lanes) * 32 + i;
            store_meta(mss + (p.meta16 ? q * mcount / 2 : q * mcount), mi_, s, p.meta16);
            if (mode == KVQ_AFFINE)
                store_meta(mzs + (p.meta16 ? q * mcount / 2 : q * mcount), mi_, z, p.meta16);
        }
        const float r = __builtin_amdgcn_rcpf(s);
        uint32_t c[8];
#pragma unroll
        for (int e = 0; e < 8; ++e)
            c[e] = code_one(x[e], s, r, z, mode, bits);
        if (!isv) {
            uint64_t word = 0;
#pragma unroll
            for (int e = 0; e < 8; ++e)
                word |= (uint64_t)c[e] << (bits * e);
            const int row = 4 * (i >> 3) + (i & 3), half = (i >> 2) & 1;
            store_piece(stg + q * cbytes, (half * 64 + row + 16 * (Ph & 3)) * (D / 32) + (Ph >> 2), bits, word);
        } else {
            *(uint2*)(vcode + (hh * 32 + i) * 256 + 8 * P) =
                make_uint2(c[0] | (c[1] << 8) | (c[2] << 16) | (c[3] << 24), c[4] | (c[5] << 8) | (c[6] << 16) | (c[7] << 24));
        }
    }
    __syncthreads();
    if (isv) {
        // value pieces (octet o, column cc): eight tokens of one channel
        for (int step = 0; step < 8; ++step) {
            const int idx = tid + kThreads * step;
            const int hh = idx >> 10, o = (idx >> 8) & 3, cc = idx & 255;
            uint64_t word = 0;
            for (int e = 0; e < 8; ++e)
                word |= (uint64_t)vcode[(hh * 32 + 8 * o + e) * 256 + cc] << (bits * e);
            const int hl = cc / D, d = cc % D, q = hh * hpt + hl;
            store_piece(stg + q * cbytes, ((d & 15) + 16 * o) * (D / 16) + (d >> 4), bits, word);
        }
        __syncthreads();
    }
    // whole blocks to the cache: codes, scales, offsets
    uint8_t* cdst = (uint8_t*)(isv ? (void*)p.vc : (void*)p.kc);
    uint8_t* sdst = (uint8_t*)(isv ? p.vs : p.ks);
    uint8_t* zdst = (uint8_t*)(isv ? p.vz : p.kz);
    for (int q = 0; q < 2 * hpt; ++q) {
        const int hh = q / hpt, hl = q % hpt;
        const int m = m0 + 128 * hh + 32 * mi;
        if (m >= p.M)
            continue;
        const int t = p.cn0 + m % p.cn_new;
        const int h = (col0 + D * hl) / D;
        const size_t blk = ((size_t)(m / p.cn_new) * p.cH + h) * NB + t / 32;
        for (int off = 16 * tid; off < cbytes; off += 16 * kThreads)
            *(u32x4*)(cdst + blk * cbytes + off) = *(const u32x4*)(stg + q * cbytes + off);
        const int mbytes = mcount * msz;
        const uint8_t* ms_ = (const uint8_t*)mss + q * mbytes;
        const uint8_t* mz_ = (const uint8_t*)mzs + q * mbytes;
        for (int off = 16 * tid; off < mbytes; off += 16 * kThreads) {
            *(u32x4*)(sdst + blk * mbytes + off) = *(const u32x4*)(ms_ + off);
            if (mode == KVQ_AFFINE)
                *(u32x4*)(zdst + blk * mbytes + off) = *(const u32x4*)(mz_ + off);
        }
    }
}

template <bool FUSE>
__global__ __launch_bounds__(kThreads) void proj_gemm_kernel(ProjParams p)
{
    extern __shared__ __attribute__((aligned(16))) uint8_t glds[];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    // tile order: XCD x (= workgroup id mod p.nxcd) takes the contiguous
    // range [x per, (x + 1) per) of tiles t, which run in groups of up to
    // kGroupM row blocks: t -> (row block g kGroupM + r % gm, column block r / gm)
    const int nbn = (p.N + kGN - 1) / kGN, nbm = (p.M + kGM - 1) / kGM;
    const int ntiles = nbn * nbm, nx = p.nxcd;
    const int per = (ntiles + nx - 1) / nx;
    const int t = (blockIdx.x % nx) * per + blockIdx.x / nx;
    if (t >= ntiles)
        return;
    constexpr int kGroupM = 4;
    const int grp = t / (kGroupM * nbn), rem = t % (kGroupM * nbn);
    const int gm = min(kGroupM, nbm - grp * kGroupM);
    const int m0 = (grp * kGroupM + rem % gm) * kGM, n0 = (rem / gm) * kGN;

    // Copies: a stage is 64 copies of 1 KiB (8 rows x 128 bytes), 0..31 the
    // A rows and 32..63 the B rows; wave w moves copies 16 w .. 16 w + 15, so
    // waves 0, 1 read A and waves 2, 3 read B, from a wave-uniform base (the
    // tile's first row) plus a 32-bit per-lane offset.  Lane i of a copy
    // writes LDS row 8 j + i / 8, chunk position i % 8, which holds source
    // chunk (i % 8) ^ sw(row).  Rows past M (N) re-read the last row; their
    // results are never stored.
    const bool wisb = wave >= 2;
    const uint64_t wbase0 = wisb ? (uint64_t)(p.w + (size_t)n0 * p.K) : (uint64_t)(p.x + (size_t)m0 * p.K);
    const uint32_t blo = __builtin_amdgcn_readfirstlane((uint32_t)wbase0);
    const uint32_t bhi = __builtin_amdgcn_readfirstlane((uint32_t)(wbase0 >> 32));
    const uint64_t wbase = ((uint64_t)bhi << 32) | blo;
    const int rlast = wisb ? p.N - 1 - n0 : p.M - 1 - m0;
    uint32_t voff[16];
#pragma unroll
    for (int c = 0; c < 16; ++c) {
        const int row = 8 * ((16 * wave + c) & 31) + (lane >> 3);
        const int chunk = (lane & 7) ^ gemm_swz(row);
        voff[c] = (uint32_t)min(row, rlast) * (uint32_t)p.K * 2u + 16u * (uint32_t)chunk;
    }
    const int nks = p.K / kGK;

    floatx16 acc[4][4];
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
        for (int ni = 0; ni < 4; ++ni)
            acc[mi][ni] = floatx16{};

    // fragment rows of this lane (A: tokens, B: weight rows); chunk c of a
    // row sits at LDS byte row * 128 + 16 (c ^ sw(row)), and the swizzle
    // depends only on the lane (the rows differ by multiples of 32)
    const int fr = lane & 31, fk = lane >> 5, sw = gemm_swz(fr);
    int aoff[4], boff[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
        aoff[kk] = (wm * 128 + fr) * 128 + 16 * ((2 * kk + fk) ^ sw);
        boff[kk] = kGM * kGK * 2 + (wn * 128 + fr) * 128 + 16 * ((2 * kk + fk) ^ sw);
    }

    // register staging: stage s's copies are loaded into R[s & 1] two stages
    // before they are written to LDS buffer s & 1; stages past the end
    // re-load the last one and land in a free buffer that is never read
    const uint8_t* gbase = (const uint8_t*)wbase;
    auto gload = [&](int kst, int j, u32x4* R) {
        const int kr = min(kst, nks - 1);
        R[j] = *(const __attribute__((address_space(1))) u32x4*)(gbase + (size_t)kr * kGK * 2 + voff[j]);
    };
    auto lstore = [&](int kst, int j, const u32x4* R) {
        *(u32x4*)(glds + (kst & 1) * kGStageBytes + (16 * wave + j) * 1024 + 16 * lane) = R[j];
    };
    auto fetch = [&](int ks, int kk, bf16x8* fa, bf16x8* fb) {
        const uint8_t* stg = glds + (ks & 1) * kGStageBytes;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            fa[i] = __builtin_bit_cast(bf16x8, *(const u32x4*)(stg + aoff[kk] + 4096 * i));
            fb[i] = __builtin_bit_cast(bf16x8, *(const u32x4*)(stg + boff[kk] + 4096 * i));
        }
    };
    // 16 MFMAs of one K = 16 step; after every 4th, one register copy moves:
    // lstore(sst, j) then gload(sst + 2, j) into the same register
    auto mma = [&](const bf16x8* fa, const bf16x8* fb, int sst, int j0, u32x4* R) {
#pragma unroll
        for (int mi = 0; mi < 4; ++mi) {
#pragma unroll
            for (int ni = 0; ni < 4; ++ni)
                acc[mi][ni] = mfma32_bf16(fa[mi], fb[ni], acc[mi][ni]);
            __builtin_amdgcn_sched_barrier(0);
            lstore(sst, j0 + mi, R);
            gload(sst + 2, j0 + mi, R);
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    u32x4 R0[16], R1[16];
#pragma unroll
    for (int j = 0; j < 16; ++j)
        gload(0, j, R0);
#pragma unroll
    for (int j = 0; j < 16; ++j)
        gload(1, j, R1);
#pragma unroll
    for (int j = 0; j < 16; ++j)
        lstore(0, j, R0);
#pragma unroll
    for (int j = 0; j < 16; ++j)
        gload(2, j, R0);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        lstore(1, j, R1);
        gload(3, j, R1);
    }
    __syncthreads();
    bf16x8 fa0[4], fb0[4], fa1[4], fb1[4];
    fetch(0, 0, fa0, fb0);
    // Pipeline, per stage ks (buffer ks & 1), four K = 16 steps t: the MFMAs
    // of step t run while the fragments of step t + 1 are read.  Steps 0..2
    // write copies 4..15 of stage ks + 1 (buffer free since the previous
    // barrier) from Rn = R[(ks + 1) & 1] and refill those registers with
    // stage ks + 3.  Between steps 2 and 3 a barrier makes stage ks + 1
    // readable and frees buffer ks & 1 (every wave has read its last
    // fragments of stage ks); step 3 then writes copies 0..3 of stage ks + 2
    // from Rc = R[ks & 1] and refills them with stage ks + 4.  A load thus
    // has two stages to land; the compiler's counters order each LDS write
    // after its load.
    auto body = [&](int ks, u32x4* Rc, u32x4* Rn) {
        fetch(ks, 1, fa1, fb1);
        __builtin_amdgcn_sched_barrier(0);
        mma(fa0, fb0, ks + 1, 4, Rn);
        fetch(ks, 2, fa0, fb0);
        __builtin_amdgcn_sched_barrier(0);
        mma(fa1, fb1, ks + 1, 8, Rn);
        fetch(ks, 3, fa1, fb1);
        __builtin_amdgcn_sched_barrier(0);
        mma(fa0, fb0, ks + 1, 12, Rn);
        __syncthreads();
        if (ks + 1 < nks)
            fetch(ks + 1, 0, fa0, fb0);
        __builtin_amdgcn_sched_barrier(0);
        mma(fa1, fb1, ks + 2, 0, Rc);
    };
    int ks = 0;
    for (; ks + 1 < nks; ks += 2) {
        body(ks, R0, R1);
        body(ks + 1, R1, R0);
    }
    if (ks < nks)
        body(ks, R0, R1);

    // adapter branch: K-extension over the rank, 16 at a time
    if (p.rank > 0) {
        const int p_lo = proj_of(p, n0), p_hi = proj_of(p, min(n0 + kGN, p.N) - 1);
        for (int proj = p_lo; proj <= p_hi; ++proj) {
            for (int k0 = 0; k0 < p.rank; k0 += 16) {
                bf16x8 wop[4];
#pragma unroll
                for (int ni = 0; ni < 4; ++ni) {
                    const int n = n0 + wn * 128 + 32 * ni + fr;
                    const bool ok = n < p.N && proj_of(p, n) == proj;
                    uint16_t v[8];
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const int k = k0 + 8 * fk + e;
                        v[e] = (ok && k < p.rank) ? p.bm[(size_t)n * p.rank + k] : (uint16_t)0;
                    }
                    u32x4 w4;
                    w4.x = v[0] | ((uint32_t)v[1] << 16);
                    w4.y = v[2] | ((uint32_t)v[3] << 16);
                    w4.z = v[4] | ((uint32_t)v[5] << 16);
                    w4.w = v[6] | ((uint32_t)v[7] << 16);
                    wop[ni] = __builtin_bit_cast(bf16x8, w4);
                }
#pragma unroll
                for (int mi = 0; mi < 4; ++mi) {
                    const int m = m0 + wm * 128 + 32 * mi + fr;
                    float v[8];
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const int k = k0 + 8 * fk + e;
                        v[e] = (m < p.M && k < p.rank) ? p.t[(size_t)m * 3 * p.rank + proj * p.rank + k] : 0.0f;
                    }
                    bf16x8 hi, lo;
                    split_bf16x8(v, &hi, &lo);
#pragma unroll
                    for (int ni = 0; ni < 4; ++ni) {
                        acc[mi][ni] = mfma32_bf16(hi, wop[ni], acc[mi][ni]);
                        acc[mi][ni] = mfma32_bf16(lo, wop[ni], acc[mi][ni]);
                    }
                }
            }
        }
    }

    // Output, one 32-row slice of each wave's sub-tile at a time through LDS
    // (the stage ring is free once every wave is past its last stage): the
    // 32x32 accumulator element e of lane l is row 8 (e / 4) + 4 (l / 32) +
    // e % 4, column l % 32 of its block; each lane then writes a pair of
    // adjacent columns of every row, rounded to bf16, so a row's 128 columns
    // are one 256-byte store per wave.
    float* xo = (float*)glds + wave * (32 * 128);
    const int rn0 = n0 + wn * 128;
    const int cpair = n0 + wn * 128 + 2 * lane;
    const int proj = proj_of(p, min(cpair, p.N - 1));
    uint16_t* ybase = proj == 0 ? p.y0 : proj == 1 ? p.y1 : p.y2;
    const int ywidth = proj == 0 ? p.n1 : proj == 1 ? p.n2 - p.n1 : p.N - p.n2;
    const int ycol = cpair - (proj == 0 ? 0 : proj == 1 ? p.n1 : p.n2);
    (void)rn0;
    const bool code_tile = FUSE && n0 >= p.n1;  // K and V tiles (tiles never straddle Q/K/V here)
#pragma unroll
    for (int mi = 0; mi < 4; ++mi) {
        __syncthreads();  // the previous slice's reads (or the last stage's) are done
#pragma unroll
        for (int ni = 0; ni < 4; ++ni)
#pragma unroll
            for (int e = 0; e < 16; ++e)
                xo[(8 * (e >> 2) + 4 * fk + (e & 3)) * 128 + 32 * ni + fr] = acc[mi][ni][e];
        __syncthreads();
        if (code_tile) {
            fused_code_slices(p, glds, m0, n0, mi, tid);
            continue;
        }
        const int mrow0 = m0 + wm * 128 + 32 * mi;
        for (int r = 0; r < 32; ++r) {
            const int m = mrow0 + r;
            const float2 v = *(const float2*)(xo + r * 128 + 2 * lane);
            if (m < p.M && cpair < p.N) {
                const uint32_t w = (uint32_t)f32_to_bf16(v.x) | ((uint32_t)f32_to_bf16(v.y) << 16);
                *(uint32_t*)(ybase + (size_t)m * ywidth + ycol) = w;
            }
        }
    }
}

// XCDs of the current device (1 when unknown), cached per device.
int gemm_xcds()
{
    static std::atomic<int> cached[64];
    int dev = 0, nx = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64)
        return 1;
    if ((nx = cached[dev].load(std::memory_order_relaxed)) > 0)
        return nx;
    if (hipDeviceGetAttribute(&nx, hipDeviceAttributeNumberOfXccs, dev) != hipSuccess || nx < 1)
        nx = 1;
    cached[dev].store(nx, std::memory_order_relaxed);
    return nx;
}

}  // namespace

hipError_t launch_project(const ProjParams& p, hipStream_t stream)
{
    if (p.M <= 0)
        return hipSuccess;
    if (p.M <= 32) {
        // fused path: W, H and (rank > 0) the adapter rows p.a in one kernel
        return p.M <= 16 ? launch_decode_proj_m<1>(p, stream) : launch_decode_proj_m<2>(p, stream);
    } else if (p.M >= kGM && p.N >= kGN && !p.yf && p.K % kGK == 0) {
        const int tiles = ((p.M + kGM - 1) / kGM) * ((p.N + kGN - 1) / kGN);
        ProjParams q = p;
        q.nxcd = gemm_xcds();
        const int per = (tiles + q.nxcd - 1) / q.nxcd;
        if (q.fuse)
            hipLaunchKernelGGL(proj_gemm_kernel<true>, dim3(per * q.nxcd), dim3(kThreads), kGLds, stream, q);
        else
            hipLaunchKernelGGL(proj_gemm_kernel<false>, dim3(per * q.nxcd), dim3(kThreads), kGLds, stream, q);
    } else {
        dim3 grid((p.N + kBN - 1) / kBN, (p.M + kBM - 1) / kBM);
        hipLaunchKernelGGL(proj_big_kernel, grid, dim3(kThreads), 0, stream, p);
    }
    return hipGetLastError();
}

}  // namespace kvq
