// Adapted Q/K/V projection (Sec. 3, Eq. (1)-(2); explicit adapter branch of
// Sec. 3.4):  y_p = W_p h + (alpha/r) B_p (A_p h)  for p in {Q, K, V}.
//
// Two passes, both on bf16 MFMA (v_mfma_f32_16x16x32_bf16, fp32 accumulate):
//   1. activation pass: t = (alpha/r) H A^T, fp32 [M][3r], into the workspace;
//   2. main pass: Y = H W^T, with the adapter branch fused as a K-extension
//      of the same accumulators: t_p (split into bf16 hi + lo parts) times
//      B_p^T, then one rounding to bf16 and routing of the columns to Q/K/V.
//
// M <= 32 (decode: one token per sequence) streams the weights from HBM
// with whole-line loads staged through LDS; its activation pass is split
// over K (see the decode section).  Larger M (prefill) uses a 256x256 tiled
// GEMM staged through LDS, or a 128x128 one for small shapes.

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
        const float t = v * p.scale;
        if (p.t_hilo) {
            // bf16 hi (nearest) and lo (remainder, nearest) of the scaled
            // activation (split_bf16x8's operands, precomputed), [M][3][2 r]:
            // in projection n / r's segment, rank column j's hi at
            // 32 (j / 16) + j % 16 and its lo 16 further, so that K stages
            // of 32 meet hi then lo of each 16 columns, the order in which
            // the K-extension after the main loop adds them
            const int r = p.N / 3, pj = n / r, j = n - pj * r;
            uint16_t* row = (uint16_t*)p.yf + (size_t)m * 2 * p.N + (size_t)pj * 2 * r + 32 * (j >> 4) + (j & 15);
            const uint16_t hi = f32_to_bf16(t);
            row[0] = hi;
            row[16] = f32_to_bf16(t - bf16_to_f32(hi));
        } else {
            p.yf[(size_t)m * p.N + n] = t;
        }
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

// ----------------------------------------------------------------- decode
// M <= 32 tokens (decode: one per sequence).  The weights stream from HBM in
// proj_stream_kernel: Y = H W^T, then the adapter branch (scale t_p) B_p^T
// as a K-extension of the same accumulators (t split into bf16 hi + lo), one
// rounding to bf16, routed to Q/K/V.  The adapter activations t = H A_p^T
// come from one of two places:
//   rank <= 16   the stream kernel computes them itself: its workgroups
//                stage the 16 rows of A_p along with W and H (A_p stays in
//                L2, read by every workgroup of projection p);
//   rank > 16    proj_tpart_kernel first writes partial sums over at most
//                kTSlices K slices (fp32 [slice][M][3r] in the workspace),
//                one workgroup per (16 adapter rows, K slice), so that the
//                larger A is read once; the stream kernel sums the slices.
//
// proj_stream_kernel: a workgroup owns RG = 8 G consecutive weight rows (G
// chosen so that the row groups cover the compute units about once) and all
// of K, with eight waves.  K is walked in 64-wide steps, step s going to wave
// s % 8, so the waves read 1 KiB runs of each row together.  Every global
// load is 16 bytes per lane over whole 128-byte lines: eight rows x 128 bytes
// per instruction.  (An MFMA operand fragment is 16 rows x 64 bytes, half
// lines, which the load path serves at a fraction of the rate, from L2 as
// well as from HBM.)  A wave writes its step's rows to its own LDS region
// (row pitch 160 bytes, which measured an order of magnitude fewer bank
// conflicts than 128 or 144 for these line writes and fragment reads), reads them back as v_mfma_f32_16x16x32_bf16 fragments
// (Y: A = 16 weight rows, B = 16 tokens; t: A = 16 tokens, B = 16 adapter
// rows) and accumulates.  Three register sets keep two steps of loads in
// flight while one is consumed.  The waves' partial sums are reduced in LDS.
// Weight tiles: 16 rows at offsets 0 and RG - 16 of the group (RG = 24: rows
// 8..15 are computed twice and stored once; RG = 8: the upper 8 fragment
// rows are never written and their outputs never stored).  A group that
// straddles a projection boundary also stages the second projection's
// adapter rows.  No group touches three projections: d_q and d_kv are
// multiples of 16 and a group of RG <= 32 rows starts at a multiple of RG, so
// it cannot hold rows on both sides of a 16-row (or longer) K block.
constexpr int kSWaves = 8;
constexpr int kSPitch = 160;   // bytes per staged row: 128 + 32
constexpr int kSXor = 0;       // chunk c of staged row r sits at chunk position c ^ (kSXor ? r & 7 : 0)

__device__ __forceinline__ int stage_off(int row, int chunk)
{
    return row * kSPitch + 16 * (kSXor ? (chunk ^ (row & 7)) : chunk);
}
constexpr int kTSlices = kProjTSlices;
constexpr int kTWaves = 4;

template <int G, int GH, bool FA>
struct StreamShape {
    static constexpr int RG = 8 * G;                   // weight rows per workgroup
    static constexpr int NTW = G <= 2 ? 1 : 2;         // 16-row weight tiles
    static constexpr int MT = (GH + 1) / 2;            // 16-token tiles
    static constexpr int WR = RG < 16 ? 16 : RG;       // staged weight rows
    static constexpr int HR = 16 * MT;                 // staged token rows
    static constexpr int AR = FA ? 32 : 0;             // staged adapter rows (two projections)
    static constexpr int WAVE_BYTES = (WR + HR + AR) * kSPitch;
    static constexpr int STAGE_BYTES = kSWaves * WAVE_BYTES;
    static constexpr int NSLOT = NTW * MT + (FA ? 2 * MT : 0);  // reduced accumulators
    static constexpr int RED_BYTES = kSWaves * NSLOT * 64 * 16;
    static constexpr int TL_OFFSET = STAGE_BYTES > RED_BYTES ? STAGE_BYTES : RED_BYTES;
};

// LDS bytes for the scaled adapter activations: two projections x M x rank fp32.
inline size_t stream_tl_bytes(int M, int rank)
{
    return (size_t)2 * M * rank * sizeof(float);
}

template <int G, int GH, bool FA>
struct StreamRegs {
    u32x4 w[G], h[GH], a[FA ? 2 : 1], a2[FA ? 2 : 1];
};

template <int G, int GH, bool FA>
__global__ __launch_bounds__(kSWaves * 64, 1) void proj_stream_kernel(ProjParams p)
{
    using S = StreamShape<G, GH, FA>;
    using Regs = StreamRegs<G, GH, FA>;
    constexpr int RG = S::RG, NTW = S::NTW, MT = S::MT, WR = S::WR, HR = S::HR;
    extern __shared__ __align__(16) uint8_t slds[];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r = lane & 15, qg = lane >> 4;
    const int r0 = blockIdx.x * RG;
    const int S64 = p.K / 64;
    const int NI = S64 > wave ? (S64 - wave + kSWaves - 1) / kSWaves : 0;  // this wave's steps
    // projections this group touches
    const int rend = min(r0 + RG, p.N);
    const int p_lo = proj_of(p, r0), p_hi = proj_of(p, rend - 1);
    const bool dual = FA && p_hi != p_lo;

    // line-load addresses: octet o covers rows 8 o + lane / 8, 16 bytes at column 8 (lane % 8)
    const int lrow = lane >> 3, lcol = 8 * (lane & 7);
    const uint16_t* wrow[G];
#pragma unroll
    for (int o = 0; o < G; ++o)
        wrow[o] = p.w + (size_t)min(r0 + 8 * o + lrow, p.N - 1) * p.K + lcol;
    const uint16_t* hrow[GH];
#pragma unroll
    for (int o = 0; o < GH; ++o)
        hrow[o] = p.x + (size_t)min(8 * o + lrow, p.M - 1) * p.K + lcol;
    const uint16_t *arow[2], *arow2[2];
#pragma unroll
    for (int o = 0; o < 2; ++o) {
        const int j = min(8 * o + lrow, max(p.rank, 1) - 1);
        arow[o] = FA ? p.a + (size_t)(p_lo * p.rank + j) * p.K + lcol : nullptr;
        arow2[o] = FA ? p.a + (size_t)(p_hi * p.rank + j) * p.K + lcol : nullptr;
    }
    uint8_t* region = slds + wave * S::WAVE_BYTES;

    // workgroups start their walk at different steps, so that the workgroups of
    // an XCD do not all read the same lines of H and A at the same time
    const int rot = NI > 0 ? (int)(blockIdx.x % (unsigned)NI) : 0;
    auto issue = [&](Regs& b, int i) {
        int ii = min(i, max(NI - 1, 0)) + rot;
        ii = ii >= NI ? ii - NI : ii;
        const int j = min(wave + kSWaves * ii, S64 - 1);
        const size_t k = (size_t)64 * j;
#pragma unroll
        for (int o = 0; o < G; ++o)
            b.w[o] = __builtin_nontemporal_load((const u32x4*)(wrow[o] + k));
#pragma unroll
        for (int o = 0; o < GH; ++o)
            b.h[o] = *(const u32x4*)(hrow[o] + k);
        if constexpr (FA) {
#pragma unroll
            for (int o = 0; o < 2; ++o)
                b.a[o] = *(const u32x4*)(arow[o] + k);
            if (dual) {
#pragma unroll
                for (int o = 0; o < 2; ++o)
                    b.a2[o] = *(const u32x4*)(arow2[o] + k);
            }
        }
        // keep the loads ahead of the step consumed next (the scheduler would sink them)
        __builtin_amdgcn_sched_barrier(0);
    };
    floatx4 acc[NTW][MT], tacc[MT][FA ? 2 : 1];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
        for (int tw = 0; tw < NTW; ++tw)
            acc[tw][mt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int u = 0; u < (FA ? 2 : 1); ++u)
            tacc[mt][u] = floatx4{0.f, 0.f, 0.f, 0.f};
    }
    auto frag = [&](int row, int hf) {
        return __builtin_bit_cast(bf16x8, *(const u32x4*)(region + stage_off(row, 4 * hf + qg)));
    };
    // line writes: octet starting at staged row r8 (a multiple of 8)
    auto put = [&](int r8, const u32x4& v) { *(u32x4*)(region + stage_off(r8 + lrow, lane & 7)) = v; };
    auto consume = [&](const Regs& b) {
#pragma unroll
        for (int o = 0; o < G; ++o)
            put(8 * o, b.w[o]);
#pragma unroll
        for (int o = 0; o < GH; ++o)
            put(WR + 8 * o, b.h[o]);
        if constexpr (FA) {
#pragma unroll
            for (int o = 0; o < 2; ++o)
                put(WR + HR + 8 * o, b.a[o]);
            if (dual) {
#pragma unroll
                for (int o = 0; o < 2; ++o)
                    put(WR + HR + 16 + 8 * o, b.a2[o]);
            }
        }
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
            bf16x8 wf[NTW], xf[MT];
#pragma unroll
            for (int tw = 0; tw < NTW; ++tw)
                wf[tw] = frag((tw == NTW - 1 ? (RG < 16 ? 0 : RG - 16) : 16 * tw) + r, hf);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
                xf[mt] = frag(WR + 16 * mt + r, hf);
#pragma unroll
            for (int tw = 0; tw < NTW; ++tw)
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                    acc[tw][mt] = mfma16_bf16(wf[tw], xf[mt], acc[tw][mt]);
            if constexpr (FA) {
                const bf16x8 af = frag(WR + HR + r, hf);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                    tacc[mt][0] = mfma16_bf16(xf[mt], af, tacc[mt][0]);
                if (dual) {
                    const bf16x8 af2 = frag(WR + HR + 16 + r, hf);
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt)
                        tacc[mt][1] = mfma16_bf16(xf[mt], af2, tacc[mt][1]);
                }
            }
        }
    };

    float* tl = (float*)(slds + S::TL_OFFSET);  // scaled t: [p - p_lo][M][rank]
    // epilogue slot of this wave (Y tile tw, token tile mt; waves below NTW MT) and
    // the extension's weight operands B_p, loaded now so that their latency
    // overlaps the main loop
    const int tw = wave / MT, mt = wave % MT;
    const int off = tw >= NTW - 1 ? (RG < 16 ? 0 : RG - 16) : 16 * tw;  // tile's first row in the group
    const int nk = (p.rank + 31) / 32;
    bf16x8 bop[2][2];
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
            bop[u][kk] = (wave < NTW * MT && p_lo + u <= p_hi && kk < nk)
                             ? lora_weight_operand(p, r0 + off + r, p_lo + u, kk, qg)
                             : zero_bf16x8();
    Regs b0, b1, b2;
    issue(b0, 0);
    issue(b1, 1);
    if (!FA && p.rank > 0) {
        // sum the partial activations of the slices
        const int per = p.M * p.rank, n = (p_hi - p_lo + 1) * per, ld = 3 * p.rank;
        for (int e = threadIdx.x; e < n; e += kSWaves * 64) {
            const int pj = e / per, m = (e % per) / p.rank, k = e % p.rank;
            const float* src = p.t + (size_t)m * ld + (p_lo + pj) * p.rank + k;
            float v[kTSlices];
#pragma unroll
            for (int s = 0; s < kTSlices; ++s)
                v[s] = src[(size_t)min(s, p.tslices - 1) * p.M * ld];
            float sum = 0.0f;
#pragma unroll
            for (int s = 0; s < kTSlices; ++s)
                sum += s < p.tslices ? v[s] : 0.0f;
            tl[e] = sum * p.scale;
        }
    }
    int i = 0;
    for (; i + 5 <= NI; i += 3) {
        issue(b2, i + 2);
        consume(b0);
        issue(b0, i + 3);
        consume(b1);
        issue(b1, i + 4);
        consume(b2);
    }
    switch (NI - i) {
    case 4:
        issue(b2, i + 2);
        consume(b0);
        issue(b0, i + 3);
        consume(b1);
        consume(b2);
        consume(b0);
        break;
    case 3:
        issue(b2, i + 2);
        consume(b0);
        consume(b1);
        consume(b2);
        break;
    case 2:
        consume(b0);
        consume(b1);
        break;
    case 1:
        consume(b0);
        break;
    default:
        break;
    }

    // reduce the waves' partials: slot v of every wave -> wave v sums it
    // (slots: Y tiles tw MT + mt, then the activations NTW MT + 2 mt + u)
    __syncthreads();
    floatx4* red = (floatx4*)slds;
    constexpr int NS = S::NSLOT;
#pragma unroll
    for (int tw = 0; tw < NTW; ++tw)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
            red[(wave * NS + tw * MT + mt) * 64 + lane] = acc[tw][mt];
    if constexpr (FA) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int u = 0; u < 2; ++u)
                red[(wave * NS + NTW * MT + 2 * mt + u) * 64 + lane] = tacc[mt][u];
    }
    __syncthreads();
    floatx4 out = floatx4{0.f, 0.f, 0.f, 0.f};
    for (int v = wave; v < NS; v += kSWaves) {
        floatx4 sum = red[v * 64 + lane];
#pragma unroll
        for (int w = 1; w < kSWaves; ++w)
            sum += red[(w * NS + v) * 64 + lane];
        if (v < NTW * MT) {
            out = sum;
        } else if (FA) {
            // activations: lane holds adapter row r (k), tokens 16 mt + 4 qg + e
            const int mt = (v - NTW * MT) / 2, u = (v - NTW * MT) % 2;
            if (u == 0 || dual) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int m = 16 * mt + 4 * qg + e;
                    if (m < p.M && r < p.rank)
                        tl[((size_t)u * p.M + m) * p.rank + r] = sum[e] * p.scale;
                }
            }
        }
    }
    if constexpr (FA)
        __syncthreads();
    if (wave >= NTW * MT)
        return;
    if (p.rank > 0) {
        const int m = 16 * mt + r;
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            if (p_lo + u > p_hi)
                break;
            const float* tp = tl + (size_t)u * p.M * p.rank + (size_t)min(m, p.M - 1) * p.rank;
#pragma unroll
            for (int kk = 0; kk < 2; ++kk) {
                if (kk >= nk)
                    break;
                float v[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int k = 32 * kk + 8 * qg + e;
                    v[e] = (m < p.M && k < p.rank) ? tp[k] : 0.0f;
                }
                bf16x8 hi, lo;
                split_bf16x8(v, &hi, &lo);
                out = mfma16_bf16(bop[u][kk], hi, out);
                out = mfma16_bf16(bop[u][kk], lo, out);
            }
        }
    }
    // lane: token 16 mt + r, rows off + 4 qg .. + 3 of the group (one projection: boundaries are multiples of 16)
    const int m = 16 * mt + r, lr = off + 4 * qg, n = r0 + lr;
    const bool mine = lr >= 16 * tw && lr < RG;  // rows this tile stores
    if (!mine || m >= p.M || n >= p.N)
        return;
    uint16_t o4[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
        o4[e] = f32_to_bf16(out[e]);
    uint16_t* dst;
    if (n < p.n1) {
        dst = p.y0 + (size_t)m * p.n1 + n;
    } else if (p.kr) {
        // window append: the bf16 value converted to fp16 (as the append of
        // the bf16 K / V stores it), at head h, channel d of the new slot
        const bool isv = n >= p.n2;
        const int col = n - (isv ? p.n2 : p.n1), h = col / p.cD, d = col % p.cD;
#pragma unroll
        for (int e = 0; e < 4; ++e)
            o4[e] = f32_to_f16_bits(bf16_to_f32(o4[e]));
        dst = (isv ? p.vr : p.kr) + (((size_t)m * p.cH + h) * p.rslots + p.rslot) * p.cD + d;
    } else if (n < p.n2) {
        dst = p.y1 + (size_t)m * (p.n2 - p.n1) + (n - p.n1);
    } else {
        dst = p.y2 + (size_t)m * (p.N - p.n2) + (n - p.n2);
    }
    *(uint2*)dst = uint2{o4[0] | ((uint32_t)o4[1] << 16), o4[2] | ((uint32_t)o4[3] << 16)};
}

// Partial adapter activations: workgroup (jt, ks) computes
// tpart[ks][m][16 jt + j] = sum over its K slice of H[m][k] A[16 jt + j][k]
// (unscaled), four waves over the slice's 32-wide steps, reduced in LDS.
// MFMA roles: A = H rows (16 tokens), B = A^T (16 adapter rows).
template <int MT>
__global__ __launch_bounds__(kTWaves * 64) void proj_tpart_kernel(ProjParams p, int slice)
{
    __shared__ floatx4 red[kTWaves][MT][64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r = lane & 15, qg = lane >> 4;
    const int jt = blockIdx.x, ks = blockIdx.y;
    const int rows = 3 * p.rank;
    const int k0 = ks * slice, k1 = min(p.K, k0 + slice);
    const uint16_t* ap = p.a + (size_t)min(16 * jt + r, rows - 1) * p.K + 8 * qg;
    const uint16_t* xp[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
        xp[mt] = p.x + (size_t)min(16 * mt + r, p.M - 1) * p.K + 8 * qg;
    floatx4 acc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
        acc[mt] = floatx4{0.f, 0.f, 0.f, 0.f};
    for (int k = k0 + 32 * wave; k < k1; k += 32 * kTWaves) {
        const bf16x8 av = load_bf16x8(ap + k);
        bf16x8 xv[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
            xv[mt] = load_bf16x8(xp[mt] + k);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
            acc[mt] = mfma16_bf16(xv[mt], av, acc[mt]);
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
        red[wave][mt][lane] = acc[mt];
    __syncthreads();
    if (wave >= MT)
        return;
    floatx4 s = red[0][wave][lane];
#pragma unroll
    for (int w = 1; w < kTWaves; ++w)
        s += red[w][wave][lane];
    // lane: adapter row 16 jt + r, tokens 16 mt + 4 qg + e
    const int j = 16 * jt + r;
    if (j >= rows)
        return;
    float* dst = p.yf + (size_t)ks * p.M * rows + j;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int m = 16 * wave + 4 * qg + e;
        if (m < p.M)
            dst[(size_t)m * rows] = s[e];
    }
}

// Compute units of the current device (256 when unknown), cached per device.
int stream_compute_units()
{
    static std::atomic<int> cached[64];
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64)
        return 256;
    if ((cus = cached[dev].load(std::memory_order_relaxed)) > 0)
        return cus;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
        cus = 256;
    cached[dev].store(cus, std::memory_order_relaxed);
    return cus;
}

template <int G, int GH, bool FA>
hipError_t launch_stream(const ProjParams& p, hipStream_t stream)
{
    using S = StreamShape<G, GH, FA>;
    const size_t lds = S::TL_OFFSET + (p.rank > 0 ? stream_tl_bytes(p.M, p.rank) : 0);
    launch_kernel((proj_stream_kernel<G, GH, FA>), dim3((p.N + S::RG - 1) / S::RG), dim3(kSWaves * 64), lds,
                       stream, p);
    return hipGetLastError();
}

template <int G, bool FA>
hipError_t launch_stream_g(const ProjParams& p, hipStream_t stream)
{
    if (p.M <= 8)
        return launch_stream<G, 1, FA>(p, stream);
    if (p.M <= 16)
        return launch_stream<G, 2, FA>(p, stream);
    return launch_stream<G, 4, FA>(p, stream);
}

template <bool FA>
hipError_t launch_stream_fa(const ProjParams& p, int G, hipStream_t stream)
{
    switch (G) {
    case 1:
        return launch_stream_g<1, FA>(p, stream);
    case 2:
        return launch_stream_g<2, FA>(p, stream);
    case 3:
        return launch_stream_g<3, FA>(p, stream);
    default:
        return launch_stream_g<4, FA>(p, stream);
    }
}

// --------------------------------------------------------------------- big
// (32 MI)x128 output tile, four waves in a 2x2 grid of (16 MI)x64 sub-tiles,
// K step 64 through double-buffered LDS (rows padded by 16 bytes).  MI = 4
// (128-row tiles), or MI = 1 for an activation pass (N = 3 r <= 192
// columns) too short to cover the compute units with 128-row tiles.
// MFMA roles: A = H rows (M-dim = tokens), B = W^T (N-dim = weight rows).
// Output lane layout: token m = row base + 4 qg + i, column n = base + lane % 16.
constexpr int kBM = 128, kBN = 128, kBK = 64, kLdsRow = kBK + 8;

template <int MI>
__global__ __launch_bounds__(kThreads) void proj_big_kernel(ProjParams p)
{
    constexpr int BM = 32 * MI;
    __shared__ uint16_t As[2][BM * kLdsRow];
    __shared__ uint16_t Bs[2][kBN * kLdsRow];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int r = lane & 15, qg = lane >> 4;
    const int wm = wave >> 1, wn = wave & 1;
    const int m0 = blockIdx.y * BM, n0 = blockIdx.x * kBN;

    // Global -> register staging: 16-byte chunks, MI per thread for the H
    // rows and 4 for the W rows.
    u32x4 ra[MI], rb[4];
    auto gload = [&](int k0) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            int idx = tid + kThreads * i;      // 0..1023
            int row = idx >> 3, c8 = (idx & 7) * 8;
            int m = m0 + row, n = n0 + row;
            if (i < MI)
                ra[i] = m < p.M ? *(const u32x4*)(p.x + (size_t)m * p.K + k0 + c8) : u32x4{0u, 0u, 0u, 0u};
            rb[i] = n < p.N ? *(const u32x4*)(p.w + (size_t)n * p.K + k0 + c8) : u32x4{0u, 0u, 0u, 0u};
        }
    };
    auto lstore = [&](int buf) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            int idx = tid + kThreads * i;
            int row = idx >> 3, c8 = (idx & 7) * 8;
            if (i < MI)
                *(u32x4*)(&As[buf][row * kLdsRow + c8]) = ra[i];
            *(u32x4*)(&Bs[buf][row * kLdsRow + c8]) = rb[i];
        }
    };

    floatx4 acc[MI][4];
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
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
            bf16x8 af[MI], bfr[4];
#pragma unroll
            for (int mi = 0; mi < MI; ++mi)
                af[mi] = __builtin_bit_cast(
                    bf16x8, *(const u32x4*)(&As[buf][(wm * 16 * MI + 16 * mi + r) * kLdsRow + 32 * kk + 8 * qg]));
#pragma unroll
            for (int ni = 0; ni < 4; ++ni)
                bfr[ni] = __builtin_bit_cast(
                    bf16x8, *(const u32x4*)(&Bs[buf][(wn * 64 + 16 * ni + r) * kLdsRow + 32 * kk + 8 * qg]));
#pragma unroll
            for (int mi = 0; mi < MI; ++mi)
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
                for (int mi = 0; mi < MI; ++mi) {
                    bf16x8 hi, lo;
                    lora_token_operand(p, m0 + wm * 16 * MI + 16 * mi + r, proj, kk, qg, &hi, &lo);
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
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int ni = 0; ni < 4; ++ni)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                store_out(p, m0 + wm * 16 * MI + 16 * mi + 4 * qg + i, n0 + wn * 64 + 16 * ni + r, acc[mi][ni][i]);
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

// Large-M main pass with plain outputs (the fused append keeps the kernel
// above): the same 256x256 output tile and tile order, computed by eight
// waves, two per SIMD, each owning a 64x128 sub-tile (2x4 accumulators of
// v_mfma_f32_32x32x16_bf16, 128 registers).  Operands reach LDS by
// global_load_lds_dwordx4 (16 bytes per lane straight into LDS, no
// registers) in a ring of kPNst stages of K = 32: rows of 64 bytes, chunk c
// of row r at chunk position c ^ ((r >> 2) & 3), which measured free of bank
// conflicts for the 32-row fragment reads (the xor of bits 1 and 3 left four
// conflict cycles per read).  The two waves of a SIMD alternate roles at
// every barrier: while one runs the 16 MFMAs of a stage from registers, the
// other reads its next stage's fragments from LDS and issues its copies four
// stages ahead (waves 0-3 copy the A rows, 4-7 the B rows).  A stage's LDS
// traffic (96 KiB of fragment reads, 32 KiB of copies) is what bounds this
// kernel; the four-wave kernel reads a third less per MFMA but cannot hide
// its barrier and copy latency with one wave per SIMD.
constexpr int kPThreads = 512, kPK = 32, kPNst = 5;
constexpr int kPStage = (kGM + kGN) * kPK * 2;    // 32 KiB: A rows then B rows
constexpr size_t kPLds = (size_t)kPNst * kPStage;  // 160 KiB

__device__ __forceinline__ int pp_swz(int row)
{
    return (row >> 2) & 3;
}

// 16 bytes per lane from global memory to LDS address lds_addr + 16 lane
// (lds_addr wave-uniform, held in M0 while the copy issues).  Inline
// assembly, so that the compiler does not make LDS reads wait for every
// outstanding copy; the kernel's own vmcnt waits order them.
__device__ __forceinline__ void pp_copy16(uint64_t base, uint32_t voff, uint32_t lds_addr)
{
    const uint32_t m0v = __builtin_amdgcn_readfirstlane(lds_addr);
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2" : : "s"(m0v), "v"(voff), "s"(base) : "memory");
}

__global__ __launch_bounds__(kPThreads, 1) void proj_gemm_pp_kernel(ProjParams p)
{
    extern __shared__ __attribute__((aligned(16))) uint8_t glds[];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int grp = wave >> 2, wm = wave & 3, wn = wave >> 2;
    // tile order as in proj_gemm_kernel
    const int nbn = (p.N + kGN - 1) / kGN, nbm = (p.M + kGM - 1) / kGM;
    const int ntiles = nbn * nbm, nx = p.nxcd;
    const int per = (ntiles + nx - 1) / nx;
    const int t = (blockIdx.x % nx) * per + blockIdx.x / nx;
    if (t >= ntiles)
        return;
    constexpr int kGroupM = 4;
    const int g = t / (kGroupM * nbn), rem = t % (kGroupM * nbn);
    const int gm = min(kGroupM, nbm - g * kGroupM);
    const int m0 = (g * kGroupM + rem % gm) * kGM, n0 = (rem / gm) * kGN;

    // copies: a stage is 32 copies of 1 KiB (16 rows x 64 bytes), 0..15 the A
    // rows and 16..31 the B rows; wave w moves copies 4 w .. 4 w + 3.  Lane i
    // of a copy writes LDS row 16 j + i / 4, chunk position i % 4, which holds
    // source chunk (i % 4) ^ swz(row).  Rows past M (N) re-read the last row;
    // their results are never stored.
    const bool wisb = wave >= 4;
    const uint64_t gbase = wisb ? (uint64_t)(p.w + (size_t)n0 * p.K) : (uint64_t)(p.x + (size_t)m0 * p.K);
    const int rlast = wisb ? p.N - 1 - n0 : p.M - 1 - m0;
    uint32_t voff[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const int row = 16 * ((4 * wave + c) & 15) + (lane >> 2);
        voff[c] = (uint32_t)min(row, rlast) * (uint32_t)p.K * 2u + 16u * (uint32_t)((lane & 3) ^ pp_swz(row));
    }
    const uint32_t lbase = (uint32_t)(uintptr_t)glds;
    const int nks = p.K / kPK;
    // With t_hilo the adapter follows as rank / 16 more stages: stage e's A
    // rows are the tile's activation rows (hi then lo of rank columns
    // 16 e .. 16 e + 15, of the tile's projection), its B rows the tile's
    // B_p rows at those 16 columns, twice.
    const bool ext = p.t_hilo && p.rank > 0;
    const int nst = nks + (ext ? p.rank / 16 : 0);
    const int tproj = proj_of(p, n0);
    constexpr int kAhead = kPNst - 1;  // stages in flight ahead of the one being read
    // copies of stage ks into ring slot ks % kPNst; stages past the end
    // re-load the last one into a slot that is never read again
    auto copy_stage = [&](int ks) {
        const int kc = min(ks, nst - 1);
        const uint32_t lds_at = lbase + (ks % kPNst) * kPStage;
        if (kc < nks) {
            const uint64_t b = gbase + (uint64_t)kc * (kPK * 2);
            const uint32_t bl = __builtin_amdgcn_readfirstlane((uint32_t)b);
            const uint32_t bh = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
            const uint64_t bs = ((uint64_t)bh << 32) | bl;
#pragma unroll
            for (int c = 0; c < 4; ++c)
                pp_copy16(bs, voff[c], lds_at + (4 * wave + c) * 1024);
        } else {
            const int e = kc - nks, r = p.rank;
            const uint64_t b = wisb ? (uint64_t)(p.bm + (size_t)n0 * r)
                                    : (uint64_t)((const uint16_t*)p.t + (size_t)m0 * 6 * r + (size_t)tproj * 2 * r + 32 * e);
            const uint32_t bl = __builtin_amdgcn_readfirstlane((uint32_t)b);
            const uint32_t bh = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
            const uint64_t bs = ((uint64_t)bh << 32) | bl;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int row = 16 * ((4 * wave + c) & 15) + (lane >> 2);
                const int src = (lane & 3) ^ pp_swz(row);
                const uint32_t rc = (uint32_t)min(row, rlast);
                const uint32_t vo = wisb ? rc * 2u * (uint32_t)r + 2u * (uint32_t)(16 * e + 8 * (src & 1))
                                         : rc * 12u * (uint32_t)r + 16u * (uint32_t)src;
                pp_copy16(bs, vo, lds_at + (4 * wave + c) * 1024);
            }
        }
    };

    // fragments: A rows 64 wm + 32 i + l % 32, B rows 128 wn + 32 j + l % 32,
    // chunk 2 kt + l / 32 of a stage
    const int fr = lane & 31, fk = lane >> 5;
    uint32_t aoff[2][2], boff[2][4];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int r = 64 * wm + 32 * i + fr;
            aoff[kt][i] = r * 64 + 16 * ((2 * kt + fk) ^ pp_swz(r));
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int r = 128 * wn + 32 * j + fr;
            boff[kt][j] = kGM * 64 + r * 64 + 16 * ((2 * kt + fk) ^ pp_swz(r));
        }
    }
    floatx16 acc[2][4];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
            acc[i][j] = floatx16{};
    bf16x8 fa[2][2], fb[2][4];
    // memory role: this stage's fragments into registers, copies kAhead stages ahead
    auto mem_phase = [&](int ks) {
        const uint8_t* sb = glds + (ks % kPNst) * kPStage;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
            for (int i = 0; i < 2; ++i)
                fa[kt][i] = __builtin_bit_cast(bf16x8, *(const u32x4*)(sb + aoff[kt][i]));
#pragma unroll
            for (int j = 0; j < 4; ++j)
                fb[kt][j] = __builtin_bit_cast(bf16x8, *(const u32x4*)(sb + boff[kt][j]));
        }
        copy_stage(ks + kAhead);
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): the reads are done before the slot is handed on
        __builtin_amdgcn_sched_barrier(0);
    };
    // compute role: the stage's 16 MFMAs
    auto mfma_phase = [&]() {
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[i][j] = mfma32_bf16(fa[kt][i], fb[kt][j], acc[i][j]);
    };
    // barrier between roles; before it every wave waits for its copies of
    // all but the two newest stages (vmcnt(8)), so the stage read next has
    // landed in LDS whichever wave copied it
    auto swap = [&]() {
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_waitcnt(0x0F78);  // vmcnt(8)
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
    };

    uint32_t m0_saved;
    asm volatile("s_mov_b32 %0, m0" : "=s"(m0_saved));
#pragma unroll
    for (int ks = 0; ks < kAhead; ++ks)
        copy_stage(ks);
    swap();
    // Wave group 1 reads stage ks while group 0 computes stage ks - 1, then
    // the roles swap; both groups pass 2 nst + 1 barriers.
    if (grp == 1) {
        for (int ks = 0; ks < nst; ++ks) {
            mem_phase(ks);
            swap();
            mfma_phase();
            swap();
        }
    } else {
        for (int ks = 0; ks < nst; ++ks) {
            if (ks > 0)
                mfma_phase();
            swap();
            mem_phase(ks);
            swap();
        }
        mfma_phase();
    }
    asm volatile("s_mov_b32 m0, %0" ::"s"(m0_saved));
    __builtin_amdgcn_s_waitcnt(0);  // the trailing copies have landed before the ring is reused

    // adapter branch without t_hilo: K-extension over the rank, 16 at a
    // time, after the main loop (its loads are then a latency of their own).
    // With the rank a multiple of 16 a lane's eight B_p values and eight
    // activations are two or three 16-byte loads (rows past M or N clamped,
    // their operands zeroed), all issued before the MFMAs of their step.
    if (p.rank > 0 && !ext) {
        const bool vec = (p.rank & 15) == 0;
        const int p_lo = proj_of(p, n0), p_hi = proj_of(p, min(n0 + kGN, p.N) - 1);
        for (int proj = p_lo; proj <= p_hi; ++proj) {
            for (int k0 = 0; k0 < p.rank; k0 += 16) {
                bf16x8 wop[4];
                float tv[2][8];
#pragma unroll
                for (int ni = 0; ni < 4; ++ni) {
                    const int n = n0 + wn * 128 + 32 * ni + fr;
                    const bool ok = n < p.N && proj_of(p, n) == proj;
                    if (vec) {
                        const u32x4 w4 = *(const u32x4*)(p.bm + (size_t)min(n, p.N - 1) * p.rank + k0 + 8 * fk);
                        wop[ni] = ok ? __builtin_bit_cast(bf16x8, w4) : zero_bf16x8();
                    } else {
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
                }
#pragma unroll
                for (int mi = 0; mi < 2; ++mi) {
                    const int m = m0 + wm * 64 + 32 * mi + fr;
                    if (vec) {
                        const float* tr = p.t + (size_t)min(m, p.M - 1) * 3 * p.rank + proj * p.rank + k0 + 8 * fk;
                        const float4 a = *(const float4*)tr, b = *(const float4*)(tr + 4);
                        const bool ok = m < p.M;
                        tv[mi][0] = ok ? a.x : 0.0f;
                        tv[mi][1] = ok ? a.y : 0.0f;
                        tv[mi][2] = ok ? a.z : 0.0f;
                        tv[mi][3] = ok ? a.w : 0.0f;
                        tv[mi][4] = ok ? b.x : 0.0f;
                        tv[mi][5] = ok ? b.y : 0.0f;
                        tv[mi][6] = ok ? b.z : 0.0f;
                        tv[mi][7] = ok ? b.w : 0.0f;
                    } else {
#pragma unroll
                        for (int e = 0; e < 8; ++e) {
                            const int k = k0 + 8 * fk + e;
                            tv[mi][e] = (m < p.M && k < p.rank) ? p.t[(size_t)m * 3 * p.rank + proj * p.rank + k] : 0.0f;
                        }
                    }
                }
#pragma unroll
                for (int mi = 0; mi < 2; ++mi) {
                    bf16x8 hi, lo;
                    split_bf16x8(tv[mi], &hi, &lo);
#pragma unroll
                    for (int ni = 0; ni < 4; ++ni) {
                        acc[mi][ni] = mfma32_bf16(hi, wop[ni], acc[mi][ni]);
                        acc[mi][ni] = mfma32_bf16(lo, wop[ni], acc[mi][ni]);
                    }
                }
            }
        }
    }


    // Output, one 32-row slice of the wave's sub-tile at a time through the
    // wave's own LDS region (the ring is free once every wave is past the
    // barrier below): accumulator element e of lane l is row 8 (e / 4) +
    // 4 (l / 32) + e % 4, column l % 32 of its block; each lane then writes a
    // pair of adjacent columns of every row, rounded to bf16.
    __syncthreads();
    float* xo = (float*)glds + wave * (32 * 128);
    const int cpair = n0 + wn * 128 + 2 * lane;
    const int proj = proj_of(p, min(cpair, p.N - 1));
    uint16_t* ybase = proj == 0 ? p.y0 : proj == 1 ? p.y1 : p.y2;
    const int ywidth = proj == 0 ? p.n1 : proj == 1 ? p.n2 - p.n1 : p.N - p.n2;
    const int ycol = cpair - (proj == 0 ? 0 : proj == 1 ? p.n1 : p.n2);
#pragma unroll
    for (int mi = 0; mi < 2; ++mi) {
        // a wave's LDS accesses are performed in order: its reads of the
        // previous slice are done before these writes, and these before the reads
#pragma unroll
        for (int ni = 0; ni < 4; ++ni)
#pragma unroll
            for (int e = 0; e < 16; ++e)
                xo[(8 * (e >> 2) + 4 * fk + (e & 3)) * 128 + 32 * ni + fr] = acc[mi][ni][e];
        const int mrow0 = m0 + wm * 64 + 32 * mi;
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

bool project_adapter_stages(int M, int d_in, int d_q, int d_kv, int rank)
{
    return rank > 0 && rank % 16 == 0 && M >= kGM && d_q + 2 * d_kv >= kGN && d_in % kGK == 0 && d_q % kGN == 0 &&
           d_kv % kGN == 0;
}

hipError_t launch_project_decode(const ProjParams& p, hipStream_t stream)
{
    if (p.M <= 0)
        return hipSuccess;
    if (p.M > 32 || p.K % 64 != 0)
        return hipErrorInvalidValue;
    ProjParams q = p;
    q.tslices = 0;
    const bool fused = p.rank > 0 && p.rank <= 16;
    if (p.rank > 16) {
        // K slices: whole 64-wide steps, at most kTSlices of them
        const int s64 = p.K / 64, per = (s64 + kTSlices - 1) / kTSlices;
        q.tslices = (s64 + per - 1) / per;
        ProjParams a = p;
        a.yf = (float*)p.t;
        dim3 grid((3 * p.rank + 15) / 16, q.tslices);
        if (p.M <= 16)
            launch_kernel(proj_tpart_kernel<1>, grid, dim3(kTWaves * 64), 0, stream, a, 64 * per);
        else
            launch_kernel(proj_tpart_kernel<2>, grid, dim3(kTWaves * 64), 0, stream, a, 64 * per);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess)
            return e;
    }
    // row groups of 8 G rows: the smallest G whose groups fit the compute units once (at most 4)
    const int octets = (p.N + 7) / 8, cus = stream_compute_units();
    const int G = min(4, max(1, (octets + cus - 1) / cus));
    return fused ? launch_stream_fa<true>(q, G, stream) : launch_stream_fa<false>(q, G, stream);
}

hipError_t launch_project(const ProjParams& p, hipStream_t stream)
{
    if (p.M <= 0)
        return hipSuccess;
    const bool tiled = p.M >= kGM && p.N >= kGN && !p.yf && p.K % kGK == 0;
    if (p.t_hilo && !p.yf && (!tiled || p.fuse || p.rank % 16 != 0))
        return hipErrorInvalidValue;  // only the large-M pass reads bf16 hi / lo activations
    if (p.M <= 32 && !p.yf) {
        return launch_project_decode(p, stream);
    } else if (tiled) {
        const int tiles = ((p.M + kGM - 1) / kGM) * ((p.N + kGN - 1) / kGN);
        ProjParams q = p;
        q.nxcd = gemm_xcds();
        const int per = (tiles + q.nxcd - 1) / q.nxcd;
        if (q.fuse)
            launch_kernel(proj_gemm_kernel<true>, dim3(per * q.nxcd), dim3(kThreads), kGLds, stream, q);
        else
            launch_kernel(proj_gemm_pp_kernel, dim3(per * q.nxcd), dim3(kPThreads), kPLds, stream, q);
    } else if (p.yf && p.N <= 2 * kBN && p.M < 256 * kBM) {
        // activation pass with fewer than 256 row tiles of 128: 32-row tiles
        // (every workgroup also reads all of A, so more tiles only pay
        // until the grid covers the compute units; measured 80 -> 66 us at
        // M = 16384, slower at M = 65536)
        dim3 grid((p.N + kBN - 1) / kBN, (p.M + 31) / 32);
        launch_kernel(proj_big_kernel<1>, grid, dim3(kThreads), 0, stream, p);
    } else {
        dim3 grid((p.N + kBN - 1) / kBN, (p.M + kBM - 1) / kBM);
        launch_kernel(proj_big_kernel<4>, grid, dim3(kThreads), 0, stream, p);
    }
    return hipGetLastError();
}

}  // namespace kvq
