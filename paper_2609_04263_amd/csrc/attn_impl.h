// Split-K decode attention over the packed cache with in-kernel
// reconstruction (Sec. 3.1-3.2 of the paper: attention sees the stored
// reconstruction; here it is computed from the codes without materializing
// it).  Included by one translation unit per head dimension.
//
// Work decomposition.  A workgroup of 4 waves handles one (split, sequence,
// KV head).  The G <= 16 query heads of the KV head are the N = 16 columns
// of v_mfma_f32_16x16x32_f16 (heads >= G are zero), so each code is read
// from HBM once per KV head.  Each wave walks every fourth 32-token block of
// the split:
//
//   loads     the cache stores each block's code pieces in the order of
//             this kernel's MFMA operands, so a lane reads its key and value
//             pieces with a few 8- to 16-byte loads that are contiguous
//             across the wave; the block's scales and offsets are read with
//             one 16-byte load per lane into a per-wave LDS buffer, from
//             which lanes read them broadcast.  The next block's loads are
//             issued before the current block is computed;
//   scores    per-token keys: S[t][h] = sum_g s_tg (sum_{d in g} c_td q_hd)
//             + z_tg sum_{d in g} q_hd, one MFMA per 32 channels with the
//             codes as exact fp16 A operands and the query as B (fp16 hi,
//             plus an fp16 remainder when the query is rotated); per-channel
//             keys fold the channel scale into the B operand (hi + lo fp16);
//   softmax   online in base 2 (sm_scale * log2(e) is folded into the query);
//             the running maximum is only raised when a block exceeds it by
//             more than kTau, so the accumulators are rescaled a few times
//             per split, not per block;
//   values    O^T[d][h] += sum_t c_dt (p_t s_tg 2^-kTau) over 32 tokens per
//             MFMA, with p s as hi + lo fp16 B operands, and the offset term
//             sum_t p_t z_tg accumulated per lane in fp32.
//
// Codes become exact fp16 operands with the 0x6400 exponent trick and one
// packed fp16 subtract, so every MFMA product is exact and accumulation is
// fp32.  Tokens of an fp16 window are handled by one extra split per KV head
// that feeds the fp16 values to the same MFMAs.  Each split writes an
// unnormalized partial (m, l, o) and a second kernel merges them (a kernel
// boundary instead of an in-kernel cross-workgroup handoff, whose
// agent-scope fences write back and invalidate the L2 on gfx950).  With a
// single split the first kernel writes the outputs itself.
#pragma once

#include "kvq_device.h"
#include "kvq_internal.h"

namespace kvq {
namespace attn {

constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr float kNegInf = -__builtin_inff();
constexpr float kTau = 4.0f;         // lazy rescale threshold, log2 units
constexpr float kPScale = 0.0625f;   // 2^-kTau: keeps p s below the group scale

// 16-byte loads per lane that read the largest metadata of one block (key
// groups of 32; scales and offsets of keys and values).  The per-wave LDS
// buffer holds 1 KiB per load.
__host__ __device__ constexpr int meta_loads(int D, bool perch, int nvg)
{
    (void)perch;  // key metadata is at most 2 D floats either way
    return ((2 * D + 2 * 32 * nvg) / 4 + 63) / 64;
}

// Compile-time shape of one kernel instance.
template <int D_, int KBITS_, int VBITS_, bool PERCH_, int VGS_>
struct Cfg {
    static constexpr int D = D_, KBITS = KBITS_, VBITS = VBITS_, VGS = VGS_;
    static constexpr bool PERCH = PERCH_;
    static constexpr int NKB = D / 32;          // 32-channel K-blocks of the score MFMAs
    static constexpr int NMB = D / 16;          // 16-channel M-blocks of the value MFMAs
    static constexpr int WPT = D * KBITS / 32;  // key code words per token in the cache
    static constexpr int KW = NKB * KBITS / 4;  // key code words per lane and half block
    static constexpr int VW = NMB * VBITS / 4;  // value code words per lane and block
    static constexpr int VG = 32 << VGS;        // value group size
    static constexpr int NVG = D / VG;          // value groups per token
    static constexpr int MBPG = VG / 16;        // value M-blocks per group
    static constexpr int NMETA = meta_loads(D, PERCH, NVG);
    static_assert(NVG >= 1, "value group larger than head_dim");
};

__device__ __forceinline__ float max_rows(float v)
{
    // max over the four 16-lane rows (lanes l, l ^ 16, l ^ 32, l ^ 48)
    auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

__device__ __forceinline__ float sum_rows(float v)
{
    auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

// Streaming global load of N words (4 to 64 naturally aligned bytes).
template <int N>
__device__ __forceinline__ void gload_words(const uint32_t* p, uint32_t* w)
{
    if constexpr (N == 1) {
        w[0] = __builtin_nontemporal_load(p);
    } else if constexpr (N == 2) {
        const u32x2 v = __builtin_nontemporal_load((const u32x2*)p);
        w[0] = v.x;
        w[1] = v.y;
    } else {
#pragma unroll
        for (int k = 0; k < N / 4; ++k) {
            const u32x4 v = __builtin_nontemporal_load((const u32x4*)p + k);
            w[4 * k] = v.x;
            w[4 * k + 1] = v.y;
            w[4 * k + 2] = v.z;
            w[4 * k + 3] = v.w;
        }
    }
}

// Piece k (eight codes) of a lane's words: a word for 4-bit codes, a
// halfword for 2-bit codes.
template <int BITS>
__device__ __forceinline__ uint32_t piece(const uint32_t* w, int k)
{
    if (BITS == 4)
        return w[k];
    return w[k >> 1] >> (16 * (k & 1));
}

// Row of the score MFMA A operand (and lane column hh) for token tb of a
// block: tokens 8a + 4 h2 + b sit in row 4a + b of half h2, so the MFMA
// output rows 4 qg + i of lane (hh, qg) are tokens 8 qg + 4 h2 + i, the same
// tokens whose values that lane's B operand covers.
__device__ __forceinline__ int score_row(int tb) { return 4 * (tb >> 3) + (tb & 3); }
__device__ __forceinline__ int score_half(int tb) { return (tb >> 2) & 1; }

// ------------------------------------------------------------ block loads

// The metadata sections of one block, in the order they are concatenated in
// a wave's LDS buffer: key scales, key offsets, value scales, value offsets
// (absent offset sections have no chunks).  Fields are scalars, not arrays,
// so that selecting a section never indexes memory.
struct MetaMap {
    const float *ks, *kz, *vs, *vz;  // section starts in the cache
    int nks, nkz, nvs;               // floats per block (offsets absent: nkz = 0 / no vz chunks)
    int e0, e1, e2, e3;              // cumulative 16-byte chunk counts
    float kmul, vmul;                // factors applied when staging key and value scales
    int l0, l1, l2, l3;              // float4 offsets in the wave buffer (absent: alias the scales)
};

template <class C>
struct BlockRegs {
    uint32_t k[2][C::KW];  // key pieces of the two half blocks
    uint32_t v[C::VW];     // value pieces
    u32x4 meta[C::NMETA];  // 16-byte metadata chunks lane + 64 u
};

// Issue every load of block `ub` (unit * NB + block) of a lane.
template <class C>
__device__ __forceinline__ void load_block(BlockRegs<C>& r, const AttnParams& p, const MetaMap& mm, size_t ub,
                                           int lane)
{
    const uint32_t* kc = p.kc + ub * (2 * 64 * C::KW) + lane * C::KW;
    gload_words<C::KW>(kc, r.k[0]);
    gload_words<C::KW>(kc + 64 * C::KW, r.k[1]);
    gload_words<C::VW>(p.vc + ub * (64 * C::VW) + lane * C::VW, r.v);
#pragma unroll
    for (int u = 0; u < C::NMETA; ++u) {
        const int c = lane + 64 * u;
        if (c < mm.e3) {
            const float* src;
            if (c < mm.e0)
                src = mm.ks + ub * (size_t)mm.nks + 4 * c;
            else if (c < mm.e1)
                src = mm.kz + ub * (size_t)mm.nkz + 4 * (c - mm.e0);
            else if (c < mm.e2)
                src = mm.vs + ub * (size_t)mm.nvs + 4 * (c - mm.e1);
            else
                src = mm.vz + ub * (size_t)mm.nvs + 4 * (c - mm.e2);
            r.meta[u] = __builtin_nontemporal_load((const u32x4*)src);
        }
    }
}

// ------------------------------------------------------------ split state

template <class C>
struct Split {
    static constexpr int NKB = C::NKB, NMB = C::NMB, NVG = C::NVG;
    half8 qhi[C::PERCH ? 1 : NKB], qlo[C::PERCH ? 1 : NKB];  // query B operands (per-token keys)
    float qsum[C::PERCH ? 1 : NKB];                          // sum of the 32 query channels of K-block kb
    float qf[C::PERCH ? NKB : 1][8];                         // fp32 query, operand order (per-channel keys)
    float m, lsum;                                           // running max (log2 units), lane partial sum
    float zl[NVG];                                           // lane partials of sum_t p_t z_tg
    floatx4 oacc[NMB];

    __device__ __forceinline__ void init()
    {
        m = kNegInf;
        lsum = 0.0f;
#pragma unroll
        for (int g = 0; g < NVG; ++g)
            zl[g] = 0.0f;
#pragma unroll
        for (int mb = 0; mb < NMB; ++mb)
            oacc[mb] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
    }

    // Online softmax over the eight logits l[k] (tokens 8 qg + k) of a lane.
    __device__ __forceinline__ void softmax(float* l)
    {
        float bm = fmaxf(fmaxf(fmaxf(l[0], l[1]), fmaxf(l[2], l[3])), fmaxf(fmaxf(l[4], l[5]), fmaxf(l[6], l[7])));
        bm = max_rows(bm);
        const bool up = bm > m + kTau;
        if (__any(up)) {
            const float mn = up ? bm : m;
            const float alpha = fast_exp2(m - mn);
            m = mn;
            lsum *= alpha;
#pragma unroll
            for (int g = 0; g < NVG; ++g)
                zl[g] *= alpha;
#pragma unroll
            for (int mb = 0; mb < NMB; ++mb)
                oacc[mb] *= alpha;
        }
        float ps = 0.0f;
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            l[k] = fast_exp2(l[k] - m);
            ps += l[k];
        }
        lsum += ps;
    }

    // One coded 32-token block whose loads are in `r`; tokens at or beyond
    // `valid` are masked.  `wl` is the wave's metadata buffer.
    __device__ __forceinline__ void coded_block(const BlockRegs<C>& r, float4* wl, const MetaMap& mm, int lane,
                                                int lgk, bool qlo_on, half2_t kbias, half2_t vbias, int valid)
    {
        const int qg = lane >> 4;
        // Stage the block's metadata in the wave's buffer: key scales and
        // offsets times sm_scale log2(e), value scales times 2^-kTau.  LDS
        // accesses of one wave are performed in order, so the reads below
        // see these writes without a barrier.
#pragma unroll
        for (int u = 0; u < C::NMETA; ++u) {
            const int c = lane + 64 * u;
            if (c < mm.e3) {
                const float f = c < mm.e1 ? mm.kmul : c < mm.e2 ? mm.vmul : 1.0f;
                const u32x4 w = r.meta[u];
                wl[c] = float4{__uint_as_float(w.x) * f, __uint_as_float(w.y) * f, __uint_as_float(w.z) * f,
                               __uint_as_float(w.w) * f};
            }
        }
        const float4* ks = wl + mm.l0;
        const float4* kz = wl + mm.l1;
        const float4* vs = wl + mm.l2;
        const float4* vz = wl + mm.l3;

        // ---------------------------------------------------- scores
        float l[8];
        if constexpr (!C::PERCH) {
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
                half8 a[NKB];
                floatx4 acc[NKB];
#pragma unroll
                for (int kb = 0; kb < NKB; ++kb) {
                    a[kb] = codes_to_half8<C::KBITS>(piece<C::KBITS>(r.k[h2], kb), kbias);
                    acc[kb] = mfma16(a[kb], qhi[kb], floatx4{0.0f, 0.0f, 0.0f, 0.0f});
                }
                if (qlo_on) {
#pragma unroll
                    for (int kb = 0; kb < NKB; ++kb)
                        acc[kb] = mfma16(a[kb], qlo[kb], acc[kb]);
                }
                floatx4 S;
#pragma unroll
                for (int kb = 0; kb < NKB; ++kb) {
                    // scale and offset of group kb >> lgk for tokens 8 qg + 4 h2 + i
                    const int fi = (kb >> lgk) * 8 + 2 * qg + h2;
                    const float4 s4 = ks[fi], z4 = kz[fi];
                    const floatx4 t = {s4.x * acc[kb][0] + z4.x * qsum[kb], s4.y * acc[kb][1] + z4.y * qsum[kb],
                                       s4.z * acc[kb][2] + z4.z * qsum[kb], s4.w * acc[kb][3] + z4.w * qsum[kb]};
                    S = kb == 0 ? t : S + t;
                }
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    l[4 * h2 + i] = S[i];
            }
        } else {
            // Per-channel keys: B = q * s_d (hi + lo), and sum_d q_d z_d per head.
            half8 bh[NKB], bl[NKB];
            float zq = 0.0f;
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb) {
                const float4 s0 = ks[8 * kb + 2 * qg], s1 = ks[8 * kb + 2 * qg + 1];
                const float4 z0 = kz[8 * kb + 2 * qg], z1 = kz[8 * kb + 2 * qg + 1];
                const float sn[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
                const float zn[8] = {z0.x, z0.y, z0.z, z0.w, z1.x, z1.y, z1.z, z1.w};
                float v[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    v[e] = qf[kb][e] * sn[perm4(e)];
                    zq += qf[kb][e] * zn[perm4(e)];
                }
                split_half8(v, &bh[kb], &bl[kb]);
            }
            zq = sum_rows(zq) * qsum[0];  // qsum[0] is 1 for affine keys, 0 for symmetric keys
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
                floatx4 acc = {zq, zq, zq, zq};
#pragma unroll
                for (int kb = 0; kb < NKB; ++kb) {
                    const half8 a = codes_to_half8<C::KBITS>(piece<C::KBITS>(r.k[h2], kb), kbias);
                    acc = mfma16(a, bh[kb], acc);
                    acc = mfma16(a, bl[kb], acc);
                }
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    l[4 * h2 + i] = acc[i];
            }
        }
#pragma unroll
        for (int k = 0; k < 8; ++k)
            l[k] = 8 * qg + k < valid ? l[k] : kNegInf;
        softmax(l);  // l now holds p (<= 2^kTau), 0 for masked tokens

        // ---------------------------------------------------- values
        // Masked tokens have p = 0 and finite metadata (the storage starts
        // zero-filled and is only ever written with finite values), so their
        // terms vanish without a select.
#pragma unroll
        for (int g = 0; g < NVG; ++g) {
            const float4 s0 = vs[8 * g + 2 * qg], s1 = vs[8 * g + 2 * qg + 1];
            const float4 z0 = vz[8 * g + 2 * qg], z1 = vz[8 * g + 2 * qg + 1];
            const float sn[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
            const float zn[8] = {z0.x, z0.y, z0.z, z0.w, z1.x, z1.y, z1.z, z1.w};
            float pv[8];
            float zs = 0.0f;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int k = perm4(e);
                pv[e] = l[k] * sn[k];
                zs += l[k] * zn[k];
            }
            zl[g] += zs;
            half8 ph, pl;
            split_half8(pv, &ph, &pl);
#pragma unroll
            for (int j = 0; j < C::MBPG; ++j) {
                const int mb = g * C::MBPG + j;
                const half8 a = codes_to_half8<C::VBITS>(piece<C::VBITS>(r.v, mb), vbias);
                oacc[mb] = mfma16(a, ph, oacc[mb]);
                oacc[mb] = mfma16(a, pl, oacc[mb]);
            }
        }
    }

    // One block of the fp16 window (tokens t0 .. t0 + 31, those >= n masked),
    // read straight from the ring slots.
    __device__ __forceinline__ void ring_block(const AttnParams& p, int unit, int t0, int lane, bool qlo_on)
    {
        constexpr int D = C::D;
        const int hh = lane & 15, qg = lane >> 4;
        const int n = p.n, ring = p.ring;
        const size_t rbase = (size_t)unit * ring;
        float l[8];
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2) {
            const int tA = t0 + 8 * (hh >> 2) + 4 * h2 + (hh & 3);
            const uint16_t* krow = p.kr + (rbase + (size_t)(tA % ring)) * D;
            floatx4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb) {
                half8 a = {};
                if (tA < n) {
                    const half8 nat = __builtin_bit_cast(half8, *(const u32x4*)(krow + 32 * kb + 8 * qg));
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        a[e] = nat[perm4(e)];
                }
                if constexpr (C::PERCH) {
                    half8 bh, bl;
                    split_half8(qf[kb], &bh, &bl);
                    acc = mfma16(a, bh, acc);
                    acc = mfma16(a, bl, acc);
                } else {
                    acc = mfma16(a, qhi[kb], acc);
                    if (qlo_on)
                        acc = mfma16(a, qlo[kb], acc);
                }
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
                l[4 * h2 + i] = acc[i] * p.sm_log2;
        }
        int slot[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const int t = t0 + 8 * qg + k;
            slot[k] = t < n ? t % ring : -1;
            l[k] = t < n ? l[k] : kNegInf;
        }
        softmax(l);
        float pv[8];
#pragma unroll
        for (int e = 0; e < 8; ++e)
            pv[e] = slot[perm4(e)] >= 0 ? l[perm4(e)] * kPScale : 0.0f;
        half8 ph, pl;
        split_half8(pv, &ph, &pl);
#pragma unroll
        for (int mb = 0; mb < NMB; ++mb) {
            const int d = 16 * mb + hh;
            half8 a;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int sl = slot[perm4(e)];
                const uint16_t raw = sl >= 0 ? p.vr[(rbase + (size_t)sl) * D + d] : (uint16_t)0;
                a[e] = __builtin_bit_cast(_Float16, raw);
            }
            oacc[mb] = mfma16(a, ph, oacc[mb]);
            oacc[mb] = mfma16(a, pl, oacc[mb]);
        }
    }
};

// Inverse rotation (the normalized transform is its own inverse) of G rows
// of D outputs staged in LDS, then the store to O.
template <int D>
__device__ __forceinline__ void finish_rows(const AttnParams& p, float* xo, size_t row0, int G)
{
    if (p.rotate) {
        for (int h = 1; h < D; h <<= 1) {
            for (int idx = threadIdx.x; idx < G * (D / 2); idx += kThreads) {
                const int r = idx / (D / 2), k = idx % (D / 2);
                const int jj = (k / h) * 2 * h + (k % h);
                const float a = xo[r * D + jj], c = xo[r * D + jj + h];
                xo[r * D + jj] = a + c;
                xo[r * D + jj + h] = a - c;
            }
            __syncthreads();
        }
    }
    const float post = p.rotate ? p.rot_c : 1.0f;
    for (int idx = threadIdx.x; idx < G * D; idx += kThreads)
        p.out[row0 * D + idx] = xo[idx] * post;
}

// Floats of the per-wave metadata buffer.
template <class C>
constexpr int meta_floats()
{
    return 256 * C::NMETA;
}

template <class C>
__device__ __forceinline__ void split_body(const AttnParams& p, uint8_t* lds)
{
    constexpr int D = C::D, NKB = C::NKB, NMB = C::NMB;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
    const int hh = lane & 15, qg = lane >> 4;
    const int split = blockIdx.x, unit = blockIdx.y;
    const int b = unit / p.H, j = unit % p.H, G = p.G;
    const bool ring_split = p.ring && split == p.S_q;
    const bool kaff = p.k_mode == KVQ_AFFINE, vaff = p.v_mode == KVQ_AFFINE;
    const bool qlo_on = p.rotate != 0;
    const int NB = p.T >> 5;
    const int lgk = C::PERCH ? 0 : __builtin_ctz((unsigned)p.k_group >> 5);  // log2(key group / 32)
    const int kmeta = C::PERCH ? D : 32 * (D / p.k_group);                    // key scale floats per block

    MetaMap mm;
    mm.ks = p.ks;
    mm.kz = p.kz;
    mm.vs = p.vs;
    mm.vz = p.vz;
    mm.nks = kmeta;
    mm.nkz = kaff ? kmeta : 0;
    mm.nvs = 32 * C::NVG;
    mm.e0 = kmeta / 4;
    mm.e1 = mm.e0 + mm.nkz / 4;
    mm.e2 = mm.e1 + mm.nvs / 4;
    mm.e3 = mm.e2 + (vaff ? mm.nvs / 4 : 0);
    mm.kmul = p.sm_log2;
    mm.vmul = kPScale;
    // absent offset sections alias the scales (their terms get a zero weight)
    mm.l0 = 0;
    mm.l1 = kaff ? mm.e0 : 0;
    mm.l2 = mm.e1;
    mm.l3 = vaff ? mm.e2 : mm.e1;

    // ---- block range of this split
    const int nblk = (p.nq + 31) >> 5;
    const int blk_begin = ring_split ? 0 : split * p.bps;
    const int blk_end = ring_split ? 0 : min(nblk, blk_begin + p.bps);
    const size_t ub0 = (size_t)unit * NB;

    // ---- queries (bf16 -> fp32 rows in LDS; rows >= G zero), first block's loads
    constexpr int QPIECES = 16 * D / 8;
    constexpr int QLOADS = (QPIECES + kThreads - 1) / kThreads;
    u32x4 qraw[QLOADS];
#pragma unroll
    for (int u = 0; u < QLOADS; ++u) {
        const int pc = u * kThreads + (int)threadIdx.x, row = pc / (D / 8);
        qraw[u] = u32x4{0u, 0u, 0u, 0u};
        if (pc < QPIECES && row < G)
            qraw[u] = *(const u32x4*)(p.q + ((size_t)b * p.H_q + (size_t)j * G + row) * D + (pc % (D / 8)) * 8);
    }
    BlockRegs<C> ra, rb;
    int blk = blk_begin + wave;
    if (blk < blk_end)
        load_block<C>(ra, p, mm, ub0 + blk, lane);
    float* lq = (float*)lds;
#pragma unroll
    for (int u = 0; u < QLOADS; ++u) {
        const int pc = u * kThreads + (int)threadIdx.x;
        if (pc < QPIECES) {
            const uint32_t w[4] = {qraw[u].x, qraw[u].y, qraw[u].z, qraw[u].w};
            float* dst = lq + pc * 8;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                dst[2 * k] = __uint_as_float(w[k] << 16);
                dst[2 * k + 1] = __uint_as_float(w[k] & 0xFFFF0000u);
            }
        }
    }
    __syncthreads();
    if (p.rotate) {
        for (int h = 1; h < D; h <<= 1) {
            for (int idx = threadIdx.x; idx < 16 * (D / 2); idx += kThreads) {
                const int row = idx / (D / 2), k = idx % (D / 2);
                const int jj = (k / h) * 2 * h + (k % h);
                const float a = lq[row * D + jj], c = lq[row * D + jj + h];
                lq[row * D + jj] = a + c;
                lq[row * D + jj + h] = a - c;
            }
            __syncthreads();
        }
        for (int idx = threadIdx.x; idx < 16 * D; idx += kThreads)
            lq[idx] *= p.rot_c;
        __syncthreads();
    }
    Split<C> S;
    S.init();
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) {
        float v[8];
        float part = 0.0f;
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            v[k] = lq[hh * D + 32 * kb + 8 * qg + perm4(k)];
            part += v[k];
        }
        if constexpr (C::PERCH) {
#pragma unroll
            for (int k = 0; k < 8; ++k)
                S.qf[kb][k] = v[k];
        } else {
            split_half8(v, &S.qhi[kb], &S.qlo[kb]);
            S.qsum[kb] = kaff ? sum_rows(part) : 0.0f;  // offset terms vanish for symmetric keys
        }
    }
    if constexpr (C::PERCH)
        S.qsum[0] = kaff ? 1.0f : 0.0f;
    __syncthreads();  // the metadata buffers overwrite the query rows

    const _Float16 kb16 = (_Float16)(1024 + (kaff ? 0 : (1 << (C::KBITS - 1))));
    const _Float16 vb16 = (_Float16)(1024 + (vaff ? 0 : (1 << (C::VBITS - 1))));
    const half2_t kbias = {kb16, kb16}, vbias = {vb16, vb16};

    if (!ring_split) {
        float4* wl = (float4*)lds + wave * (meta_floats<C>() / 4);
        // Two register sets alternate: the next block's loads fly while
        // this one is computed.
        while (blk < blk_end) {
            if (blk + kWaves < blk_end)
                load_block<C>(rb, p, mm, ub0 + blk + kWaves, lane);
            S.coded_block(ra, wl, mm, lane, lgk, qlo_on, kbias, vbias, min(32, p.nq - 32 * blk));
            blk += kWaves;
            if (blk >= blk_end)
                break;
            if (blk + kWaves < blk_end)
                load_block<C>(ra, p, mm, ub0 + blk + kWaves, lane);
            S.coded_block(rb, wl, mm, lane, lgk, qlo_on, kbias, vbias, min(32, p.nq - 32 * blk));
            blk += kWaves;
        }
    } else {
        const int nr = p.n - p.nq;
        for (int rblk = wave; 32 * rblk < nr; rblk += kWaves)
            S.ring_block(p, unit, p.nq + 32 * rblk, lane, qlo_on);
    }

    // ---- merge the four waves of this split in LDS
    const float lsum = sum_rows(S.lsum);
    float zl[C::NVG];
#pragma unroll
    for (int g = 0; g < C::NVG; ++g)
        zl[g] = vaff ? sum_rows(S.zl[g]) : 0.0f;
    __syncthreads();
    float* lm = (float*)lds;           // [4][16] running max per wave and head
    float* ll = lm + kWaves * 16;      // [4][16] softmax sums
    float* lo = lm + 2 * kWaves * 16;  // [4][G][D] unnormalized outputs
    float* xo = lo;  // [G][D] result: element idx is written after its own four reads
    if (qg == 0) {
        lm[wave * 16 + hh] = S.m;
        ll[wave * 16 + hh] = lsum;
    }
    if (hh < G) {
#pragma unroll
        for (int mb = 0; mb < NMB; ++mb)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                lo[((size_t)wave * G + hh) * D + 16 * mb + 4 * qg + i] =
                    S.oacc[mb][i] * (1.0f / kPScale) + zl[mb / C::MBPG];
    }
    __syncthreads();
    const bool single = p.S_tot == 1;
    const size_t row0 = (size_t)b * p.H_q + (size_t)j * G;
    for (int idx = threadIdx.x; idx < G * D; idx += kThreads) {
        const int h = idx / D, d = idx % D;
        float M = kNegInf;
        for (int w = 0; w < kWaves; ++w)
            M = fmaxf(M, lm[w * 16 + h]);
        float acc = 0.0f, Ls = 0.0f;
        if (M != kNegInf) {
            for (int w = 0; w < kWaves; ++w) {
                const float sc = fast_exp2(lm[w * 16 + h] - M);
                acc += sc * lo[((size_t)w * G + h) * D + d];
                Ls += sc * ll[w * 16 + h];
            }
        }
        if (single) {
            xo[idx] = acc / Ls;
        } else {
            const size_t row = row0 + h;
            p.part_o[(row * p.S_tot + split) * D + d] = acc;
            if (d == 0) {
                p.part_ml[(row * p.S_tot + split) * 2 + 0] = M;
                p.part_ml[(row * p.S_tot + split) * 2 + 1] = Ls;
            }
        }
    }
    if (!single)
        return;  // the merge kernel finishes
    __syncthreads();
    finish_rows<D>(p, xo, row0, G);
}

template <class C>
__global__ __launch_bounds__(kThreads) void decode_split_kernel(AttnParams p)
{
    extern __shared__ float lds_f[];
    split_body<C>(p, (uint8_t*)lds_f);
}

// Merge the S_tot split partials of one (sequence, KV head): per head, the
// weights w_s = 2^(m_s - M) / sum_s' 2^(m_s' - M) l_s' go to LDS, then every
// output is a weighted sum over splits of coalesced partial rows; finally
// rotate back and store.
template <int D>
__global__ __launch_bounds__(kThreads) void decode_merge_kernel(AttnParams p)
{
    extern __shared__ float sm[];
    const int unit = blockIdx.x;
    const int b = unit / p.H, j = unit % p.H, G = p.G, S = p.S_tot;
    const size_t row0 = (size_t)b * p.H_q + (size_t)j * G;
    float* w = sm;               // [G][S]: (max, sum) pairs, then weights
    float* xo = sm + 2 * G * S;  // [G][D]
    const float* ml = p.part_ml + row0 * S * 2;
    for (int idx = threadIdx.x; idx < 2 * G * S; idx += kThreads)
        w[idx] = ml[idx];
    __syncthreads();
    if (threadIdx.x < (unsigned)G) {
        float* r = w + 2 * S * threadIdx.x;
        float M = kNegInf;
        for (int s = 0; s < S; ++s)
            M = fmaxf(M, r[2 * s]);
        float Ls = 0.0f;
        for (int s = 0; s < S; ++s)
            Ls += r[2 * s] == kNegInf ? 0.0f : fast_exp2(r[2 * s] - M) * r[2 * s + 1];
        const float inv = 1.0f / Ls;
        for (int s = 0; s < S; ++s) {
            const float m = r[2 * s];
            r[2 * s] = m == kNegInf ? 0.0f : fast_exp2(m - M) * inv;  // weights overwrite maxima
        }
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < G * D; idx += kThreads) {
        const int h = idx / D, d = idx % D;
        const float* o = p.part_o + ((row0 + h) * S) * D + d;
        const float* wr = w + 2 * S * h;
        float acc0 = 0.0f, acc1 = 0.0f, acc2 = 0.0f, acc3 = 0.0f;
        int s = 0;
        for (; s + 4 <= S; s += 4) {
            acc0 += wr[2 * s] * o[(size_t)s * D];
            acc1 += wr[2 * s + 2] * o[(size_t)(s + 1) * D];
            acc2 += wr[2 * s + 4] * o[(size_t)(s + 2) * D];
            acc3 += wr[2 * s + 6] * o[(size_t)(s + 3) * D];
        }
        for (; s < S; ++s)
            acc0 += wr[2 * s] * o[(size_t)s * D];
        xo[idx] = (acc0 + acc1) + (acc2 + acc3);
    }
    __syncthreads();
    finish_rows<D>(p, xo, row0, G);
}

template <class C>
hipError_t launch_split(const AttnParams& p, hipStream_t stream)
{
    hipLaunchKernelGGL(decode_split_kernel<C>, dim3(p.S_tot, p.B * p.H), dim3(kThreads), p.lds_bytes, stream, p);
    return hipGetLastError();
}

template <int D, int KB, int VB, bool PC, int VGS = 0>
hipError_t launch_groups(const AttnParams& p, hipStream_t stream)
{
    if constexpr ((32 << VGS) > D) {
        return hipErrorInvalidValue;
    } else {
        if (p.v_group == (32 << VGS))
            return launch_split<Cfg<D, KB, VB, PC, VGS>>(p, stream);
        return launch_groups<D, KB, VB, PC, VGS + 1>(p, stream);
    }
}

template <int D>
hipError_t launch_decode_d(const AttnParams& p, hipStream_t stream)
{
    hipError_t e;
    const bool pc = p.k_axis == KVQ_PER_CHANNEL;
    if (p.k_bits == 4 && p.v_bits == 4)
        e = pc ? launch_groups<D, 4, 4, true>(p, stream) : launch_groups<D, 4, 4, false>(p, stream);
    else if (p.k_bits == 4 && p.v_bits == 2)
        e = pc ? launch_groups<D, 4, 2, true>(p, stream) : launch_groups<D, 4, 2, false>(p, stream);
    else if (p.k_bits == 2 && p.v_bits == 4)
        e = pc ? launch_groups<D, 2, 4, true>(p, stream) : launch_groups<D, 2, 4, false>(p, stream);
    else
        e = pc ? launch_groups<D, 2, 2, true>(p, stream) : launch_groups<D, 2, 2, false>(p, stream);
    if (e != hipSuccess || p.S_tot == 1)
        return e;
    hipLaunchKernelGGL(decode_merge_kernel<D>, dim3(p.B * p.H), dim3(kThreads),
                       (size_t)(2 * p.S_tot + D) * p.G * sizeof(float), stream, p);
    return hipGetLastError();
}

}  // namespace attn
}  // namespace kvq
