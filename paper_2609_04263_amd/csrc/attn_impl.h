// Split-K decode attention over the packed cache with in-kernel
// reconstruction (Sec. 3.1-3.2 of the paper: attention sees the stored
// reconstruction; here it is computed from the codes without materializing
// it).  The split kernels are instantiated by attn_part.hip, once per (head
// size, metadata width, key axis) family; the merge kernels by attn.hip.
//
// Work decomposition.  A workgroup of W waves (waves_for: 4, or at
// head_dim 128 a whole compute unit of 8 or 12) handles one (split,
// sequence, KV head).  The MFMA v_mfma_f32_16x16x32_f16 has 16 columns; the G <= 16
// query heads of the KV head take G of them, so every code is read from HBM
// once per KV head.  When the value groups of a token times G fit in the 16
// columns, each value group gets its own copy of the G head columns
// (column r G + h: head h, value group r) and one pass of the value-side
// arithmetic serves every group; otherwise groups are taken one per pass.
// The split's 32-token blocks are dealt to the waves round robin, in whole
// rounds of W blocks (a wave whose block lies past the end skips its
// arithmetic but keeps the loop shape, so the prefetch wait stays exact):
//
//   loads     the cache stores each block's code pieces in the order of
//             this kernel's MFMA operands, so a lane reads its key and value
//             pieces with a few 8- to 16-byte loads that are contiguous
//             across the wave; the block's scales and offsets pass through a
//             per-wave LDS buffer, from which lanes read them broadcast.  The
//             next block's loads are issued before the current one is
//             computed, and every lane issues the same loads, so the wait
//             before a block only covers that block;
//   codes     a piece of eight codes becomes an exact fp16 MFMA operand
//             A = B0 + c with two bit operations per pair (the exponent of
//             B0 = 16 for 4-bit, 4 for 2-bit codes gives the code bits unit
//             weight); the bias is folded into a staged offset
//             z' = z - B0 s (z = -2^(b-1) s for symmetric codes), so that
//             every reconstructed element is A s + z';
//   scores    per-token keys: S[t][h] = sum_g s_tg (sum_{d in g} A_td q_hd)
//             + z'_tg sum_{d in g} q_hd, one MFMA per 32 channels with the
//             query as B (fp16 hi, plus an fp16 remainder when the query is
//             rotated); per-channel keys fold the channel scale into the B
//             operand (hi + lo fp16) and sum_d z'_d q_d into the accumulator;
//   softmax   online in base 2 (scales and offsets carry sm_scale log2(e));
//             the running maximum is only raised when a block exceeds it by
//             more than kTau, so the accumulators are rescaled a few times
//             per split, not per block;
//   values    O^T[d][h] += sum_t A_dt (p_t s_tg 2^-kTau) over 32 tokens per
//             MFMA, with p s as hi + lo fp16 B operands, plus the offset term
//             sum_t p_t z'_tg accumulated per lane in fp32.
//
// Every MFMA product is exact (fp16 x fp16 in fp32) and accumulation is
// fp32.  Tokens of an fp16 window (a sink prefix, or the unflushed tail) are
// 32-token blocks too: after its coded blocks every split takes a share of
// them, round robin over splits and waves, reads the fp16 keys as MFMA
// operands directly and the values through a transposed copy in the wave's
// LDS region.  The waves of a workgroup then merge their states in LDS.
// Each split writes an unnormalized partial (m, l, o) and a second kernel
// merges them (a kernel boundary instead of an in-kernel cross-workgroup
// handoff, whose agent-scope fences write back and invalidate the L2 on
// gfx950).  With a single split the first kernel writes the outputs itself.
#pragma once

#include <atomic>

#include "kvq_device.h"
#include "kvq_internal.h"

namespace kvq {
namespace attn {

constexpr float kNegInf = -__builtin_inff();
constexpr float kTau = 4.0f;        // lazy rescale threshold, log2 units
constexpr float kPScale = 0.0625f;  // 2^-kTau: keeps p s below the group scale

// 16-byte metadata chunk pairs (scale, offset) per lane that cover the
// largest metadata of one block: key groups of 32 (or per-channel keys, D
// floats each) and D / v_group value groups, 32 tokens each.  The per-wave
// LDS buffer holds 2 KiB per pair.
__host__ __device__ constexpr int meta_pairs(int D, int nvg)
{
    return ((D + 32 * nvg) / 4 + 63) / 64;
}

// Waves per split workgroup.  At head_dim 128 one workgroup fills a compute
// unit: eight waves (two per SIMD), or twelve (three per SIMD) for 2-bit
// per-channel keys with 2-bit values, whose state fits 168 registers.  With
// as many (sequence, KV head) units as compute units, one split per unit
// then covers the device and no merge is needed.  The other head sizes use
// four.
__host__ __device__ constexpr int waves_for(int D, bool perch, int kbits, int vbits)
{
    return D != 128 ? 4 : (perch && kbits == 2 && vbits == 2) ? 12 : 8;
}

// Compile-time shape of one kernel instance.
template <int D_, int KBITS_, int VBITS_, bool PERCH_, int VGS_, bool M16_ = false>
struct Cfg {
    static constexpr int WAVES = waves_for(D_, PERCH_, KBITS_, VBITS_), THREADS = 64 * WAVES;
    static constexpr int D = D_, KBITS = KBITS_, VBITS = VBITS_, VGS = VGS_;
    static constexpr bool PERCH = PERCH_;
    static constexpr bool M16 = M16_;           // fp16 scales and offsets
    static constexpr int NKB = D / 32;          // 32-channel K-blocks of the score MFMAs
    static constexpr int NMB = D / 16;          // 16-channel M-blocks of the value MFMAs
    static constexpr int KW = NKB * KBITS / 4;  // key code words per lane and half block
    static constexpr int VW = NMB * VBITS / 4;  // value code words per lane and block
    static constexpr int VG = 32 << VGS;        // value group size
    static constexpr int NVG = D / VG;          // value groups per token
    static constexpr int MBPG = VG / 16;        // value M-blocks per group
    static constexpr int NPAIR = meta_pairs(D, NVG);
    // Register sets of the block pipeline: a wave computes one block while
    // the loads of the next NBUF - 1 are in flight.  Wider heads run fewer
    // waves per SIMD, so each wave keeps more bytes in flight.
    static constexpr int NBUF = KBITS == 8 ? 2 : D == 64 ? 2 : 3;
    static_assert(NVG >= 1, "value group larger than head_dim");
};

// Per-channel keys (KIVI): the score operand q_hd s_d changes with every
// 32-token block.  Its G D products are formed once per block, eight per
// (head, channel octet) item spread over the wave's lanes, and exchanged
// through the wave's LDS slots into the MFMA operand layout.
struct PerchCtx {
    const float* qw;  // LDS [G][D] fp32 queries (rotated when the format rotates)
    uint8_t* slots;   // this wave's LDS slots: item i = (head i / (D/8), octet i % (D/8)) at 32 i, hi then lo
    int items;        // G D / 8
    int rbase;        // byte offset of this lane's operand slot at K-block 0 (+128 per K-block)
    int zsrc, zj;     // lane (x4) and writer iteration holding this column's key offset term
    int hn;           // head of this lane's column (below G)
};

// Split kernel LDS, in bytes from its start: the rotated query rows
// ([16][D] fp32, rotating formats); for per-channel keys the fp32 query rows
// [G][D]; then one region per wave.  During the coded blocks a wave's region
// holds its metadata buffer (npair 2 KiB) and, for per-channel keys, its
// operand slots (G D 4 bytes); the fp16 blocks come after the coded ones and
// reuse it for a transposed value block ([D][kVtPitch] halves).  The final
// merge of the waves reuses everything from the start.
constexpr int kVtPitch = 40;  // halves per channel row of a transposed fp16 value block

__host__ __device__ constexpr size_t lds_qw(int D)
{
    return (size_t)16 * D * 4;
}

__host__ __device__ constexpr size_t lds_waves(int D, bool perch, int G)
{
    return lds_qw(D) + (perch ? (size_t)G * D * 4 : 0);
}

__host__ __device__ constexpr size_t lds_per_wave(int D, int npair, bool perch, int G, bool fp16)
{
    const size_t coded = (size_t)npair * 2048 + (perch ? (size_t)G * D * 4 : 0);
    const size_t vt = fp16 ? (size_t)D * kVtPitch * 2 : 0;
    return ((coded > vt ? coded : vt) + 15) / 16 * 16;
}

// Sum over aligned groups of NL lanes (NL = 8, 16 or 32), every lane of a
// group receiving the group's sum (DPP quad xors, half-row and row mirrors,
// then a swap of adjacent rows).
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float x)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}

template <int NL>
__device__ __forceinline__ float group_sum(float v)
{
    v += dpp_f32<0xB1>(v);   // quad_perm [1, 0, 3, 2]
    v += dpp_f32<0x4E>(v);   // quad_perm [2, 3, 0, 1]
    v += dpp_f32<0x141>(v);  // row_half_mirror
    if constexpr (NL >= 16)
        v += dpp_f32<0x140>(v);  // row_mirror
    if constexpr (NL >= 32) {
        auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
        v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    }
    return v;
}

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

// ------------------------------------------------------------ code operands

// Operand bias B0 of a code width: A = B0 + c exactly in binary16.  The
// operand's rounding error on the other MFMA side (q, or p s) is multiplied
// by A and cancels only against the exact offset term, so |A| is kept small:
// 8-bit codes are centred (c - 128) rather than biased by 1024.
template <int BITS>
__device__ constexpr float code_bias()
{
    return BITS == 8 ? -128.0f : BITS == 4 ? 16.0f : 4.0f;
}

typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

// Bit constants of the conversion, kept in registers (a VOP3 operation
// cannot take two literals on gfx950); mag16 is the exponent pair of 16 for
// the 2-bit conversion with mixed biases.
struct CodeBits {
    uint32_t mask, magic, mag16;
};

template <int BITS>
__device__ __forceinline__ CodeBits code_bits()
{
    // 8-bit: code at mantissa bits 0..7 under exponent 2^10 (1024 + c),
    //        then -1152 added as a packed pair (mask holds binary16 -1152);
    // 4-bit: code at mantissa bits 6..9 under exponent 2^4 (16 + c);
    // 2-bit: code at mantissa bits 8..9 under exponent 2^2 (4 + c).
    uint32_t mask = BITS == 8 ? 0xE480E480u : BITS == 4 ? 0x03C003C0u : 0x03000300u;
    uint32_t magic = BITS == 8 ? 0x64006400u : BITS == 4 ? 0x4C004C00u : 0x44004400u;
    uint32_t mag16 = 0x4C004C00u;
    // opaque to constant folding, so they stay in registers
    asm volatile("" : "+v"(mask), "+v"(magic));
    if constexpr (BITS == 2)
        asm volatile("" : "+v"(mag16));
    return CodeBits{mask, magic, mag16};
}

// Piece k (eight codes, code j at bits BITS j) of a lane's words -> the
// MFMA operand (B0 + c_j, B0 + c_{j+4}) in dword j, i.e. element e holds
// code perm4(e).  MIXED (2-bit codes): dwords 0 and 2 take their codes at
// mantissa bits 6..7 under 2^4 (B = 16), dwords 1 and 3 at bits 8..9 under
// 2^2 (B = 4), so that one shift serves two dwords: seven operations per
// piece instead of nine.  The extra 12 of dwords 0 and 2 is folded into the
// staged offsets with the rest of B.
template <int BITS>
__host__ __device__ constexpr float mixed_extra_bias(int j)
{
    return BITS == 2 && (j & 1) == 0 ? 12.0f : 0.0f;
}

template <int BITS, bool MIXED = false>
__device__ __forceinline__ half8 biased_codes(const uint32_t* w, int k, const CodeBits& cb)
{
    u32x4 v;
    if constexpr (BITS == 8) {
        // a piece is two words (codes 0..3, codes 4..7): byte j of each to
        // bytes 0 and 2 of dword j, then (1024 + c) - 1152 = c - 128, exact
        const uint32_t lo = w[2 * k], hi = w[2 * k + 1];
        const f16x2 nb = __builtin_bit_cast(f16x2, cb.mask);
        auto centred = [&](uint32_t sel) {
            const uint32_t x = __builtin_amdgcn_perm(hi, lo, sel) | cb.magic;
            return __builtin_bit_cast(uint32_t, __builtin_bit_cast(f16x2, x) + nb);
        };
        v.x = centred(0x0c040c00u);
        v.y = centred(0x0c050c01u);
        v.z = centred(0x0c060c02u);
        v.w = centred(0x0c070c03u);
    } else if constexpr (BITS == 4) {
        const uint32_t x = w[k];
        v.x = ((x << 6) & cb.mask) | cb.magic;
        v.y = ((x << 2) & cb.mask) | cb.magic;
        v.z = ((x >> 2) & cb.mask) | cb.magic;
        v.w = ((x >> 6) & cb.mask) | cb.magic;
    } else if constexpr (MIXED) {
        // codes j, j + 4 at bits 2j, 16 + 2j of z; z << 6 puts codes 0 and 1
        // at bits 6..7 and 8..9, z << 2 codes 2 and 3
        const uint32_t z = __builtin_amdgcn_perm(0u, w[k >> 1], (k & 1) ? 0x0c030c02u : 0x0c010c00u);
        const uint32_t t1 = z << 6, t2 = z << 2;
        v.x = (t1 & 0x00C000C0u) | cb.mag16;
        v.y = (t1 & cb.mask) | cb.magic;
        v.z = (t2 & 0x00C000C0u) | cb.mag16;
        v.w = (t2 & cb.mask) | cb.magic;
    } else {
        // bytes (c0..c3) and (c4..c7) of the piece to bytes 0 and 2
        const uint32_t z = __builtin_amdgcn_perm(0u, w[k >> 1], (k & 1) ? 0x0c030c02u : 0x0c010c00u);
        v.x = ((z << 8) & cb.mask) | cb.magic;
        v.y = ((z << 6) & cb.mask) | cb.magic;
        v.z = ((z << 4) & cb.mask) | cb.magic;
        v.w = ((z << 2) & cb.mask) | cb.magic;
    }
    return __builtin_bit_cast(half8, v);
}

// fp32 -> fp16 hi + lo: hi is v with its binary32 mantissa cut to binary16
// width (so v - hi is exact in binary32) and lo is that remainder, both
// converted to nearest.  An MFMA pair over (hi, lo) carries about 22
// significant bits; where lo falls below the binary16 normal range its
// rounding error (at most 2^-25 absolute) is unbiased, which matters because
// the value-side sum of biased codes times p s cancels against the offset
// term.
__device__ __forceinline__ void split_pairs(const float* v, half8* hi, half8* lo)
{
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const float a = __uint_as_float(__float_as_uint(v[e]) & 0xFFFFE000u);
        (*hi)[e] = (_Float16)a;
        (*lo)[e] = (_Float16)(v[e] - a);
    }
}

// ------------------------------------------------------------ block loads

// Metadata of one block: nk key floats (scales; offsets alike) and nv value
// floats, taken as nk / 4 + nv / 4 chunk pairs (scale chunk, offset chunk).
// In the wave's LDS buffer: key scales, key offsets z', value scales, value
// offsets z' (float4 offsets in coded_block).
struct MetaMap {
    const uint8_t* ks;   // key scales; the other sections are at byte offsets from it
    long dkz, dvs, dvz;  // kz - ks (0 for symmetric keys), vs - ks, vz - ks (vs - ks when symmetric)
    int esz;             // bytes per scale or offset: 4 (fp32) or 2 (fp16, Cfg::M16)
    int nk, nv;          // floats per block
    int kp, np;          // key chunk pairs, all chunk pairs
    float kmul, vmul;    // sm_scale log2(e) for keys, 2^-kTau for value scales
    float kz0, kzs;      // key z' = kz0 z + kzs s: z - B0 s (affine) or -(2^(b-1) + B0) s (symmetric)
    float vz0, vzs;      // value z' alike
};

template <class C>
struct BlockRegs {
    uint32_t k[2][C::KW];              // key pieces of the two half blocks
    uint32_t v[C::VW];                 // value pieces
    u32x4 ms[C::NPAIR], mz[C::NPAIR];  // metadata chunk pairs lane + 64 u
};

// A lane's load addresses for block 0 of its (sequence, KV head) unit; block
// b is at a fixed stride from them.  The metadata chunk a lane loads (a key
// or a value chunk, fixed per lane) is selected once, so the loads of a block
// need no per-block selects or branches.
template <class C>
struct LoadMap {
    const uint32_t* kc;              // key code words of this lane
    const uint32_t* vc;              // value code words of this lane
    const uint8_t* ms[C::NPAIR];     // scale chunk of pair u
    long dz[C::NPAIR];               // offset chunk - scale chunk (bytes)
    uint32_t mstride[C::NPAIR];      // metadata bytes per block of the chunk's section
};

template <class C>
__device__ __forceinline__ LoadMap<C> load_map(const AttnParams& p, const MetaMap& mm, size_t ub0, int lane)
{
    LoadMap<C> L;
    L.kc = p.kc + ub0 * (2 * 64 * C::KW) + lane * C::KW;
    L.vc = p.vc + ub0 * (64 * C::VW) + lane * C::VW;
#pragma unroll
    for (int u = 0; u < C::NPAIR; ++u) {
        // every lane issues the same loads whatever the format: surplus
        // lanes re-read the last chunk pair, so the loads in flight are fixed
        const int c = min(lane + 64 * u, mm.np - 1);
        const bool key = c < mm.kp;
        const long off = key ? ((long)ub0 * mm.nk + 4 * c) * mm.esz
                             : mm.dvs + ((long)ub0 * mm.nv + 4 * (c - mm.kp)) * mm.esz;
        L.ms[u] = mm.ks + off;
        L.dz[u] = key ? mm.dkz : mm.dvz - mm.dvs;
        L.mstride[u] = (uint32_t)((key ? mm.nk : mm.nv) * mm.esz);
    }
    return L;
}

// Issue every load of block `blk` (within the unit) of a lane.
template <class C>
__device__ __forceinline__ void load_block(BlockRegs<C>& r, const LoadMap<C>& L, int blk)
{
    const uint32_t* kc = L.kc + (size_t)blk * (2 * 64 * C::KW);
    gload_words<C::KW>(kc, r.k[0]);
    gload_words<C::KW>(kc + 64 * C::KW, r.k[1]);
    gload_words<C::VW>(L.vc + (size_t)blk * (64 * C::VW), r.v);
#pragma unroll
    for (int u = 0; u < C::NPAIR; ++u) {
        const uint8_t* ms = L.ms[u] + (size_t)blk * L.mstride[u];
        if constexpr (!C::M16) {
            r.ms[u] = __builtin_nontemporal_load((const u32x4*)ms);
            r.mz[u] = __builtin_nontemporal_load((const u32x4*)(ms + L.dz[u]));
        } else {  // four fp16 values, widened when staged
            const u32x2 s2 = __builtin_nontemporal_load((const u32x2*)ms);
            const u32x2 z2 = __builtin_nontemporal_load((const u32x2*)(ms + L.dz[u]));
            r.ms[u] = u32x4{s2.x, s2.y, 0u, 0u};
            r.mz[u] = u32x4{z2.x, z2.y, 0u, 0u};
        }
    }
}

// ------------------------------------------------------------ split state

template <class C>
struct Split {
    static constexpr int NKB = C::NKB, NMB = C::NMB, NVG = C::NVG;
    half8 qhi[C::PERCH ? 1 : NKB], qlo[C::PERCH ? 1 : NKB];  // query B operands (per-token keys)
    float qsum[C::PERCH ? 1 : NKB];                          // sum of the 32 query channels of K-block kb
    float m, lsum;                                           // running max (log2 units), lane partial sum
    float zl[NVG];                                           // lane partials of sum_t p_t z'_tg
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

    // Per-token key scores of the 32 tokens of a block (l[4 h2 + i]: token
    // 8 qg + 4 h2 + i): per group of 2^GKS K-blocks one chained MFMA sum
    // acc_g = sum_d A_d q_d, then S = sum_g s_g acc_g + z'_g sum_{d in g} q_d.
    template <int GKS>
    __device__ __forceinline__ void token_key_scores(const BlockRegs<C>& r, const float4* ks, const float4* kz,
                                                     int qg, bool qlo_on, const CodeBits& kcb, float* l)
    {
        constexpr int GK = (1 << GKS) < NKB ? (1 << GKS) : NKB;  // K-blocks per group
        constexpr int NG = NKB / GK;
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2) {
            floatx4 acc[NG];
#pragma unroll
            for (int g = 0; g < NG; ++g) {
                acc[g] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
                for (int u = 0; u < GK; ++u) {
                    const int kb = g * GK + u;
                    const half8 a = biased_codes<C::KBITS>(r.k[h2], kb, kcb);
                    acc[g] = mfma16(a, qhi[kb], acc[g]);
                    if (qlo_on)
                        acc[g] = mfma16(a, qlo[kb], acc[g]);
                }
            }
            floatx4 S;
#pragma unroll
            for (int g = 0; g < NG; ++g) {
                float qs = qsum[g * GK];
#pragma unroll
                for (int u = 1; u < GK; ++u)
                    qs += qsum[g * GK + u];
                // scale and offset of group g for tokens 8 qg + 4 h2 + i
                const int fi = g * 8 + 2 * qg + h2;
                const float4 s4 = ks[fi], z4 = kz[fi];
                const floatx4 t = {s4.x * acc[g][0] + z4.x * qs, s4.y * acc[g][1] + z4.y * qs,
                                   s4.z * acc[g][2] + z4.z * qs, s4.w * acc[g][3] + z4.w * qs};
                S = g == 0 ? t : S + t;
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
                l[4 * h2 + i] = S[i];
        }
    }

    // One coded 32-token block whose loads are in `r`; tokens at or beyond
    // `valid` are masked.  `wl` is the wave's metadata buffer; `vg` the value
    // group of this lane's column when every group has its own columns.
    __device__ __forceinline__ void coded_block(const BlockRegs<C>& r, float4* wl, const MetaMap& mm, int lane,
                                                int lgk, bool qlo_on, bool rep, int vg, const CodeBits& kcb,
                                                const CodeBits& vcb, int valid, const PerchCtx& pc)
    {
        const int qg = lane >> 4;
        // Stage the block's metadata: key scales and z' times sm_scale log2(e),
        // value scales times 2^-kTau.  LDS accesses of one wave are performed
        // in order, so the reads below see these writes without a barrier.
        const int vp = mm.np - mm.kp;
#pragma unroll
        for (int u = 0; u < C::NPAIR; ++u) {
            const int c = lane + 64 * u;
            if (c < mm.np) {
                const bool key = c < mm.kp;
                const float f = key ? mm.kmul : 1.0f;
                const float fs = key ? mm.kmul : mm.vmul;
                const float z0 = key ? mm.kz0 : mm.vz0, zs = key ? mm.kzs : mm.vzs;
                const u32x4 s = r.ms[u], z = r.mz[u];
                float sv[4], zv[4];
                if constexpr (!C::M16) {
                    sv[0] = __uint_as_float(s.x);
                    sv[1] = __uint_as_float(s.y);
                    sv[2] = __uint_as_float(s.z);
                    sv[3] = __uint_as_float(s.w);
                    zv[0] = __uint_as_float(z.x);
                    zv[1] = __uint_as_float(z.y);
                    zv[2] = __uint_as_float(z.z);
                    zv[3] = __uint_as_float(z.w);
                } else {
                    sv[0] = f16_bits_to_f32((uint16_t)s.x);
                    sv[1] = f16_bits_to_f32((uint16_t)(s.x >> 16));
                    sv[2] = f16_bits_to_f32((uint16_t)s.y);
                    sv[3] = f16_bits_to_f32((uint16_t)(s.y >> 16));
                    zv[0] = f16_bits_to_f32((uint16_t)z.x);
                    zv[1] = f16_bits_to_f32((uint16_t)(z.x >> 16));
                    zv[2] = f16_bits_to_f32((uint16_t)z.y);
                    zv[3] = f16_bits_to_f32((uint16_t)(z.y >> 16));
                }
                const int ds = key ? c : 2 * mm.kp + (c - mm.kp);
                const int dz = key ? mm.kp + c : 2 * mm.kp + vp + (c - mm.kp);
                wl[ds] = float4{sv[0] * fs, sv[1] * fs, sv[2] * fs, sv[3] * fs};
                // the mixed 2-bit operands' extra bias of even components
                // (channel or token i of a chunk sits in operand dword i)
                const float xb = key ? (C::PERCH ? mixed_extra_bias<C::KBITS>(0) : 0.0f) : mixed_extra_bias<C::VBITS>(0);
                const float zse = zs - xb;
                wl[dz] = float4{(z0 * zv[0] + zse * sv[0]) * f, (z0 * zv[1] + zs * sv[1]) * f,
                                (z0 * zv[2] + zse * sv[2]) * f, (z0 * zv[3] + zs * sv[3]) * f};
            }
        }
        const float4* ks = wl;
        const float4* kz = wl + mm.kp;
        const float4* vs = wl + 2 * mm.kp;
        const float4* vz = wl + 2 * mm.kp + vp;

        // ---------------------------------------------------- scores
        float l[8];
        if constexpr (!C::PERCH) {
            // key groups of 32 << lgk channels: one MFMA chain and one scale per group
            switch (lgk) {
            case 0:
                token_key_scores<0>(r, ks, kz, qg, qlo_on, kcb, l);
                break;
            case 1:
                token_key_scores<1>(r, ks, kz, qg, qlo_on, kcb, l);
                break;
            case 2:
                token_key_scores<2>(r, ks, kz, qg, qlo_on, kcb, l);
                break;
            default:
                token_key_scores<3>(r, ks, kz, qg, qlo_on, kcb, l);
                break;
            }
        } else {
            // Per-channel keys: B = q s_d (hi + lo), and sum_d q_d z'_d per head.
            // Writer: item it = lane + 64 j forms the eight products of its
            // (head, octet) in operand order and the octet's offset partial;
            // lanes past the last item repeat it without storing.
            constexpr int NO = C::D / 8, JMAX = (16 * NO + 63) / 64;
            float zsum[JMAX];
#pragma unroll
            for (int jj = 0; jj < JMAX; ++jj) {
                zsum[jj] = 0.0f;
                if (64 * jj < pc.items) {
                    const int it = lane + 64 * jj;
                    const int ic = min(it, pc.items - 1);
                    const int h = ic / NO, o = ic % NO;
                    const float4 qa = *(const float4*)(pc.qw + h * C::D + 8 * o);
                    const float4 qb = *(const float4*)(pc.qw + h * C::D + 8 * o + 4);
                    const float4 s0 = ks[2 * o], s1 = ks[2 * o + 1];
                    const float4 z0 = kz[2 * o], z1 = kz[2 * o + 1];
                    const float qn[8] = {qa.x, qa.y, qa.z, qa.w, qb.x, qb.y, qb.z, qb.w};
                    const float sn[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
                    const float zn[8] = {z0.x, z0.y, z0.z, z0.w, z1.x, z1.y, z1.z, z1.w};
                    float v[8];
                    float zp = 0.0f;
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        v[e] = qn[perm4(e)] * sn[perm4(e)];
                        zp += qn[e] * zn[e];
                    }
                    half8 hi, lo;
                    split_pairs(v, &hi, &lo);
                    if (it < pc.items) {
                        *(half8*)(pc.slots + 32 * it) = hi;
                        *(half8*)(pc.slots + 32 * it + 16) = lo;
                    }
                    zsum[jj] = group_sum<NO>(zp);
                }
            }
            // Reader: this column's offset term from the first lane of its
            // head's items, then the operand slots (written by this wave
            // above; a wave's LDS accesses are performed in order).
            float zq = 0.0f;
#pragma unroll
            for (int jj = 0; jj < JMAX; ++jj) {
                if (64 * jj < pc.items) {
                    const float t = __int_as_float(__builtin_amdgcn_ds_bpermute(pc.zsrc, __float_as_int(zsum[jj])));
                    zq = jj == pc.zj ? t : zq;
                }
            }
            floatx4 acc0 = {zq, zq, zq, zq}, acc1 = acc0;
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb) {
                const half8 bh = *(const half8*)(pc.slots + pc.rbase + 128 * kb);
                const half8 bl = *(const half8*)(pc.slots + pc.rbase + 128 * kb + 16);
                const half8 a0 = biased_codes<C::KBITS, true>(r.k[0], kb, kcb);
                const half8 a1 = biased_codes<C::KBITS, true>(r.k[1], kb, kcb);
                acc0 = mfma16(a0, bh, acc0);
                acc0 = mfma16(a0, bl, acc0);
                acc1 = mfma16(a1, bh, acc1);
                acc1 = mfma16(a1, bl, acc1);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                l[i] = acc0[i];
                l[4 + i] = acc1[i];
            }
        }
        if (valid < 32) {
#pragma unroll
            for (int k = 0; k < 8; ++k)
                l[k] = 8 * qg + k < valid ? l[k] : kNegInf;
        }
        softmax(l);  // l now holds p (<= 2^kTau), 0 for masked tokens

        // ---------------------------------------------------- values
        // Masked tokens have p = 0.  The slots past the cached length may hold
        // anything (storage that was never written, or left by an earlier
        // window), so in a partial block their scales and offsets are replaced
        // by zeros before they meet p; full blocks need no select.  With one
        // column set per group the B operand built in the first pass holds
        // every group.
        half8 ph, pl;
#pragma unroll
        for (int pass = 0; pass < NVG; ++pass) {
            if (pass == 0 || !rep) {
                const int g = rep ? vg : pass;
                const float4 s0 = vs[8 * g + 2 * qg], s1 = vs[8 * g + 2 * qg + 1];
                const float4 z0 = vz[8 * g + 2 * qg], z1 = vz[8 * g + 2 * qg + 1];
                float sn[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
                float zn[8] = {z0.x, z0.y, z0.z, z0.w, z1.x, z1.y, z1.z, z1.w};
                if (valid < 32) {
#pragma unroll
                    for (int k = 0; k < 8; ++k) {
                        const bool live = 8 * qg + k < valid;
                        sn[k] = live ? sn[k] : 0.0f;
                        zn[k] = live ? zn[k] : 0.0f;
                    }
                }
                float pv[8];
                float zs = 0.0f;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int k = perm4(e);
                    pv[e] = l[k] * sn[k];
                    zs += l[k] * zn[k];
                }
                zl[pass] += zs;
                split_pairs(pv, &ph, &pl);
            }
#pragma unroll
            for (int j = 0; j < C::MBPG; ++j) {
                const int mb = pass * C::MBPG + j;
                const half8 a = biased_codes<C::VBITS, true>(r.v, mb, vcb);
                oacc[mb] = mfma16(a, ph, oacc[mb]);
                oacc[mb] = mfma16(a, pl, oacc[mb]);
            }
        }
    }

    // One block of fp16 tokens (t0 .. t0 + 31, those >= n masked) read from
    // rows [unit][rows][D] at slot t mod rows: the window ring (rows = R + F)
    // or the sink (rows = sink, slot t).  Key rows feed the score operands
    // directly (a lane's eight channels are contiguous); the value operands
    // need eight tokens of one channel per lane, so the value rows are read
    // in 16-byte pieces and written transposed into the wave's LDS buffer
    // vt ([D][kVtPitch] halves, the tokens of each octet in operand order).
    __device__ __forceinline__ void fp16_block(const AttnParams& p, const uint16_t* kr, const uint16_t* vr, int ring,
                                               int n, int unit, int t0, int lane, bool qlo_on, const PerchCtx& pc,
                                               uint16_t* vt)
    {
        constexpr int D = C::D;
        const int hh = lane & 15, qg = lane >> 4;
        const size_t rbase = (size_t)unit * ring;
        // value rows -> vt (every piece of the block, masked tokens as zeros)
#pragma unroll 2
        for (int i = 0; i < D / 16; ++i) {
            const int idx = lane + 64 * i;
            const int r = idx / (D / 8), c8 = 8 * (idx % (D / 8));
            const int t = t0 + r;
            u32x4 w = {0u, 0u, 0u, 0u};
            if (t < n)
                w = *(const u32x4*)(vr + (rbase + (size_t)(t % ring)) * D + c8);
            const int e = r & 7;
            const int pos = (r & ~7) + (e < 4 ? 2 * e : 2 * (e - 4) + 1);  // operand slot of token r
            const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
            for (int k = 0; k < 8; ++k)
                vt[(c8 + k) * kVtPitch + pos] = (uint16_t)(ww[k >> 1] >> (16 * (k & 1)));
        }
        float l[8];
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2) {
            const int tA = t0 + 8 * (hh >> 2) + 4 * h2 + (hh & 3);
            const uint16_t* krow = kr + (rbase + (size_t)(tA % ring)) * D;
            half8 a[NKB];
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb) {
                a[kb] = half8{};
                if (tA < n) {
                    const half8 nat = __builtin_bit_cast(half8, *(const u32x4*)(krow + 32 * kb + 8 * qg));
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        a[kb][e] = nat[perm4(e)];
                }
            }
            floatx4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb) {
                if constexpr (C::PERCH) {
                    const float* qr = pc.qw + pc.hn * D + 32 * kb + 8 * qg;
                    const float4 qa = *(const float4*)qr, qb = *(const float4*)(qr + 4);
                    const float qn[8] = {qa.x, qa.y, qa.z, qa.w, qb.x, qb.y, qb.z, qb.w};
                    float v[8];
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        v[e] = qn[perm4(e)];
                    half8 bh, bl;
                    split_pairs(v, &bh, &bl);
                    acc = mfma16(a[kb], bh, acc);
                    acc = mfma16(a[kb], bl, acc);
                } else {
                    acc = mfma16(a[kb], qhi[kb], acc);
                    if (qlo_on)
                        acc = mfma16(a[kb], qlo[kb], acc);
                }
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
                l[4 * h2 + i] = acc[i] * p.sm_log2;
        }
#pragma unroll
        for (int k = 0; k < 8; ++k)
            l[k] = t0 + 8 * qg + k < n ? l[k] : kNegInf;
        softmax(l);  // masked tokens get p = 0 (their value rows are zeros too)
        float pv[8];
#pragma unroll
        for (int e = 0; e < 8; ++e)
            pv[e] = l[perm4(e)] * kPScale;
        half8 ph, pl;
        split_pairs(pv, &ph, &pl);
#pragma unroll
        for (int mb = 0; mb < NMB; ++mb) {
            const half8 va = *(const half8*)(vt + (16 * mb + hh) * kVtPitch + 8 * qg);
            oacc[mb] = mfma16(va, ph, oacc[mb]);
            oacc[mb] = mfma16(va, pl, oacc[mb]);
        }
    }
};

// Inverse rotation (the normalized transform is its own inverse) of G rows
// of D outputs staged in LDS, then the store to O.
template <int D, int NT>
__device__ __forceinline__ void finish_rows(const AttnParams& p, float* xo, size_t row0, int G)
{
    if (p.rotate) {
        for (int h = 1; h < D; h <<= 1) {
            for (int idx = threadIdx.x; idx < G * (D / 2); idx += NT) {
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
    for (int idx = threadIdx.x; idx < G * D; idx += NT)
        p.out[row0 * D + idx] = xo[idx] * post;
}

template <class C>
__device__ __forceinline__ void split_body(const AttnParams& p, uint8_t* lds)
{
    constexpr int D = C::D, NKB = C::NKB, NMB = C::NMB, W = C::WAVES, NT = C::THREADS;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
    const int hh = lane & 15, qg = lane >> 4;
    const int split = blockIdx.x, unit = blockIdx.y;
    const int b = unit / p.H, j = unit % p.H, G = p.G;
    const bool kaff = p.k_mode == KVQ_AFFINE, vaff = p.v_mode == KVQ_AFFINE;
    const bool qlo_on = p.rotate != 0;
    const int NB = p.T >> 5;
    const int lgk = C::PERCH ? 0 : __builtin_ctz((unsigned)p.k_group >> 5);  // log2(key group / 32)
    const int kmeta = C::PERCH ? D : 32 * (D / p.k_group);                    // key scale floats per block
    constexpr int vmeta = 32 * C::NVG;

    // Column roles: with one column set per value group, column hh is head
    // hh % G of value group hh / G; otherwise head hh.
    const bool rep = G * C::NVG <= 16 && C::NVG > 1;
    const int vg = rep ? hh / G : 0;
    const int head = rep ? hh - vg * G : hh;
    const bool active = rep ? vg < C::NVG : hh < G;

    MetaMap mm;
    mm.ks = (const uint8_t*)p.ks;
    mm.dkz = kaff ? (const uint8_t*)p.kz - (const uint8_t*)p.ks : 0;
    mm.dvs = (const uint8_t*)p.vs - (const uint8_t*)p.ks;
    mm.dvz = vaff ? (const uint8_t*)p.vz - (const uint8_t*)p.ks : mm.dvs;
    mm.esz = p.meta16 ? 2 : 4;
    mm.nk = kmeta;
    mm.nv = vmeta;
    mm.kp = kmeta / 4;
    mm.np = mm.kp + vmeta / 4;
    mm.kmul = p.sm_log2;
    mm.vmul = kPScale;
    {
        const float kb0 = code_bias<C::KBITS>(), vb0 = code_bias<C::VBITS>();
        mm.kz0 = kaff ? 1.0f : 0.0f;
        mm.kzs = kaff ? -kb0 : -((float)(1 << (C::KBITS - 1)) + kb0);
        mm.vz0 = vaff ? 1.0f : 0.0f;
        mm.vzs = vaff ? -vb0 : -((float)(1 << (C::VBITS - 1)) + vb0);
    }

    // ---- block range of this split
    const int nblk = (p.nq + 31) >> 5;
    const int blk_begin = min(nblk, split * p.bps);
    const int blk_end = min(nblk, blk_begin + p.bps);
    const size_t ub0 = (size_t)unit * NB;
    const LoadMap<C> ldm = load_map<C>(p, mm, ub0, lane);

    // ---- queries.  Without rotation each lane reads its own operand
    // pieces (head `head`, channels 32 kb + 8 qg .. + 7) straight from
    // global memory; a rotated query is first transformed as fp32 rows in LDS.
    const size_t qrow = (size_t)b * p.H_q + (size_t)j * G;
    u32x4 qpc[NKB];
    if (!p.rotate) {
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb)
            qpc[kb] = active ? *(const u32x4*)(p.q + (qrow + head) * D + 32 * kb + 8 * qg) : u32x4{0u, 0u, 0u, 0u};
    }
    BlockRegs<C> rbuf[C::NBUF];
    int blk = blk_begin + wave;
    const int last = blk_end - 1;
    // the first NBUF - 1 blocks of this wave go in flight before the query
    // setup (past the end they re-read the last block)
    if (blk_end > blk_begin) {
#pragma unroll
        for (int u = 0; u + 1 < C::NBUF; ++u)
            load_block<C>(rbuf[u], ldm, min(blk + W * u, last));
    }
    float* lq = (float*)lds;
    if (p.rotate) {
        constexpr int QPIECES = 16 * D / 8;
        for (int pc = threadIdx.x; pc < QPIECES; pc += NT) {
            const int row = pc / (D / 8);
            u32x4 raw = {0u, 0u, 0u, 0u};
            if (row < G)
                raw = *(const u32x4*)(p.q + (qrow + row) * D + (pc % (D / 8)) * 8);
            const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
            float* dst = lq + pc * 8;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                dst[2 * k] = __uint_as_float(w[k] << 16);
                dst[2 * k + 1] = __uint_as_float(w[k] & 0xFFFF0000u);
            }
        }
        __syncthreads();
        for (int h = 1; h < D; h <<= 1) {
            for (int idx = threadIdx.x; idx < 16 * (D / 2); idx += NT) {
                const int row = idx / (D / 2), k = idx % (D / 2);
                const int jj = (k / h) * 2 * h + (k % h);
                const float a = lq[row * D + jj], c = lq[row * D + jj + h];
                lq[row * D + jj] = a + c;
                lq[row * D + jj + h] = a - c;
            }
            __syncthreads();
        }
        for (int idx = threadIdx.x; idx < 16 * D; idx += NT)
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
            if (p.rotate) {
                v[k] = active ? lq[head * D + 32 * kb + 8 * qg + perm4(k)] : 0.0f;
            } else {
                // element perm4(k) of the eight bf16 channels: word perm4(k) / 2, half perm4(k) % 2
                const uint32_t w = qpc[kb][perm4(k) >> 1];
                v[k] = __uint_as_float((perm4(k) & 1) ? (w & 0xFFFF0000u) : (w << 16));
            }
            part += v[k];
        }
        if constexpr (!C::PERCH) {
            split_pairs(v, &S.qhi[kb], &S.qlo[kb]);
            S.qsum[kb] = sum_rows(part);
        }
    }
    // This wave's LDS region, and for per-channel keys the G query rows as
    // fp32 (after the rotated rows) and this lane's slot addresses.
    const bool fp16_tokens = p.ring || p.sink;
    uint8_t* region = lds + lds_waves(D, C::PERCH, G) + (size_t)wave * lds_per_wave(D, C::NPAIR, C::PERCH, G, fp16_tokens);
    PerchCtx pc = {};
    if constexpr (C::PERCH) {
        constexpr int NO = D / 8;
        float* qw = (float*)(lds + lds_qw(D));
        for (int idx = threadIdx.x; idx < G * D; idx += NT)
            qw[idx] = p.rotate ? lq[idx] : bf16_to_f32(p.q[qrow * D + idx]);
        pc.qw = qw;
        pc.slots = region + C::NPAIR * 2048;
        pc.items = G * NO;
        pc.hn = head < G ? head : 0;
        pc.rbase = (pc.hn * NO + qg) * 32;
        const int first = pc.hn * NO;  // the head's first item
        pc.zj = first >> 6;
        pc.zsrc = (first & 63) * 4;
        __syncthreads();
    }

    const CodeBits kcb = code_bits<C::KBITS>();
    const CodeBits vcb = C::KBITS == C::VBITS ? kcb : code_bits<C::VBITS>();
    {
        float4* wl = (float4*)region;
        // NBUF register sets rotate: while block blk is computed, the loads
        // of the next NBUF - 1 blocks of this wave are in flight.
        // Whole rounds of NBUF blocks, the compute of blocks past the end
        // skipped: the loop has one exit, at the top of a round, so the
        // compiler's wait counts see the same loads in flight on every path.
        for (int left = (blk_end - blk + W - 1) / W; left > 0; left -= C::NBUF) {
#pragma unroll
            for (int u = 0; u < C::NBUF; ++u) {
                load_block<C>(rbuf[(u + C::NBUF - 1) % C::NBUF], ldm, min(blk + W * (C::NBUF - 1), last));
                if (blk < blk_end)
                    S.coded_block(rbuf[u], wl, mm, lane, lgk, qlo_on, rep, vg, kcb, vcb, min(32, p.nq - 32 * blk),
                                  pc);
                blk += W;
            }
        }
    }
    // fp16 blocks (sink blocks, then window blocks): block f of the unit's
    // fp16 tokens goes to split f % S and wave (f / S) % W, round robin.
    if (fp16_tokens) {
        const int nsb = (p.n_sink + 31) >> 5, nrb = (p.n - p.nq + 31) >> 5;
        uint16_t* vt = (uint16_t*)region;  // the coded blocks are done with it
        for (int f = split + p.S_tot * wave; f < nsb + nrb; f += p.S_tot * W) {
            if (f < nsb)
                S.fp16_block(p, p.kq, p.vq, p.sink, p.n_sink, unit, 32 * f, lane, qlo_on, pc, vt);
            else
                S.fp16_block(p, p.kr, p.vr, p.ring, p.n, unit, p.nq + 32 * (f - nsb), lane, qlo_on, pc, vt);
        }
    }

    // ---- merge the W waves of this split in LDS
    const float lsum = sum_rows(S.lsum);
    float zl[C::NVG];
#pragma unroll
    for (int g = 0; g < C::NVG; ++g)
        zl[g] = sum_rows(S.zl[g]);
    __syncthreads();
    float* lm = (float*)lds;      // [W][16] running max per wave and head
    float* ll = lm + W * 16;      // [W][16] softmax sums
    float* lo = lm + 2 * W * 16;  // [W][G][D] unnormalized outputs
    float* xo = lo;  // [G][D] result: element idx is written after its own W reads
    if (qg == 0 && vg == 0 && active) {
        lm[wave * 16 + head] = S.m;
        ll[wave * 16 + head] = lsum;
    }
    if (active) {
#pragma unroll
        for (int mb = 0; mb < NMB; ++mb) {
            const int g = mb / C::MBPG;
            // with one column set per group, a column holds its own group's channels
            if (!rep || g == vg) {
                const float z = zl[rep ? 0 : g];
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    lo[((size_t)wave * G + head) * D + 16 * mb + 4 * qg + i] =
                        S.oacc[mb][i] * (1.0f / kPScale) + z;
            }
        }
    }
    __syncthreads();
    const bool single = p.S_tot == 1;
    const size_t row0 = (size_t)b * p.H_q + (size_t)j * G;
    for (int idx = threadIdx.x; idx < G * D; idx += NT) {
        const int h = idx / D, d = idx % D;
        float M = kNegInf;
        for (int w = 0; w < W; ++w)
            M = fmaxf(M, lm[w * 16 + h]);
        float acc = 0.0f, Ls = 0.0f;
        if (M != kNegInf) {
            for (int w = 0; w < W; ++w) {
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
    finish_rows<D, NT>(p, xo, row0, G);
}

// Waves per SIMD the register allocation is held to: 3 at head_dim 64 (the
// block state fits without spills), a workgroup's share of a compute unit at
// head_dim 128, 1 at head_dim 256.
template <class C>
constexpr int split_waves_per_simd()
{
    return C::D == 64 ? 3 : C::D == 128 ? C::WAVES / 4 : 1;
}

template <class C>
__global__ __launch_bounds__(C::THREADS, split_waves_per_simd<C>()) void decode_split_kernel(AttnParams p)
{
    extern __shared__ float lds_f[];
    split_body<C>(p, (uint8_t*)lds_f);
}

// Merge the S_tot split partials: one thread per output element (row, d),
// kMergeThreads / D rows per workgroup.  A thread reads the (max, sum) pairs
// and partial outputs of its row in chunks of up to kMergeChunk splits, all
// loads of a chunk in flight together (no loads past the last split), and
// combines them online: O = sum_s 2^(m_s - M) o_s / sum_s 2^(m_s - M) l_s.
// The rows are then rotated back when the format rotates, and stored.
constexpr int kMergeChunk = 8, kMergeThreads = 256;

template <int D>
__global__ __launch_bounds__(kMergeThreads) void decode_merge_kernel(AttnParams p)
{
    constexpr int R = kMergeThreads / D;  // rows per workgroup
    __shared__ float xo[kMergeThreads];
    const int t = threadIdx.x, rl = t / D, d = t % D;
    const size_t rows = (size_t)p.B * p.H_q;
    const size_t row = (size_t)blockIdx.x * R + rl;
    const int S = p.S_tot;
    float Mx = kNegInf, acc = 0.0f, Ls = 0.0f;
    if (row < rows) {
        const float2* ml = (const float2*)p.part_ml + row * S;
        const float* po = p.part_o + row * S * D + d;
        for (int s0 = 0; s0 < S; s0 += kMergeChunk) {
            float2 m[kMergeChunk];
            float o[kMergeChunk];
#pragma unroll
            for (int k = 0; k < kMergeChunk; ++k) {
                if (s0 + k < S) {
                    m[k] = ml[s0 + k];
                    o[k] = po[(size_t)(s0 + k) * D];
                } else {
                    m[k] = float2{kNegInf, 0.0f};
                    o[k] = 0.0f;
                }
            }
            float cm = kNegInf;
#pragma unroll
            for (int k = 0; k < kMergeChunk; ++k)
                cm = fmaxf(cm, m[k].x);
            const float nm = fmaxf(Mx, cm);
            if (nm != kNegInf) {
                const float sc = Mx == kNegInf ? 0.0f : fast_exp2(Mx - nm);
                acc *= sc;
                Ls *= sc;
#pragma unroll
                for (int k = 0; k < kMergeChunk; ++k) {
                    const float w = m[k].x == kNegInf ? 0.0f : fast_exp2(m[k].x - nm);
                    acc += w * o[k];
                    Ls += w * m[k].y;
                }
                Mx = nm;
            }
        }
    }
    const float v = row < rows ? acc / Ls : 0.0f;
    if (!p.rotate) {
        if (row < rows)
            p.out[row * D + d] = v;
        return;
    }
    // inverse rotation of the R rows in LDS (the normalized transform is its own inverse)
    xo[t] = v;
    __syncthreads();
    for (int h = 1; h < D; h <<= 1) {
        float nv = 0.0f;
        if (t < R * D) {
            const int partner = (d & h) ? t - h : t + h;
            const float a = xo[t], c = xo[partner];
            nv = (d & h) ? c - a : a + c;
        }
        __syncthreads();
        xo[t] = nv;
        __syncthreads();
    }
    if (row < rows)
        p.out[row * D + d] = xo[t] * p.rot_c;
}

// Workgroups of the split kernel instance for `p` that fit on one compute
// unit at once (occupancy from its registers and LDS).  The answer is cached
// per instance, keyed by the LDS size.
template <class C>
int resident_per_cu(const AttnParams& p)
{
    static std::atomic<unsigned long long> cache{0};  // (lds_bytes << 32) | count, 0 = empty
    const unsigned long long lds = (unsigned long long)p.lds_bytes;
    const unsigned long long hit = cache.load(std::memory_order_relaxed);
    if (hit != 0 && (hit >> 32) == lds)
        return (int)(hit & 0xFFFFFFFFu);
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, decode_split_kernel<C>, C::THREADS, p.lds_bytes) != hipSuccess)
        n = 1;
    if (n < 1)
        n = 1;
    cache.store((lds << 32) | (unsigned)n, std::memory_order_relaxed);
    return n;
}

template <class C>
hipError_t launch_split(const AttnParams& p, hipStream_t stream)
{
    launch_kernel(decode_split_kernel<C>, dim3(p.S_tot, p.B * p.H), dim3(C::THREADS), p.lds_bytes, stream, p);
    return hipGetLastError();
}

// Calls F<Cfg<...>>::run(p, args...) for the instance that serves p.
template <template <class> class F, int D, int KB, int VB, bool PC, bool M16, int VGS = 0, class... A>
auto by_groups(const AttnParams& p, A... args)
{
    if constexpr ((32 << VGS) >= D) {
        return F<Cfg<D, KB, VB, PC, VGS, M16>>::run(p, args...);
    } else {
        if (p.v_group == (32 << VGS))
            return F<Cfg<D, KB, VB, PC, VGS, M16>>::run(p, args...);
        return by_groups<F, D, KB, VB, PC, M16, VGS + 1>(p, args...);
    }
}

template <template <class> class F, int D, bool M16, bool PC, class... A>
auto by_bits(const AttnParams& p, A... args)
{
    if (p.k_bits == 8)  // 8-bit codes come as K and V both 8-bit
        return by_groups<F, D, 8, 8, PC, M16>(p, args...);
    if (p.k_bits == 4 && p.v_bits == 4)
        return by_groups<F, D, 4, 4, PC, M16>(p, args...);
    if (p.k_bits == 4 && p.v_bits == 2)
        return by_groups<F, D, 4, 2, PC, M16>(p, args...);
    if (p.k_bits == 2 && p.v_bits == 4)
        return by_groups<F, D, 2, 4, PC, M16>(p, args...);
    return by_groups<F, D, 2, 2, PC, M16>(p, args...);
}

template <class C>
struct LaunchSplit {
    static hipError_t run(const AttnParams& p, hipStream_t stream) { return launch_split<C>(p, stream); }
};

template <class C>
struct Resident {
    static int run(const AttnParams& p) { return resident_per_cu<C>(p); }
};

// The split kernels of one (head size, metadata width, key axis) family:
// one translation unit each (attn_part.hip, built once per family).
template <int D, bool M16, bool PC>
hipError_t launch_split_family(const AttnParams& p, hipStream_t stream)
{
    return by_bits<LaunchSplit, D, M16, PC>(p, stream);
}

template <int D, bool M16, bool PC>
int resident_family(const AttnParams& p)
{
    return by_bits<Resident, D, M16, PC>(p);
}

template <int D>
hipError_t launch_merge(const AttnParams& p, hipStream_t stream)
{
    const int rows = p.B * p.H_q, per = kMergeThreads / D;
    launch_kernel(decode_merge_kernel<D>, dim3((rows + per - 1) / per), dim3(kMergeThreads), 0, stream, p);
    return hipGetLastError();
}

}  // namespace attn
}  // namespace kvq
