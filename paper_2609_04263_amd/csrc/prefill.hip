// Chunked prefill attention over the packed cache (Sec. 3.1: evaluation
// consumes chunks; the chunk's states are coded and appended, then its
// queries attend causally over the reconstruction of everything stored).
//
// One workgroup per (sequence, KV head, tile of query rows); query rows are
// the (chunk token, head of the KV group) pairs in token-major order.  Each
// of the eight waves owns 16 QN query rows (the block reconstruction below
// is shared by all of them, so a workgroup takes as many rows as the
// registers allow: 128 / 256 / 512 at D = 256 / 128 / 64); the workgroup
// walks the 32-token key blocks up to its newest query's position:
//   1. the block is reconstructed into LDS (all 512 threads, one eight-code
//      piece of K and one of V each per step) from a raw copy of its codes
//      and metadata that was fetched into LDS while the previous block was
//      computed (each section of the cache is blocked by 32 tokens, so a
//      block's bytes are six contiguous ranges): k_hat in fp32 stored as
//      fp16 hi + lo (hi + lo carries ~22 bits) as [token][D], v_hat as fp16,
//      transposed [D][token];
//   2. scores S^T = K Q^T with v_mfma_f32_16x16x32_f16 (keys as rows, query
//      rows as columns; hi x hi + hi x lo + lo x hi), queries pre-scaled by
//      sm_scale * log2(e) so the softmax runs in base 2, online per column
//      (the running maximum moves only in steps of more than 2^8);
//   3. O^T += V^T P^T in fp16 (probabilities in [0, 1] and values each
//      carry an 11-bit relative rounding, well inside the output bound; the
//      logits are the precision-critical product).  A lane holds
//      score rows 4 q + i of the block's two 16-key tiles, which are exactly
//      the eight k-slots 8 q .. 8 q + 7 its next MFMA operand needs when the
//      keys of slot 8 q + e are taken as 4 q + e (e < 4) and 16 + 4 q + e - 4:
//      V^T is read in that key order, so probabilities never cross lanes.
// Sink tokens (fp16 rows) are walked first as blocks of their own, so every
// query row holds a finite running maximum before the coded tail; fp16
// window tokens past the coded ones are read from the ring in step 1.
// Rotated formats transform the queries (FWHT in LDS) and the outputs back.

#include "kvq_internal.h"
#include "kvq_device.h"

namespace kvq {
namespace pre {

constexpr int kWaves = 8, kThreads = 512;

// query rows per wave (16 QN): the accumulators take D QN / 4 registers
template <int D>
constexpr int qn()
{
    return D == 64 ? 4 : D == 128 ? 2 : 1;
}

template <int D>
constexpr int rows_per_tile()
{
    return kWaves * 16 * qn<D>();
}

// Raw bytes of one 32-token block: codes (4 D pieces of at most 4 bytes, 8
// for 8-bit codes) and metadata (at most D floats per section) of K and V.
template <int D, bool W8>
constexpr int raw_bytes()
{
    return 2 * 4 * D * (W8 ? 8 : 4) + 4 * D * 4;
}

// LDS (bytes): K hi/lo [32][D + 8], V^T [D][40] (fp16), then the raw block;
// the query and output rotation buffers ([rows][D] fp32) reuse the K/V part.
template <int D>
constexpr size_t kv_bytes()
{
    return 2 * 32 * (D + 8) * 2 + D * 40 * 2;
}

template <int D, bool W8>
constexpr size_t lds_bytes()
{
    constexpr size_t rot = (size_t)rows_per_tile<D>() * D * 4;
    return (kv_bytes<D>() > rot ? kv_bytes<D>() : rot) + raw_bytes<D, W8>();
}

__device__ __forceinline__ float dq(int mode, int bits, uint32_t c, float s, float z)
{
    return mode == KVQ_AFFINE ? (float)c * s + z : ((float)c - (float)(1 << (bits - 1))) * s;
}

// scale or offset i of a raw metadata range (fp32, or fp16 with meta16)
__device__ __forceinline__ float meta(const uint8_t* sec, int i, bool m16)
{
    return m16 ? f16_bits_to_f32(((const uint16_t*)sec)[i]) : ((const float*)sec)[i];
}

// eight consecutive scales or offsets from element i (a multiple of 8)
__device__ __forceinline__ void meta8(const uint8_t* sec, int i, bool m16, float* v)
{
    if (m16) {
        const u32x4 h = *(const u32x4*)(sec + 2 * i);
        const uint32_t w[4] = {h.x, h.y, h.z, h.w};
#pragma unroll
        for (int e = 0; e < 8; ++e)
            v[e] = f16_bits_to_f32((uint16_t)(w[e >> 1] >> (16 * (e & 1))));
    } else {
        const floatx4 a = *(const floatx4*)(sec + 4 * i), b = *(const floatx4*)(sec + 4 * i + 16);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            v[e] = a[e];
            v[e + 4] = b[e];
        }
    }
}

typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

// Eight codes of piece idx of a raw code range (8-bit: two u32; 4-bit: one
// u32; 2-bit: one u16), as the words holding codes 0..3 and 4..7 (the same
// word unless the codes are 8-bit).
struct Piece {
    uint32_t lo, hi;
};

template <bool W8>
__device__ __forceinline__ Piece piece(const uint8_t* sec, int idx, int bits)
{
    if constexpr (W8) {
        const u32x2 w = ((const u32x2*)sec)[idx];
        return Piece{w.x, w.y};
    }
    const uint32_t w = bits == 4 ? ((const uint32_t*)sec)[idx] : ((const uint16_t*)sec)[idx];
    return Piece{w, w};
}

// Code e (0..7) of a piece.
__device__ __forceinline__ uint32_t code_of(const Piece& w, int bits, int e)
{
    const uint32_t x = e < 4 ? w.lo : w.hi;
    return (x >> ((bits * e) & 31)) & ((1u << bits) - 1u);
}


__device__ __forceinline__ void split8(const float* v, uint16_t* hi, uint16_t* lo)
{
    half8 h, l;
    split_half8(v, &h, &l);
    *(u32x4*)hi = __builtin_bit_cast(u32x4, h);
    *(u32x4*)lo = __builtin_bit_cast(u32x4, l);
}

// In-place unnormalized FWHT of rows [rows][D] fp32 in LDS, then * c.
template <int D>
__device__ void fwht_rows(float* x, int rows, float c)
{
    for (int h = 1; h < D; h <<= 1) {
        for (int idx = threadIdx.x; idx < rows * (D / 2); idx += kThreads) {
            const int row = idx / (D / 2), k = idx % (D / 2);
            const int j = (k / h) * 2 * h + (k % h);
            const float a = x[row * D + j], b = x[row * D + j + h];
            x[row * D + j] = a + b;
            x[row * D + j + h] = a - b;
        }
        __syncthreads();
    }
    for (int idx = threadIdx.x; idx < rows * D; idx += kThreads)
        x[idx] *= c;
    __syncthreads();
}

// W8: both code widths are 8 bits (a raw block twice as large); otherwise
// 2 or 4 bits each.
template <int D, bool W8>
__global__ __launch_bounds__(kThreads) void prefill_kernel(AttnParams p)
{
    constexpr int QN = qn<D>(), RT = rows_per_tile<D>(), NKS = D / 32, NCT = D / 16;
    constexpr int KP = D + 8, VP = 40;  // LDS pitches (fp16 units)
    extern __shared__ __attribute__((aligned(16))) uint8_t plds[];
    uint16_t* kh = (uint16_t*)plds;
    uint16_t* kl = kh + 32 * KP;
    uint16_t* vh = kl + 32 * KP;
    constexpr size_t kRawOff = lds_bytes<D, W8>() - raw_bytes<D, W8>();
    uint8_t* raw = plds + kRawOff;

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int col = lane & 15, qg = lane >> 4;
    const int unit = blockIdx.y, b = unit / p.H, h = unit % p.H;
    const int G = p.G, C = p.C;
    const int rows = C * G;
    const int r0 = blockIdx.x * RT;
    // Positions are tail indices (token minus sink); sink tokens sit at
    // -sink .. -1, so a chunk that starts in the sink has negative positions.
    const int first_pos = p.n - C;  // position of chunk token 0

    // ---- queries: lane's columns are rows r0 + 16 (QN wave + c) + col
    half8 qh[QN][NKS], ql[QN][NKS];
    {
        float* xq = (float*)plds;  // [RT][D] fp32
        for (int idx = threadIdx.x; idx < RT * (D / 8); idx += kThreads) {
            const int rr = idx / (D / 8), d8 = 8 * (idx % (D / 8));
            const int R = r0 + rr;
            u32x4 qw = {0u, 0u, 0u, 0u};
            if (R < rows) {
                const int i = R / G, g = R % G;
                qw = *(const u32x4*)(p.q + (((size_t)b * C + i) * p.H_q + (size_t)h * G + g) * D + d8);
            }
            const uint32_t w[4] = {qw.x, qw.y, qw.z, qw.w};
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                xq[rr * D + d8 + 2 * k] = __uint_as_float(w[k] << 16);
                xq[rr * D + d8 + 2 * k + 1] = __uint_as_float(w[k] & 0xFFFF0000u);
            }
        }
        __syncthreads();
        if (p.rotate)
            fwht_rows<D>(xq, RT, p.rot_c);
#pragma unroll
        for (int c = 0; c < QN; ++c) {
            const int rr = 16 * (QN * wave + c) + col;
#pragma unroll
            for (int ks = 0; ks < NKS; ++ks) {
                float v[8];
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    v[e] = xq[rr * D + 32 * ks + 8 * qg + e] * p.sm_log2;
                split_half8(v, &qh[c][ks], &ql[c][ks]);
            }
        }
        __syncthreads();  // the K/V buffers overwrite the query rows
    }

    // position of each of this lane's query columns (kNoRow: no such row,
    // every key masked)
    constexpr int kNoRow = -(1 << 30);
    int qpos[QN];
    int newest;
#pragma unroll
    for (int c = 0; c < QN; ++c) {
        const int R = r0 + 16 * (QN * wave + c) + col;
        qpos[c] = R < rows ? first_pos + R / G : kNoRow;
    }
    {
        const int Rlast = min(r0 + RT, rows) - 1;
        newest = first_pos + Rlast / G;
    }

    floatx4 acc[QN][NCT];
    float m[QN], lsum[QN];
#pragma unroll
    for (int c = 0; c < QN; ++c) {
        m[c] = -INFINITY;
        lsum[c] = 0.0f;
#pragma unroll
        for (int t = 0; t < NCT; ++t)
            acc[c][t] = floatx4{0.f, 0.f, 0.f, 0.f};
    }

    const int NB = p.T >> 5;
    const size_t ub0 = (size_t)unit * NB;
    const int nkb = newest >= 0 ? newest / 32 + 1 : 0;  // coded-tail blocks
    // sink blocks holding a token no later than the newest query
    const int nsb = min((p.n_sink + 31) >> 5, (newest + p.sink) / 32 + 1);
    const int sb0 = p.sink >> 5;  // sink block j is tail block j - sb0
    const int kbits = W8 ? 8 : p.k_bits, vbits = W8 ? 8 : p.v_bits;
    const bool kaff = p.k_mode == KVQ_AFFINE, vaff = p.v_mode == KVQ_AFFINE;

    // Byte ranges of one block's raw data, in the order they sit in LDS: Kc,
    // Ks, Kz, Vc, Vs, Vz (Kz, Vz empty for symmetric codes).  Kept in scalars
    // (selects, no indexed arrays) so nothing lands in scratch memory.
    const int msz = p.meta16 ? 2 : 4;  // bytes per scale or offset
    const int kmeta = p.k_axis == KVQ_PER_TOKEN ? (D / p.k_group) * 32 * msz : D * msz;
    const int vmeta = (D / p.v_group) * 32 * msz;
    const int len0 = 4 * D * kbits, len1 = kmeta, len2 = kaff ? kmeta : 0;
    const int len3 = 4 * D * vbits, len4 = vmeta, len5 = vaff ? vmeta : 0;
    const int st1 = len0, st2 = st1 + len1, st3 = st2 + len2, st4 = st3 + len3, st5 = st4 + len4;
    const int st6 = st5 + len5;
    // this thread's 16-byte units of a block's raw data
    constexpr int UPT = (raw_bytes<D, W8>() / 16 + kThreads - 1) / kThreads;
    u32x4 pre[UPT];
    auto fetch_raw = [&](int blk) {
        const size_t ibf = ub0 + blk;
#pragma unroll
        for (int k = 0; k < UPT; ++k) {
            const int off = 16 * ((int)threadIdx.x + kThreads * k);
            pre[k] = u32x4{0u, 0u, 0u, 0u};
            if (off < st6) {
                const uint8_t* src;
                if (off < st1)
                    src = (const uint8_t*)p.kc + ibf * len0 + off;
                else if (off < st2)
                    src = (const uint8_t*)p.ks + ibf * len1 + (off - st1);
                else if (off < st3)
                    src = (const uint8_t*)p.kz + ibf * len2 + (off - st2);
                else if (off < st4)
                    src = (const uint8_t*)p.vc + ibf * len3 + (off - st3);
                else if (off < st5)
                    src = (const uint8_t*)p.vs + ibf * len4 + (off - st4);
                else
                    src = (const uint8_t*)p.vz + ibf * len5 + (off - st5);
                pre[k] = *(const u32x4*)src;
            }
        }
    };
    auto store_raw = [&]() {
#pragma unroll
        for (int k = 0; k < UPT; ++k) {
            const int off = 16 * ((int)threadIdx.x + kThreads * k);
            if (off < st6)
                *(u32x4*)(raw + off) = pre[k];
        }
    };
    const uint8_t* rkc = raw;
    const uint8_t* rks = raw + st1;
    const uint8_t* rkz = raw + st2;
    const uint8_t* rvc = raw + st3;
    const uint8_t* rvs = raw + st4;
    const uint8_t* rvz = raw + st5;
    const bool m16 = p.meta16 != 0;

    if (nkb > 0) {
        fetch_raw(0);
        store_raw();
    }
    __syncthreads();
    for (int it = 0; it < nsb + nkb; ++it) {
        const int blk = it < nsb ? it - sb0 : it - nsb;
        if (blk >= 0 && blk + 1 < nkb)
            fetch_raw(blk + 1);  // lands while this block is computed
        if (blk < 0) {
            // ---- a sink block: fp16 rows, tokens past n_sink zero
            const size_t sbase = (size_t)unit * p.sink;
            for (int pc = threadIdx.x; pc < 4 * D; pc += kThreads) {
                {
                    const int tau = pc / (D / 8), P = pc % (D / 8);
                    const int t = p.sink + 32 * blk + tau;
                    float v[8];
                    if (t < p.n_sink) {
                        const u32x4 rw = *(const u32x4*)(p.kq + (sbase + t) * D + 8 * P);
                        const uint32_t w4[4] = {rw.x, rw.y, rw.z, rw.w};
#pragma unroll
                        for (int e = 0; e < 8; ++e)
                            v[e] = f16_bits_to_f32((uint16_t)(w4[e >> 1] >> (16 * (e & 1))));
                    } else {
#pragma unroll
                        for (int e = 0; e < 8; ++e)
                            v[e] = 0.0f;
                    }
                    split8(v, kh + tau * KP + 8 * P, kl + tau * KP + 8 * P);
                }
                {
                    const int o = pc / D, d = pc % D;
                    const int t0 = p.sink + 32 * blk + 8 * o;
                    uint16_t hv[8];
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        hv[e] = t0 + e < p.n_sink ? p.vq[(sbase + t0 + e) * D + d] : (uint16_t)0;
                    *(u32x4*)(vh + d * VP + 8 * o) =
                        u32x4{hv[0] | ((uint32_t)hv[1] << 16), hv[2] | ((uint32_t)hv[3] << 16),
                              hv[4] | ((uint32_t)hv[5] << 16), hv[6] | ((uint32_t)hv[7] << 16)};
                }
            }
        } else {
        // ---- reconstruct the block into LDS: 4 D pieces of K and of V
        for (int pc = threadIdx.x; pc < 4 * D; pc += kThreads) {
            // K piece: token tau = pc / (D / 8), channels 8 P .. 8 P + 7
            {
                const int tau = pc / (D / 8), P = pc % (D / 8);
                const int t = 32 * blk + tau;
                float v[8];
                if (t < p.nq) {
                    const int row = 4 * (tau / 8) + tau % 4, half = (tau / 4) % 2;
                    const int idx = (half * 64 + row + 16 * (P % 4)) * (D / 32) + P / 4;
                    const Piece w = piece<W8>(rkc, idx, kbits);
                    if (p.k_axis == KVQ_PER_TOKEN) {
                        const int mi = ((8 * P) / p.k_group) * 32 + tau;
                        const float sc = meta(rks, mi, m16), z = kaff ? meta(rkz, mi, m16) : 0.0f;
#pragma unroll
                        for (int e = 0; e < 8; ++e)
                            v[e] = dq(p.k_mode, kbits, code_of(w, kbits, e), sc, z);
                    } else {
#pragma unroll
                        for (int e = 0; e < 8; ++e) {
                            const int mi = 8 * P + e;
                            v[e] = dq(p.k_mode, kbits, code_of(w, kbits, e), meta(rks, mi, m16),
                                      kaff ? meta(rkz, mi, m16) : 0.0f);
                        }
                    }
                } else {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        v[e] = 0.0f;
                }
                split8(v, kh + tau * KP + 8 * P, kl + tau * KP + 8 * P);
            }
            // V piece: octet o = pc / D (tokens 8 o .. 8 o + 7), channel d
            {
                const int o = pc / D, d = pc % D;
                float v[8];
                const int t0 = 32 * blk + 8 * o;
                const int idx = (d % 16 + 16 * o) * (D / 16) + d / 16;
                const Piece w = t0 < p.nq ? piece<W8>(rvc, idx, vbits) : Piece{0u, 0u};
                // the octet's eight scales (and offsets) are consecutive
                const int mi = (d / p.v_group) * 32 + 8 * o;
                float sv[8], zv[8];
                meta8(rvs, mi, m16, sv);
                if (vaff)
                    meta8(rvz, mi, m16, zv);
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float sc = sv[e], z = vaff ? zv[e] : 0.0f;
                    v[e] = t0 + e < p.nq ? dq(p.v_mode, vbits, code_of(w, vbits, e), sc, z) : 0.0f;
                }
                *(u32x4*)(vh + d * VP + 8 * o) = __builtin_bit_cast(u32x4, pack_half8(v));
            }
        }
        // tokens of the fp16 window (past the coded ones): the same pieces,
        // from the ring in global memory, in a pass of their own so that
        // the coded pass never waits on global loads
        if (32 * blk + 31 >= p.nq && 32 * blk < p.n) {
            for (int pc = threadIdx.x; pc < 4 * D; pc += kThreads) {
                {
                    const int tau = pc / (D / 8), P = pc % (D / 8);
                    const int t = 32 * blk + tau;
                    if (t >= p.nq && t < p.n) {
                        const u32x4 rw = *(const u32x4*)(p.kr + (((size_t)unit * p.ring) + t % p.ring) * D + 8 * P);
                        const uint32_t w4[4] = {rw.x, rw.y, rw.z, rw.w};
                        float v[8];
#pragma unroll
                        for (int e = 0; e < 8; ++e)
                            v[e] = f16_bits_to_f32((uint16_t)(w4[e >> 1] >> (16 * (e & 1))));
                        split8(v, kh + tau * KP + 8 * P, kl + tau * KP + 8 * P);
                    }
                }
                {
                    const int o = pc / D, d = pc % D;
                    const int t0 = 32 * blk + 8 * o;
                    if (t0 + 7 >= p.nq && t0 < p.n) {
                        uint16_t hv[8];
#pragma unroll
                        for (int e = 0; e < 8; ++e) {
                            const int t = t0 + e;
                            hv[e] = (t >= p.nq && t < p.n) ? p.vr[(((size_t)unit * p.ring) + t % p.ring) * D + d]
                                                           : vh[d * VP + 8 * o + e];
                        }
                        *(u32x4*)(vh + d * VP + 8 * o) =
                            u32x4{hv[0] | ((uint32_t)hv[1] << 16), hv[2] | ((uint32_t)hv[3] << 16),
                                  hv[4] | ((uint32_t)hv[5] << 16), hv[6] | ((uint32_t)hv[7] << 16)};
                    }
                }
            }
        }
        }  // coded-tail block
        __syncthreads();

        // ---- scores S^T (keys x query rows), two 16-key tiles
        floatx4 s[QN][2];
#pragma unroll
        for (int c = 0; c < QN; ++c)
            s[c][0] = s[c][1] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
            for (int ks = 0; ks < NKS; ++ks) {
                const int off = (16 * kt + col) * KP + 32 * ks + 8 * qg;
                const half8 ah = __builtin_bit_cast(half8, *(const u32x4*)(kh + off));
                const half8 al = __builtin_bit_cast(half8, *(const u32x4*)(kl + off));
#pragma unroll
                for (int c = 0; c < QN; ++c) {
                    s[c][kt] = mfma16(ah, qh[c][ks], s[c][kt]);
                    s[c][kt] = mfma16(ah, ql[c][ks], s[c][kt]);
                    s[c][kt] = mfma16(al, qh[c][ks], s[c][kt]);
                }
            }
        }

        // ---- online softmax per query column; P^T operands
        half8 ph[QN];
#pragma unroll
        for (int c = 0; c < QN; ++c) {
            float x[8];
            float bm = -INFINITY;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int key = 32 * blk + (e < 4 ? 4 * qg + e : 16 + 4 * qg + e - 4);
                x[e] = key <= qpos[c] ? s[c][e >> 2][e & 3] : -INFINITY;
                bm = fmaxf(bm, x[e]);
            }
            bm = xor_max16_32(bm);
            // the running maximum is raised only when a block exceeds it by
            // more than 8 (log2 units): probabilities stay below 2^8, and the
            // accumulators are rescaled a few times per row, not per block
            if (bm > m[c] + 8.0f) {
                const float alpha = m[c] == -INFINITY ? 0.0f : fast_exp2(m[c] - bm);
                m[c] = bm;
                lsum[c] *= alpha;
#pragma unroll
                for (int t = 0; t < NCT; ++t)
                    acc[c][t] *= alpha;
            }
            const float mn = m[c];
            float pv[8];
            float ps = 0.0f;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                pv[e] = x[e] == -INFINITY ? 0.0f : fast_exp2(x[e] - mn);
                ps += pv[e];
            }
            lsum[c] += ps;
            ph[c] = pack_half8(pv);
        }

        // ---- O^T += V^T P^T, 16 channels per tile, keys in the slot order above
#pragma unroll
        for (int t = 0; t < NCT; ++t) {
            const int d = 16 * t + col;
            const uint2 h0 = *(const uint2*)(vh + d * VP + 4 * qg);
            const uint2 h1 = *(const uint2*)(vh + d * VP + 16 + 4 * qg);
            const half8 ah = __builtin_bit_cast(half8, u32x4{h0.x, h0.y, h1.x, h1.y});
#pragma unroll
            for (int c = 0; c < QN; ++c)
                acc[c][t] = mfma16(ah, ph[c], acc[c][t]);
        }
        if (blk >= 0 && blk + 1 < nkb)
            store_raw();  // the raw block was consumed before the barrier above
        __syncthreads();  // the next block overwrites K, V and the raw copy
    }

    // ---- normalize and write: lane holds O[row][16 t + 4 qg + i]
    float inv[QN];
#pragma unroll
    for (int c = 0; c < QN; ++c) {
        const float l = xor_sum16_32(lsum[c]);
        inv[c] = l > 0.0f ? 1.0f / l : 0.0f;
    }
    if (!p.rotate) {
#pragma unroll
        for (int c = 0; c < QN; ++c) {
            const int R = r0 + 16 * (QN * wave + c) + col;
            if (R >= rows)
                continue;
            const int i = R / G, g = R % G;
            float* dst = p.out + (((size_t)b * C + i) * p.H_q + (size_t)h * G + g) * D;
#pragma unroll
            for (int t = 0; t < NCT; ++t)
                *(floatx4*)(dst + 16 * t + 4 * qg) = acc[c][t] * inv[c];
        }
        return;
    }
    float* xo = (float*)plds;  // [RT][D] fp32
#pragma unroll
    for (int c = 0; c < QN; ++c) {
        const int rr = 16 * (QN * wave + c) + col;
#pragma unroll
        for (int t = 0; t < NCT; ++t)
            *(floatx4*)(xo + rr * D + 16 * t + 4 * qg) = acc[c][t] * inv[c];
    }
    __syncthreads();
    fwht_rows<D>(xo, RT, p.rot_c);
    for (int idx = threadIdx.x; idx < RT * (D / 4); idx += kThreads) {
        const int rr = idx / (D / 4), d4 = 4 * (idx % (D / 4));
        const int R = r0 + rr;
        if (R >= rows)
            continue;
        const int i = R / G, g = R % G;
        *(floatx4*)(p.out + (((size_t)b * C + i) * p.H_q + (size_t)h * G + g) * D + d4) =
            *(const floatx4*)(xo + rr * D + d4);
    }
}

template <int D>
hipError_t launch(const AttnParams& p, hipStream_t stream)
{
    constexpr int RT = rows_per_tile<D>();
    const dim3 grid((p.C * p.G + RT - 1) / RT, p.B * p.H);
    const bool w8 = p.k_bits == 8;  // 8-bit codes come as K and V both 8-bit
    void (*kern)(AttnParams) = w8 ? prefill_kernel<D, true> : prefill_kernel<D, false>;
    const size_t lds = w8 ? lds_bytes<D, true>() : lds_bytes<D, false>();
    launch_kernel(kern, grid, dim3(kThreads), lds, stream, p);
    return hipGetLastError();
}

}  // namespace pre

hipError_t launch_prefill(const AttnParams& p, int D, hipStream_t stream)
{
    switch (D) {
    case 64:
        return pre::launch<64>(p, stream);
    case 128:
        return pre::launch<128>(p, stream);
    case 256:
        return pre::launch<256>(p, stream);
    default:
        return hipErrorInvalidValue;
    }
}

}  // namespace kvq
