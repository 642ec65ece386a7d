// Split-K decode attention over the packed cache with in-kernel
// reconstruction (Sec. 3.1-3.2 of the paper: attention sees the stored
// reconstruction; here it is computed from codes without materializing it).
//
// Work decomposition: one workgroup of 4 waves per (split, sequence, KV
// head).  The G query heads that share a KV head form the N = 16 columns of
// v_mfma_f32_16x16x32_f16 (heads >= G are zero), so every code is read from
// HBM once per KV head.  Each wave walks aligned 32-token blocks:
//
//   scores   per-token keys: S^T[t][h] = sum_g s_g (sum_{d in g} c[t][d] q[h][d])
//            + z_g sum_{d in g} q[h][d], with the codes as exact fp16 MFMA
//            operands (A) and the queries as B (fp16; rotated queries use an
//            extra fp16 remainder operand); per-channel keys fold the channel
//            scale into the query operand (hi + lo fp16 parts);
//   softmax  online, base 2, max/sum reduced across the four 16-lane rows;
//   values   O^T[d][h] += sum_t c[t][d] (p_t s_t) + sum_t p_t z_t with value
//            codes packed along tokens (A) and p * s as hi + lo fp16 parts (B).
//
// Codes become exact fp16 operands with the 0x6400 exponent trick and one
// packed fp16 subtract, so every product in the MFMAs is exact and the
// accumulation is fp32.  Tokens of the fp16 window (KIVI) are handled by one
// extra split per KV head that feeds the fp16 values to the same MFMAs.  Each
// split writes an unnormalized partial (m, l, o) to the workspace and a
// second kernel merges them (a kernel boundary instead of an in-kernel
// cross-workgroup handoff, whose agent-scope fences write back and
// invalidate the whole L2 on gfx950).  With a single split the first kernel
// writes the outputs itself.

#include "kvq_device.h"
#include "kvq_internal.h"

namespace kvq {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr float kNegInf = -__builtin_inff();

template <int BITS>
__device__ __forceinline__ uint32_t key_code_word(const uint32_t* row, int kb, int qg)
{
    // Eight codes along head_dim: d = 32 kb + 8 qg + 0..7.
    if (BITS == 4)
        return row[4 * kb + qg];
    return row[2 * kb + (qg >> 1)] >> (16 * (qg & 1));
}

template <int BITS>
__device__ __forceinline__ uint32_t value_code_word(const uint32_t* vc, int D, int t8, int d)
{
    // Eight codes along tokens: t = t8 .. t8 + 7 (t8 a multiple of 8, relative
    // to a 32-token-aligned base), channel d.
    if (BITS == 4)
        return vc[(t8 >> 3) * D + d];
    return vc[(t8 >> 4) * D + d] >> (16 * ((t8 >> 3) & 1));
}

// Bytes one 32-token block of coded tokens occupies in the LDS stage:
// key codes, key scales (+ offsets), value codes, value scales (+ offsets).
struct BlockBytes {
    int kc, ks, kz, vc, vs, vz;
    __host__ __device__ int total() const { return kc + ks + kz + vc + vs + vz; }
};

__host__ __device__ inline BlockBytes block_bytes(int D, int k_bits, int v_bits, int k_axis, int k_group,
                                                  int v_group, int k_mode, int v_mode)
{
    BlockBytes r;
    r.kc = 32 * (D * k_bits / 32) * 4;
    r.ks = k_axis == KVQ_PER_TOKEN ? 32 * (D / k_group) * 4 : D * 4;
    r.kz = k_mode == KVQ_AFFINE ? r.ks : 0;
    r.vc = v_bits * D * 4;
    r.vs = 32 * (D / v_group) * 4;
    r.vz = v_mode == KVQ_AFFINE ? r.vs : 0;
    return r;
}

// Up to six contiguous 16-byte-aligned chunks copied from global memory
// into LDS by the whole workgroup: chunk k has n_k 16-byte units read from
// src_k and written consecutively from LDS 16-byte index o_k = n_0 + ... +
// n_(k-1).  issue() starts every load of a thread (kStageLoads 16-byte
// loads, enough for kStageBytes) before any is used, so a split pays one
// memory round trip; commit() writes them to LDS.
constexpr int kStageBytes = 64 * 1024;
constexpr int kStageLoads = kStageBytes / (16 * kThreads);

struct Chunks {
    const u32x4* src[6];
    int end[6];  // cumulative 16-byte counts
};

struct Stager {
    u32x4 r[kStageLoads];

    __device__ __forceinline__ void issue(const Chunks& c)
    {
#pragma unroll
        for (int u = 0; u < kStageLoads; ++u) {
            const int idx = u * kThreads + (int)threadIdx.x;
            if (idx < c.end[5]) {
                const u32x4* src;
                int off;
                if (idx < c.end[0]) { src = c.src[0]; off = idx; }
                else if (idx < c.end[1]) { src = c.src[1]; off = idx - c.end[0]; }
                else if (idx < c.end[2]) { src = c.src[2]; off = idx - c.end[1]; }
                else if (idx < c.end[3]) { src = c.src[3]; off = idx - c.end[2]; }
                else if (idx < c.end[4]) { src = c.src[4]; off = idx - c.end[3]; }
                else { src = c.src[5]; off = idx - c.end[4]; }
                r[u] = src[off];
            }
        }
    }

    __device__ __forceinline__ void commit(const Chunks& c, u32x4* lds16)
    {
#pragma unroll
        for (int u = 0; u < kStageLoads; ++u) {
            const int idx = u * kThreads + (int)threadIdx.x;
            if (idx < c.end[5])
                lds16[idx] = r[u];
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
                int r = idx / (D / 2), k = idx % (D / 2);
                int jj = (k / h) * 2 * h + (k % h);
                float a = xo[r * D + jj], c = xo[r * D + jj + h];
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

template <int D, int KBITS, int VBITS, bool PERCH>
__device__ __forceinline__ void run_split(const AttnParams& p, float* lds)
{
    constexpr int NKB = D / 32;   // 32-wide K-blocks of the score MFMA
    constexpr int NMB = D / 16;   // 16-row M-blocks of the value MFMA
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int hh = lane & 15, qg = lane >> 4;
    const int split = blockIdx.x, unit = blockIdx.y;
    const int b = unit / p.H, j = unit % p.H;
    const bool ring_split = p.ring && split == p.S_q;

    // ---- split range
    int t_begin, t_end, blk_begin, blk_end;
    if (ring_split) {
        t_begin = p.nq;
        t_end = p.n;
        blk_begin = 0;
        blk_end = (p.n - p.nq + 31) / 32;
    } else {
        t_begin = 0;
        t_end = p.nq;
        int nblk = (p.nq + 31) / 32;
        blk_begin = split * p.bps;
        blk_end = min(nblk, blk_begin + p.bps);
    }
    const int T = p.T;
    constexpr int WPT = D * KBITS / 32;  // key code words per token
    const int kng = D / p.k_group, vng = D / p.v_group;
    const int ta = 32 * blk_begin;  // first token of the split

    // ---- LDS: [stage of the split's coded tokens][queries fp32 16 x D]
    const BlockBytes bb = block_bytes(D, KBITS, VBITS, PERCH ? KVQ_PER_CHANNEL : KVQ_PER_TOKEN, p.k_group,
                                      p.v_group, p.k_mode, p.v_mode);
    const int nb = ring_split ? 0 : blk_end - blk_begin;
    uint8_t* stage = (uint8_t*)lds;
    const uint32_t* lkc = (const uint32_t*)stage;
    const float* lks = (const float*)(stage + nb * bb.kc);
    const float* lkz = (const float*)(stage + nb * (bb.kc + bb.ks));
    const uint32_t* lvc = (const uint32_t*)(stage + nb * (bb.kc + bb.ks + bb.kz));
    const float* lvs = (const float*)(stage + nb * (bb.kc + bb.ks + bb.kz + bb.vc));
    const float* lvz = (const float*)(stage + nb * (bb.kc + bb.ks + bb.kz + bb.vc + bb.vs));
    float* lq = (float*)(stage + p.q_lds_offset);

    // ---- one round of loads: queries (8 bf16 per 16-byte load) + the stage
    constexpr int QPIECES = 16 * D / 8;
    constexpr int QLOADS = (QPIECES + kThreads - 1) / kThreads;
    u32x4 qraw[QLOADS];
#pragma unroll
    for (int u = 0; u < QLOADS; ++u) {
        const int piece = u * kThreads + (int)threadIdx.x, row = piece / (D / 8);
        qraw[u] = u32x4{0u, 0u, 0u, 0u};
        if (piece < QPIECES && row < p.G)
            qraw[u] = *(const u32x4*)(p.q + ((size_t)b * p.H_q + (size_t)j * p.G + row) * D + (piece % (D / 8)) * 8);
    }
    Stager st;
    Chunks ch;
    if (!ring_split) {
        const size_t kmeta = PERCH ? ((size_t)unit * (T / 32) + blk_begin) * D : ((size_t)unit * T + ta) * kng;
        ch.src[0] = (const u32x4*)(p.kc + ((size_t)unit * T + ta) * WPT);
        ch.src[1] = (const u32x4*)(p.ks + kmeta);
        ch.src[2] = (const u32x4*)(p.kz + kmeta);
        ch.src[3] = (const u32x4*)(p.vc + ((size_t)unit * (T * VBITS / 32) + ta * VBITS / 32) * D);
        ch.src[4] = (const u32x4*)(p.vs + ((size_t)unit * T + ta) * vng);
        ch.src[5] = (const u32x4*)(p.vz + ((size_t)unit * T + ta) * vng);
        ch.end[0] = nb * bb.kc / 16;
        ch.end[1] = ch.end[0] + nb * bb.ks / 16;
        ch.end[2] = ch.end[1] + nb * bb.kz / 16;
        ch.end[3] = ch.end[2] + nb * bb.vc / 16;
        ch.end[4] = ch.end[3] + nb * bb.vs / 16;
        ch.end[5] = ch.end[4] + nb * bb.vz / 16;
        st.issue(ch);
    }
#pragma unroll
    for (int u = 0; u < QLOADS; ++u) {
        const int piece = u * kThreads + (int)threadIdx.x;
        if (piece < QPIECES) {
            const uint32_t w[4] = {qraw[u].x, qraw[u].y, qraw[u].z, qraw[u].w};
            float* dst = lq + piece * 8;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                dst[2 * e] = __uint_as_float(w[e] << 16);
                dst[2 * e + 1] = __uint_as_float(w[e] & 0xFFFF0000u);
            }
        }
    }
    if (!ring_split)
        st.commit(ch, (u32x4*)stage);
    __syncthreads();
    if (p.rotate) {
        for (int h = 1; h < D; h <<= 1) {
            for (int idx = threadIdx.x; idx < 16 * (D / 2); idx += kThreads) {
                int row = idx / (D / 2), k = idx % (D / 2);
                int jj = (k / h) * 2 * h + (k % h);
                float a = lq[row * D + jj], c = lq[row * D + jj + h];
                lq[row * D + jj] = a + c;
                lq[row * D + jj + h] = a - c;
            }
            __syncthreads();
        }
        for (int idx = threadIdx.x; idx < 16 * D; idx += kThreads)
            lq[idx] *= p.rot_c;
        __syncthreads();
    }
    // Query operand per K-block: fp16 hi part (exact for bf16 queries) and,
    // when the query is not bf16 (rotated), the fp16 remainder as a lo part.
    const bool qlo = p.rotate != 0;
    float qf[NKB][8];      // fp32 query elements of this lane, operand order
    half8 qhi[NKB], qlop[NKB];
    float qsum[NKB];       // sum of the 32 query elements of K-block kb (head hh)
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) {
        float part = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            qf[kb][e] = lq[hh * D + 32 * kb + 8 * qg + perm4(e)];
            part += qf[kb][e];
        }
        split_half8(qf[kb], &qhi[kb], &qlop[kb]);
        qsum[kb] = xor_sum16_32(part);
    }

    const bool kaff = p.k_mode == KVQ_AFFINE, vaff = p.v_mode == KVQ_AFFINE;
    const _Float16 kb16 = (_Float16)(1024 + (kaff ? 0 : (1 << (KBITS - 1))));
    const _Float16 vb16 = (_Float16)(1024 + (vaff ? 0 : (1 << (VBITS - 1))));
    const half2_t kbias = {kb16, kb16}, vbias = {vb16, vb16};

    float m = kNegInf, lsum = 0.0f;
    floatx4 oacc[NMB];
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb)
        oacc[mb] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};


    for (int blk = blk_begin + wave; blk < blk_end; blk += kWaves) {
        const int t0 = t_begin + 32 * blk;
        floatx4 S[2];
        // ------------------------------------------------ scores
        if (ring_split) {
            // fp16 window: K rows are exact fp16 operands.
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
                int tA = t0 + 8 * (hh >> 2) + 4 * h2 + (hh & 3);
                const uint16_t* krow = p.kr + ((size_t)unit * p.ring + (size_t)(tA % p.ring)) * D;
                floatx4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
                for (int kb = 0; kb < NKB; ++kb) {
                    half8 a = {};
                    if (tA < t_end) {
                        u32x4 raw = *(const u32x4*)(krow + 32 * kb + 8 * qg);
                        half8 nat = __builtin_bit_cast(half8, raw);
#pragma unroll
                        for (int e = 0; e < 8; ++e)
                            a[e] = nat[perm4(e)];
                    }
                    acc = mfma16(a, qhi[kb], acc);
                    if (qlo)
                        acc = mfma16(a, qlop[kb], acc);
                }
                S[h2] = acc;
            }
        } else if (!PERCH) {
            // Per-token keys: S = sum_g s_g (q . c_g) + z_g sum_{d in g} q.
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
                int tA = t0 + 8 * (hh >> 2) + 4 * h2 + (hh & 3);
                const uint32_t* krow = lkc + (tA - ta) * WPT;
                const int tS = t0 + 8 * qg + 4 * h2 - ta;  // split-relative tokens of this lane's outputs: tS + i
                floatx4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
                floatx4 Sacc = {0.0f, 0.0f, 0.0f, 0.0f};
                float qs = 0.0f;
#pragma unroll
                for (int kb = 0; kb < NKB; ++kb) {
                    half8 a = codes_to_half8<KBITS>(key_code_word<KBITS>(krow, kb, qg), kbias);
                    acc = mfma16(a, qhi[kb], acc);
                    if (qlo)
                        acc = mfma16(a, qlop[kb], acc);
                    qs += qsum[kb];
                    if ((32 * (kb + 1)) % p.k_group == 0) {
                        int g = (32 * kb) / p.k_group;
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            int mi = (tS + i) * kng + g;
                            float s = lks[mi];
                            Sacc[i] += s * acc[i];
                            if (kaff)
                                Sacc[i] += lkz[mi] * qs;
                        }
                        acc = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
                        qs = 0.0f;
                    }
                }
                S[h2] = Sacc;
            }
        } else {
            // Per-channel keys: one 32-token group per block; the channel
            // scale folds into the query operand (hi + lo fp16 parts) and the
            // offsets give one constant per head: sum_d q_d z_d.
            const int meta = (blk - blk_begin) * D;
            half8 qkh[NKB], qkl[NKB];
            float c2 = 0.0f;
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb) {
                float qs[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    int d = 32 * kb + 8 * qg + perm4(e);
                    qs[e] = qf[kb][e] * lks[meta + d];
                    if (kaff)
                        c2 += qf[kb][e] * lkz[meta + d];
                }
                split_half8(qs, &qkh[kb], &qkl[kb]);
            }
            const float zq = xor_sum16_32(c2);
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
                int tA = t0 + 8 * (hh >> 2) + 4 * h2 + (hh & 3);
                const uint32_t* krow = lkc + (tA - ta) * WPT;
                floatx4 acc = {zq, zq, zq, zq};
#pragma unroll
                for (int kb = 0; kb < NKB; ++kb) {
                    half8 a = codes_to_half8<KBITS>(key_code_word<KBITS>(krow, kb, qg), kbias);
                    acc = mfma16(a, qkh[kb], acc);
                    acc = mfma16(a, qkl[kb], acc);
                }
                S[h2] = acc;
            }
        }

        // ------------------------------------------------ softmax (base 2)
        float pr[8];  // probabilities of tokens t0 + 8 qg + k, k = 4 h2 + i
        float bm = kNegInf;
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                int t = t0 + 8 * qg + 4 * h2 + i;
                float l = t < t_end ? S[h2][i] * p.sm_log2 : kNegInf;
                pr[4 * h2 + i] = l;
                bm = fmaxf(bm, l);
            }
        bm = xor_max16_32(bm);
        const float mnew = fmaxf(m, bm);
        const float alpha = fast_exp2(m - mnew);
        m = mnew;
        float psum = 0.0f;
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            pr[k] = fast_exp2(pr[k] - mnew);
            psum += pr[k];
        }
        lsum = lsum * alpha + psum;
#pragma unroll
        for (int mb = 0; mb < NMB; ++mb)
            oacc[mb] *= alpha;

        // ------------------------------------------------ values
        if (ring_split) {
            float pv[8];
#pragma unroll
            for (int e = 0; e < 8; ++e)
                pv[e] = pr[perm4(e)];
            half8 ph, pl;
            split_half8(pv, &ph, &pl);
#pragma unroll
            for (int mb = 0; mb < NMB; ++mb) {
                int d = 16 * mb + hh;
                half8 a;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    int t = t0 + 8 * qg + perm4(e);
                    uint16_t raw = 0;
                    if (t < t_end)
                        raw = p.vr[((size_t)unit * p.ring + (size_t)(t % p.ring)) * D + d];
                    a[e] = __builtin_bit_cast(_Float16, raw);
                }
                oacc[mb] = mfma16(a, ph, oacc[mb]);
                oacc[mb] = mfma16(a, pl, oacc[mb]);
            }
        } else {
            // O^T[d][h] += sum_t c[t][d] (p_t s_t) + sum_t p_t z_t, per V group.
            const int t8 = t0 + 8 * qg - ta;  // split-relative
            half8 ph, pl;
            float zp = 0.0f;
#pragma unroll
            for (int mb = 0; mb < NMB; ++mb) {
                if ((16 * mb) % p.v_group == 0) {
                    int g = (16 * mb) / p.v_group;
                    float pv[8], po[8];
                    float c2 = 0.0f;
#pragma unroll
                    for (int k = 0; k < 8; ++k) {
                        int mi = (t8 + k) * vng + g;
                        pv[k] = pr[k] * lvs[mi];
                        if (vaff)
                            c2 += pr[k] * lvz[mi];
                    }
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        po[e] = pv[perm4(e)];
                    split_half8(po, &ph, &pl);
                    zp = vaff ? xor_sum16_32(c2) : 0.0f;
                }
                int d = 16 * mb + hh;
                half8 a = codes_to_half8<VBITS>(value_code_word<VBITS>(lvc, D, t8, d), vbias);
                oacc[mb] = mfma16(a, ph, oacc[mb]);
                oacc[mb] = mfma16(a, pl, oacc[mb]);
                if (vaff)
                    oacc[mb] += zp;
            }
        }
    }

    // ---- merge the four waves of this split in LDS.
    // The merge area overlaps the query staging area, which other waves may
    // still be reading: wait for every wave to leave the block loop first.
    lsum = xor_sum16_32(lsum);
    __syncthreads();
    const int G = p.G;
    float* lm = lds;                       // [4][16] running max per wave and head
    float* ll = lds + kWaves * 16;         // [4][16] softmax sums
    float* lo = lds + 2 * kWaves * 16;     // [4][G][D] unnormalized outputs
    float* xo = lo;  // [G][D] result: element idx is written after its own four reads
    if (qg == 0) {
        lm[wave * 16 + hh] = m;
        ll[wave * 16 + hh] = lsum;
    }
    if (hh < G) {
#pragma unroll
        for (int mb = 0; mb < NMB; ++mb)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                lo[((size_t)wave * G + hh) * D + 16 * mb + 4 * qg + i] = oacc[mb][i];
    }
    __syncthreads();
    const bool single = p.S_tot == 1;
    const size_t row0 = (size_t)b * p.H_q + (size_t)j * G;
    for (int idx = threadIdx.x; idx < G * D; idx += kThreads) {
        int h = idx / D, d = idx % D;
        float M = kNegInf;
        for (int w = 0; w < kWaves; ++w)
            M = fmaxf(M, lm[w * 16 + h]);
        float acc = 0.0f, L = 0.0f;
        if (M != kNegInf) {
            for (int w = 0; w < kWaves; ++w) {
                float sc = fast_exp2(lm[w * 16 + h] - M);
                acc += sc * lo[((size_t)w * G + h) * D + d];
                L += sc * ll[w * 16 + h];
            }
        }
        if (single) {
            xo[idx] = acc / L;
        } else {
            size_t row = row0 + h;
            p.part_o[(row * p.S_tot + split) * D + d] = acc;
            if (d == 0) {
                p.part_ml[(row * p.S_tot + split) * 2 + 0] = M;
                p.part_ml[(row * p.S_tot + split) * 2 + 1] = L;
            }
        }
    }
    if (!single)
        return;  // the merge kernel finishes
    __syncthreads();
    finish_rows<D>(p, xo, row0, G);
}

template <int D, int KBITS, int VBITS, bool PERCH>
__global__ __launch_bounds__(kThreads) void decode_split_kernel(AttnParams p)
{
    extern __shared__ float lds[];
    run_split<D, KBITS, VBITS, PERCH>(p, lds);
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
    float* w = sm;                    // [G][S]: (max, sum) pairs, then weights
    float* xo = sm + 2 * G * S;       // [G][D]
    const float* ml = p.part_ml + row0 * S * 2;
    for (int idx = threadIdx.x; idx < 2 * G * S; idx += kThreads)
        w[idx] = ml[idx];
    __syncthreads();
    if (threadIdx.x < (unsigned)G) {
        float* r = w + 2 * S * threadIdx.x;
        float M = kNegInf;
        for (int s = 0; s < S; ++s)
            M = fmaxf(M, r[2 * s]);
        float L = 0.0f;
        for (int s = 0; s < S; ++s)
            L += r[2 * s] == kNegInf ? 0.0f : fast_exp2(r[2 * s] - M) * r[2 * s + 1];
        const float inv = 1.0f / L;
        for (int s = 0; s < S; ++s) {
            float m = r[2 * s];
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

template <int D, int KBITS, int VBITS, bool PERCH>
hipError_t launch_split(const AttnParams& p, hipStream_t stream)
{
    hipLaunchKernelGGL((decode_split_kernel<D, KBITS, VBITS, PERCH>), dim3(p.S_tot, p.B * p.H), dim3(kThreads),
                       p.lds_bytes, stream, p);
    return hipGetLastError();
}

template <int D>
hipError_t launch_decode_d(const AttnParams& p, hipStream_t stream)
{
    hipError_t e;
    const bool perch = p.k_axis == KVQ_PER_CHANNEL;
    if (p.k_bits == 4 && p.v_bits == 4 && !perch)
        e = launch_split<D, 4, 4, false>(p, stream);
    else if (p.k_bits == 4 && p.v_bits == 2 && !perch)
        e = launch_split<D, 4, 2, false>(p, stream);
    else if (p.k_bits == 2 && p.v_bits == 4 && !perch)
        e = launch_split<D, 2, 4, false>(p, stream);
    else if (p.k_bits == 2 && p.v_bits == 2 && !perch)
        e = launch_split<D, 2, 2, false>(p, stream);
    else if (p.k_bits == 4 && p.v_bits == 4)
        e = launch_split<D, 4, 4, true>(p, stream);
    else if (p.k_bits == 4 && p.v_bits == 2)
        e = launch_split<D, 4, 2, true>(p, stream);
    else if (p.k_bits == 2 && p.v_bits == 4)
        e = launch_split<D, 2, 4, true>(p, stream);
    else
        e = launch_split<D, 2, 2, true>(p, stream);
    if (e != hipSuccess || p.S_tot == 1)
        return e;
    hipLaunchKernelGGL(decode_merge_kernel<D>, dim3(p.B * p.H), dim3(kThreads),
                       (size_t)(2 * p.S_tot + D) * p.G * sizeof(float), stream, p);
    return hipGetLastError();
}

}  // namespace

// Split planning.  A split stages all its coded tokens in LDS, so its size
// is capped by kStageBytes; within that cap, aim for about kTargetGroups
// workgroups over the 256 compute units so several are resident per CU and
// one's loads overlap another's arithmetic.
constexpr int kTargetGroups = 512;

static int max_blocks_per_split(int D, const kvq_format& f)
{
    BlockBytes bb = block_bytes(D, f.k_bits, f.v_bits, f.k_axis, f.k_group, f.v_group, f.k_mode, f.v_mode);
    int m = kStageBytes / bb.total();
    return m < 1 ? 1 : m;
}

void decode_plan(int B, int H, int D, const kvq_format& f, int nq, int* S_q, int* bps)
{
    const int nblk = (nq + 31) / 32;
    const int units = B * H;
    const int s_want = (kTargetGroups + units - 1) / units;
    int per = (nblk + s_want - 1) / s_want;
    const int cap = max_blocks_per_split(D, f);
    if (per > cap)
        per = cap;
    if (per < 1)
        per = 1;
    *bps = per;
    *S_q = nblk == 0 ? 0 : (nblk + per - 1) / per;
}

int decode_split_bound(int B, int H, int D, const kvq_format& f, int nq)
{
    // S_q <= max(s_want, ceil(nblk / cap)) for every coded count up to nq.
    const int nblk = (nq + 31) / 32;
    const int units = B * H;
    const int s_want = (kTargetGroups + units - 1) / units;
    const int cap = max_blocks_per_split(D, f);
    const int by_cap = (nblk + cap - 1) / cap;
    int s = s_want > by_cap ? s_want : by_cap;
    return s < 1 ? 1 : s;
}

size_t decode_lds_bytes(int D, const kvq_format& f, int bps, int G, int* q_offset)
{
    // [stage of bps blocks][fp32 queries 16 x D]; the merge area reuses the front.
    BlockBytes bb = block_bytes(D, f.k_bits, f.v_bits, f.k_axis, f.k_group, f.v_group, f.k_mode, f.v_mode);
    size_t stage = ((size_t)bps * bb.total() + 15) / 16 * 16;
    *q_offset = (int)stage;
    size_t total = stage + 16 * (size_t)D * sizeof(float);
    size_t merge = (2 * kWaves * 16 + (size_t)kWaves * G * D) * sizeof(float);
    return total > merge ? total : merge;
}

hipError_t launch_decode(const AttnParams& p, int D, hipStream_t stream)
{
    switch (D) {
    case 64:
        return launch_decode_d<64>(p, stream);
    case 128:
        return launch_decode_d<128>(p, stream);
    case 256:
        return launch_decode_d<256>(p, stream);
    default:
        return hipErrorInvalidValue;
    }
}

}  // namespace kvq
