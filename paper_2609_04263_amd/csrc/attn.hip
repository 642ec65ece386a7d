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
// split writes an unnormalized partial (m, l, o) to the workspace and counts
// itself in a per-KV-head counter; the last split to arrive merges the
// partials, divides by the softmax sum, applies the inverse rotation, writes
// the outputs and resets the counter.  With a single split the partial is
// skipped.

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
__device__ __forceinline__ uint32_t value_code_word(const uint32_t* vc_unit, int T, int D, int t8, int d)
{
    // Eight codes along tokens: t = t8 .. t8 + 7 (t8 a multiple of 8), channel d.
    if (BITS == 4)
        return vc_unit[(size_t)(t8 >> 3) * D + d];
    return vc_unit[(size_t)(t8 >> 4) * D + d] >> (16 * ((t8 >> 3) & 1));
}

template <int D, int KBITS, int VBITS, bool PERCH>
__device__ void run_split(const AttnParams& p, float* lds)
{
    constexpr int NKB = D / 32;   // 32-wide K-blocks of the score MFMA
    constexpr int NMB = D / 16;   // 16-row M-blocks of the value MFMA
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int hh = lane & 15, qg = lane >> 4;
    const int split = blockIdx.x, unit = blockIdx.y;
    const int b = unit / p.H, j = unit % p.H;
    const bool ring_split = p.ring && split == p.S_q;

    // ---- queries: stage [16][D] fp32 (heads >= G zero), rotate if needed
    for (int idx = threadIdx.x; idx < 16 * D; idx += kThreads) {
        int h = idx / D, d = idx % D;
        float v = 0.0f;
        if (h < p.G)
            v = bf16_to_f32(p.q[((size_t)b * p.H_q + (size_t)j * p.G + h) * D + d]);
        lds[idx] = v;
    }
    __syncthreads();
    if (p.rotate) {
        for (int h = 1; h < D; h <<= 1) {
            for (int idx = threadIdx.x; idx < 16 * (D / 2); idx += kThreads) {
                int row = idx / (D / 2), k = idx % (D / 2);
                int jj = (k / h) * 2 * h + (k % h);
                float a = lds[row * D + jj], c = lds[row * D + jj + h];
                lds[row * D + jj] = a + c;
                lds[row * D + jj + h] = a - c;
            }
            __syncthreads();
        }
        for (int idx = threadIdx.x; idx < 16 * D; idx += kThreads)
            lds[idx] *= p.rot_c;
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
            qf[kb][e] = lds[hh * D + 32 * kb + 8 * qg + perm4(e)];
            part += qf[kb][e];
        }
        split_half8(qf[kb], &qhi[kb], &qlop[kb]);
        qsum[kb] = xor_sum16_32(part);
    }
    __syncthreads();  // lds is reused below

    const int T = p.T;
    const uint32_t* kc_unit = p.kc + (size_t)unit * T * (D * KBITS / 32);
    const uint32_t* vc_unit = p.vc + (size_t)unit * (T * VBITS / 32) * D;
    const int kng = D / p.k_group, vng = D / p.v_group;
    const bool kaff = p.k_mode == KVQ_AFFINE, vaff = p.v_mode == KVQ_AFFINE;
    const _Float16 kb16 = (_Float16)(1024 + (kaff ? 0 : (1 << (KBITS - 1))));
    const _Float16 vb16 = (_Float16)(1024 + (vaff ? 0 : (1 << (VBITS - 1))));
    const half2_t kbias = {kb16, kb16}, vbias = {vb16, vb16};

    float m = kNegInf, lsum = 0.0f;
    floatx4 oacc[NMB];
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb)
        oacc[mb] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};

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
                const uint32_t* krow = kc_unit + (size_t)tA * (D * KBITS / 32);
                const int tS = t0 + 8 * qg + 4 * h2;  // tokens of this lane's outputs: tS + i
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
                            size_t mi = ((size_t)unit * T + tS + i) * kng + g;
                            float s = p.ks[mi];
                            Sacc[i] += s * acc[i];
                            if (kaff)
                                Sacc[i] += p.kz[mi] * qs;
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
            const size_t meta = ((size_t)unit * (T / 32) + (size_t)(t0 / 32)) * D;
            half8 qkh[NKB], qkl[NKB];
            float c2 = 0.0f;
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb) {
                float qs[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    int d = 32 * kb + 8 * qg + perm4(e);
                    qs[e] = qf[kb][e] * p.ks[meta + d];
                    if (kaff)
                        c2 += qf[kb][e] * p.kz[meta + d];
                }
                split_half8(qs, &qkh[kb], &qkl[kb]);
            }
            const float zq = xor_sum16_32(c2);
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
                int tA = t0 + 8 * (hh >> 2) + 4 * h2 + (hh & 3);
                const uint32_t* krow = kc_unit + (size_t)tA * (D * KBITS / 32);
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
            const int t8 = t0 + 8 * qg;
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
                        size_t mi = ((size_t)unit * T + t8 + k) * vng + g;
                        pv[k] = pr[k] * p.vs[mi];
                        if (vaff)
                            c2 += pr[k] * p.vz[mi];
                    }
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        po[e] = pv[perm4(e)];
                    split_half8(po, &ph, &pl);
                    zp = vaff ? xor_sum16_32(c2) : 0.0f;
                }
                int d = 16 * mb + hh;
                half8 a = codes_to_half8<VBITS>(value_code_word<VBITS>(vc_unit, T, D, t8, d), vbias);
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
    float* xo = lo + (size_t)kWaves * G * D;  // [G][D] this workgroup's result
    int* flag = (int*)(xo + (size_t)G * D);
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
    if (!single) {
        // Publish this split's partial; the last split of the KV head to
        // arrive merges all of them (no workgroup ever waits for another).
        __threadfence();
        __syncthreads();
        if (threadIdx.x == 0) {
            unsigned prev = atomicAdd(&p.counters[unit], 1u);
            *flag = prev == (unsigned)(p.S_tot - 1);
        }
        __syncthreads();
        if (!*flag)
            return;
        __threadfence();
        for (int idx = threadIdx.x; idx < G * D; idx += kThreads) {
            int h = idx / D, d = idx % D;
            size_t row = row0 + h;
            const float* ml = p.part_ml + row * p.S_tot * 2;
            float M = kNegInf;
            for (int s = 0; s < p.S_tot; ++s)
                M = fmaxf(M, ml[2 * s]);
            float acc = 0.0f, L = 0.0f;
            for (int s = 0; s < p.S_tot; ++s) {
                float ms = ml[2 * s];
                if (ms == kNegInf)
                    continue;
                float sc = fast_exp2(ms - M);
                L += sc * ml[2 * s + 1];
                acc += sc * p.part_o[(row * p.S_tot + s) * D + d];
            }
            xo[idx] = acc / L;
        }
        if (threadIdx.x == 0)
            p.counters[unit] = 0u;  // ready for the next call
    }
    __syncthreads();
    // ---- inverse rotation (the normalized transform is its own inverse)
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
__global__ __launch_bounds__(kThreads) void decode_split_kernel(AttnParams p)
{
    extern __shared__ float lds[];
    run_split<D, KBITS, VBITS, PERCH>(p, lds);
}

template <int D, int KBITS, int VBITS, bool PERCH>
hipError_t launch_split(const AttnParams& p, hipStream_t stream)
{
    size_t lds_floats = 16 * D;
    size_t merge = 2 * kWaves * 16 + (size_t)(kWaves + 1) * p.G * D + 1;
    if (merge > lds_floats)
        lds_floats = merge;
    hipLaunchKernelGGL((decode_split_kernel<D, KBITS, VBITS, PERCH>), dim3(p.S_tot, p.B * p.H), dim3(kThreads),
                       lds_floats * sizeof(float), stream, p);
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
    return e;
}

}  // namespace

// Aim for about 2048 workgroups over the 256 compute units, with at least
// two 32-token blocks per wave (8 per split) so the loop can pipeline.
static int split_target(int B, int H, int nblk)
{
    const int units = B * H;
    int want = (2048 + units - 1) / units;
    int max_splits = (nblk + 7) / 8;
    int s = want < max_splits ? want : max_splits;
    return s < 1 ? 1 : s;
}

int decode_split_bound(int B, int H, int nq)
{
    return split_target(B, H, (nq + 31) / 32);  // non-decreasing in nq
}

void decode_plan(int B, int H, int nq, int* S_q, int* bps)
{
    const int nblk = (nq + 31) / 32;
    const int s = split_target(B, H, nblk);
    int per = (nblk + s - 1) / s;
    if (per < 1)
        per = 1;
    *bps = per;
    *S_q = nblk == 0 ? 0 : (nblk + per - 1) / per;
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
