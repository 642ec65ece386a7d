// Quantize-and-pack append into the physically packed incremental cache
// (Sec. 3.1 of the paper: new key/value states are coded with Eq. (3) or the
// symmetric control, bit-packed and appended; KIVI keeps an fp16 window).
//
// Bit-exactness: codes and metadata must equal the CPU reference bit for
// bit, so this file is compiled with -ffp-contract=off and the coder takes
// exactly the reference's IEEE binary32 steps: subtract, correctly rounded
// divide, round half to even, clamp (the rounded quotient comes from a
// reciprocal product wherever that provably gives the same code; see
// rint_quotient).  Min/max are exact.
//
// One workgroup (256 threads) codes one aligned block of 32 tokens of one
// (sequence, KV head): the block's K rows are staged in LDS as fp32 (rotated
// by the fixed Hadamard butterflies when the format rotates, rounded to fp16
// when a window exists), group statistics are reduced per (token, group) or
// per channel, and every output piece (eight codes) is assembled by one
// thread.  V rows follow through the same LDS buffer.  V codes are packed
// along tokens: a piece shared with tokens outside the block range keeps
// earlier tokens' bits and clears later ones, so the image is independent of
// call boundaries.
//
// Pieces are stored in the order the decode kernel consumes them (per
// 32-token block, a 64-lane MFMA layout; see include/kvq.h): token tau of a
// block is row 4 (tau / 8) + tau % 4 of half (tau / 4) % 2, and the lane of
// key piece P is row + 16 (P % 4); value piece (octet o, channel d) belongs
// to lane d % 16 + 16 o.

#include "coder.h"
#include "kvq_device.h"
#include "kvq_internal.h"

namespace kvq {
namespace {

constexpr int kThreads = 256;
constexpr int kBlockTok = 32;

// Index of key piece P (channels 8P..8P+7) of position tau in block `blk`
// (blk counted over the whole section: unit * NB + block).
template <int D>
__device__ __forceinline__ size_t key_piece(size_t blk, int tau, int P)
{
    const int row = 4 * (tau >> 3) + (tau & 3), half = (tau >> 2) & 1;
    return ((blk * 2 + half) * 64 + row + 16 * (P & 3)) * (D / 32) + (P >> 2);
}

// Index of value piece (octet o of the block, channel d).
template <int D>
__device__ __forceinline__ size_t value_piece(size_t blk, int o, int d)
{
    return (blk * 64 + (d & 15) + 16 * o) * (D / 16) + (d >> 4);
}

// Fixed normalized Hadamard transform of `rows` rows of D fp32 values in LDS:
// butterflies with half-width 1, 2, ..., D/2 then one multiply by c.  Rows
// with use[row] == 0 are left untouched.
template <int D>
__device__ void fwht_rows(float* xs, int rows, const int* use, float c)
{
    for (int h = 1; h < D; h <<= 1) {
        for (int idx = threadIdx.x; idx < rows * (D / 2); idx += kThreads) {
            int row = idx / (D / 2), k = idx % (D / 2);
            if (!use[row])
                continue;
            int j = (k / h) * 2 * h + (k % h);
            float a = xs[row * D + j], b = xs[row * D + j + h];
            xs[row * D + j] = a + b;
            xs[row * D + j + h] = a - b;
        }
        __syncthreads();
    }
    for (int idx = threadIdx.x; idx < rows * D; idx += kThreads)
        if (use[idx / D])
            xs[idx] = xs[idx] * c;
    __syncthreads();
}

// Staging of the block's rows of K (which = 0) or V (which = 1) as the coder
// sees them.  Row i is token tb + i; rows outside [q0, q1) are zero.  Thread
// j moves eight channels of one row per step (one 16-byte load); the D / 8
// threads of a row are consecutive lanes of one wave.
template <int D>
struct RowStage {
    static constexpr int kSteps = kBlockTok * (D / 8) / kThreads;
    static_assert(kSteps >= 1 && kBlockTok * (D / 8) % kThreads == 0, "uniform staging steps");
    u32x4 w[kSteps];

    __device__ static int row(int k) { return ((int)threadIdx.x + kThreads * k) / (D / 8); }
    __device__ static int chan(int k) { return 8 * (((int)threadIdx.x + kThreads * k) % (D / 8)); }

    // Issue the loads (bf16 input for tokens of this call, fp16 window slots
    // for tokens appended earlier).
    __device__ void load(const AppendParams& p, int which, int b, int h, int tb)
    {
        const uint16_t* in = which ? p.vin : p.kin;
        const uint16_t* ring = which ? p.vr : p.kr;
#pragma unroll
        for (int k = 0; k < kSteps; ++k) {
            const int t = tb + row(k), d8 = chan(k);
            w[k] = u32x4{0u, 0u, 0u, 0u};
            if (t >= p.q0 && t < p.q1)
                w[k] = t >= p.n0 ? *(const u32x4*)(in + (((size_t)b * p.n_new + (t - p.n0)) * p.H + h) * D + d8)
                                 : *(const u32x4*)(ring + (((size_t)b * p.H + h) * p.ring + t % p.ring) * D + d8);
        }
    }

    // Widen to fp32; for tokens of this call, rotate (the butterflies of
    // fwht_rows: half widths 1, 2, 4 inside a thread's eight values, 8 .. D/2
    // across lanes, then one multiply by rot_c) and round to fp16 when a
    // window exists; store() writes the rows to xs.  Every butterfly adds or
    // subtracts the same two values as the serial transform, so results are
    // identical.
    __device__ void store(const AppendParams& p, int tb, float* xs) const
    {
#pragma unroll
        for (int k = 0; k < kSteps; ++k) {
            float v[8];
            widen(p, tb, k, v);
            float* dst = xs + row(k) * D + chan(k);
            *(float4*)dst = make_float4(v[0], v[1], v[2], v[3]);
            *(float4*)(dst + 4) = make_float4(v[4], v[5], v[6], v[7]);
        }
    }

    // The eight values of step k as the coder sees them.
    __device__ __forceinline__ void widen(const AppendParams& p, int tb, int k, float* v) const
    {
        {
            const int t = tb + row(k);
            const bool fresh = !(t >= p.q0 && t < p.q1) || t >= p.n0;  // bf16 (zero rows: zero words)
            const uint32_t ww[4] = {w[k].x, w[k].y, w[k].z, w[k].w};
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                if (fresh) {
                    v[2 * q] = __uint_as_float(ww[q] << 16);
                    v[2 * q + 1] = __uint_as_float(ww[q] & 0xFFFF0000u);
                } else {
                    v[2 * q] = f16_bits_to_f32((uint16_t)ww[q]);
                    v[2 * q + 1] = f16_bits_to_f32((uint16_t)(ww[q] >> 16));
                }
            }
            const bool input = t >= p.q0 && t < p.q1 && t >= p.n0;
            if (p.rotate) {
                float r[8];
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    r[e] = v[e];
#pragma unroll
                for (int hw = 1; hw < 8; hw <<= 1) {
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        if (e & hw)
                            continue;
                        const float a = r[e], c = r[e + hw];
                        r[e] = a + c;
                        r[e + hw] = a - c;
                    }
                }
                const int lane_bits = chan(k) >> 3;  // this thread's piece index within the row
#pragma unroll
                for (int hl = 1; hl < D / 8; hl <<= 1) {
                    const bool upper = (lane_bits & hl) != 0;
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const float other = __shfl_xor(r[e], hl);
                        r[e] = upper ? other - r[e] : r[e] + other;
                    }
                }
                if (input) {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        v[e] = r[e] * p.rot_c;
                }
            }
            if (p.ring && input) {
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    v[e] = f16_bits_to_f32(f32_to_f16_bits(v[e]));
            }
        }
    }
};

// 16-byte copy of `bytes` (a multiple of 16) from LDS to global memory.
__device__ __forceinline__ void copy_out(const uint8_t* src, uint8_t* dst, int bytes)
{
    for (int off = 16 * (int)threadIdx.x; off < bytes; off += 16 * kThreads)
        *(u32x4*)(dst + off) = *(const u32x4*)(src + off);
}

// One workgroup per (32-token block, sequence and KV head).  Per-token
// groups: each thread takes the eight channels of one piece, the group's
// statistics are reduced across the group's lanes, and the thread codes its
// piece (keys: a piece as is; values: bytes, then packed along tokens).
// Per-channel keys: one thread per channel over the block.  A block that
// this call writes whole is assembled in LDS and stored with contiguous
// 16-byte stores (each section holds a block's bytes as one range); a block
// shared with earlier or later calls is written piece by piece.
template <int D, bool PERCH>
__global__ __launch_bounds__(kThreads) void append_code_kernel(AppendParams p)
{
    __shared__ __attribute__((aligned(16))) float xs[PERCH ? kBlockTok * D : 4];  // per-channel keys only
    __shared__ __attribute__((aligned(16))) uint8_t vcode[kBlockTok * D];  // value codes [token][D]
    __shared__ __attribute__((aligned(16))) uint8_t ob[kBlockTok * D];     // a block's pieces (<= 8-bit codes)
    __shared__ __attribute__((aligned(16))) float mb[2][kBlockTok * 8];    // its scales, offsets (<= 1 KB each)
    __shared__ float ms[D];
    __shared__ float mz[D];
    static_assert(kBlockTok * 8 >= D, "per-channel metadata fits the staging buffer");

    const int unit = blockIdx.y;
    const int b = unit / p.H, h = unit % p.H;
    const int tb = (p.q0 / kBlockTok + (int)blockIdx.x) * kBlockTok;
    const int lo = max(p.q0, tb), hi = min(p.q1, tb + kBlockTok);
    const bool full = lo == tb && hi == tb + kBlockTok;
    const size_t bh = (size_t)unit;
    const int msz = p.meta16 ? 2 : 4;

    // ------------------------------------------------------------ keys
    const size_t blk = bh * (size_t)(p.T / kBlockTok) + (size_t)(tb / kBlockTok);
    RowStage<D> kst, vst;
    kst.load(p, 0, b, h, tb);
    vst.load(p, 1, b, h, tb);  // in flight while the keys are coded
    if constexpr (PERCH) {
        kst.store(p, tb, xs);
        __syncthreads();
    }
    const int kb = p.k_bits;
    constexpr int PPT = D / 8;  // pieces per token
    float* kss = full ? mb[0] : p.ks;  // where scales and offsets go, and their block base
    float* kzs = full ? mb[1] : p.kz;
    void* kcs = full ? (void*)ob : (void*)p.kc;
    const size_t kcb = full ? 0 : blk;
    int kmeta;  // metadata elements per block
    if constexpr (!PERCH) {
        const int lanes = p.k_group / 8, ng = D / p.k_group;
        kmeta = ng * kBlockTok;
        const size_t mbase = full ? 0 : blk * (size_t)kmeta;
#pragma unroll
        for (int k = 0; k < RowStage<D>::kSteps; ++k) {
            const int i = RowStage<D>::row(k), P = RowStage<D>::chan(k) / 8, t = tb + i;
            float x[8];
            kst.widen(p, tb, k, x);
            float s, z;
            piece_group_stats(x, lanes, p.k_mode, kb, &s, &z);
            round_meta(p.meta16, &s, &z);
            if (t < lo || t >= hi)
                continue;
            if (P % lanes == 0) {
                const size_t mi = mbase + (size_t)(P / lanes) * kBlockTok + i;
                store_meta(kss, mi, s, p.meta16);
                if (p.k_mode == KVQ_AFFINE)
                    store_meta(kzs, mi, z, p.meta16);
            }
            const float r = __builtin_amdgcn_rcpf(s);
            uint64_t word = 0;
#pragma unroll
            for (int e = 0; e < 8; ++e)
                word |= (uint64_t)code_one(x[e], s, r, z, p.k_mode, kb) << (kb * e);
            store_piece(kcs, key_piece<D>(kcb, i, P), kb, word);
        }
    } else {
        // Per-channel keys: the block is one whole 32-token group.
        kmeta = D;
        const size_t mbase = full ? 0 : blk * (size_t)D;
        for (int d = threadIdx.x; d < D; d += kThreads) {
            float s, z;
            group_stats(xs + d, D, kBlockTok, p.k_mode, kb, &s, &z);
            round_meta(p.meta16, &s, &z);
            ms[d] = s;
            mz[d] = z;
            store_meta(kss, mbase + d, s, p.meta16);
            if (p.k_mode == KVQ_AFFINE)
                store_meta(kzs, mbase + d, z, p.meta16);
        }
        __syncthreads();
        for (int idx = threadIdx.x; idx < kBlockTok * PPT; idx += kThreads) {
            int i = idx / PPT, P = idx % PPT;
            uint64_t word = 0;
            for (int e = 0; e < 8; ++e) {
                int d = 8 * P + e;
                word |= (uint64_t)code_one(xs[i * D + d], ms[d], __builtin_amdgcn_rcpf(ms[d]), mz[d], p.k_mode, kb)
                        << (kb * e);
            }
            store_piece(kcs, key_piece<D>(kcb, i, P), kb, word);
        }
    }
    __syncthreads();
    if (full) {
        copy_out(ob, (uint8_t*)p.kc + blk * (size_t)(4 * D * kb), 4 * D * kb);
        copy_out((const uint8_t*)mb[0], (uint8_t*)p.ks + blk * (size_t)(kmeta * msz), kmeta * msz);
        if (p.k_mode == KVQ_AFFINE)
            copy_out((const uint8_t*)mb[1], (uint8_t*)p.kz + blk * (size_t)(kmeta * msz), kmeta * msz);
    }

    // ---------------------------------------------------------- values
    __syncthreads();  // the key copies have read ob and mb
    const int vb = p.v_bits;
    const int vlanes = p.v_group / 8, vmeta = (D / p.v_group) * kBlockTok;
    {
        float* vss = full ? mb[0] : p.vs;
        float* vzs = full ? mb[1] : p.vz;
        const size_t mbase = full ? 0 : blk * (size_t)vmeta;
#pragma unroll
        for (int k = 0; k < RowStage<D>::kSteps; ++k) {
            const int i = RowStage<D>::row(k), P = RowStage<D>::chan(k) / 8, t = tb + i;
            float x[8];
            vst.widen(p, tb, k, x);
            float s, z;
            piece_group_stats(x, vlanes, p.v_mode, vb, &s, &z);
            round_meta(p.meta16, &s, &z);
            if (t >= lo && t < hi && P % vlanes == 0) {
                const size_t mi = mbase + (size_t)(P / vlanes) * kBlockTok + i;
                store_meta(vss, mi, s, p.meta16);
                if (p.v_mode == KVQ_AFFINE)
                    store_meta(vzs, mi, z, p.meta16);
            }
            const float r = __builtin_amdgcn_rcpf(s);
            uint32_t c[8];
#pragma unroll
            for (int e = 0; e < 8; ++e)
                c[e] = code_one(x[e], s, r, z, p.v_mode, vb);
            *(uint2*)(vcode + i * D + 8 * P) =
                make_uint2(c[0] | (c[1] << 8) | (c[2] << 16) | (c[3] << 24), c[4] | (c[5] << 8) | (c[6] << 16) | (c[7] << 24));
        }
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < (kBlockTok / 8) * D; idx += kThreads) {
        int o = idx / D, d = idx % D;
        int tfirst = tb + 8 * o;
        if (tfirst + 8 <= lo || tfirst >= hi)
            continue;
        uint64_t word = 0;
        if (tfirst < lo) {  // keep the bits of tokens appended earlier (never in a full block)
            int keep_n = lo - tfirst;
            word = load_piece(p.vc, value_piece<D>(blk, o, d), vb) & low_codes(vb, keep_n);
        }
        for (int e = 0; e < 8; ++e) {
            int t = tfirst + e;
            if (t < lo || t >= hi)
                continue;
            word |= (uint64_t)vcode[(t - tb) * D + d] << (vb * e);
        }
        if (full)
            store_piece(ob, value_piece<D>(0, o, d), vb, word);
        else
            store_piece(p.vc, value_piece<D>(blk, o, d), vb, word);
    }
    if (full) {
        __syncthreads();
        copy_out(ob, (uint8_t*)p.vc + blk * (size_t)(4 * D * vb), 4 * D * vb);
        copy_out((const uint8_t*)mb[0], (uint8_t*)p.vs + blk * (size_t)(vmeta * msz), vmeta * msz);
        if (p.v_mode == KVQ_AFFINE)
            copy_out((const uint8_t*)mb[1], (uint8_t*)p.vz + blk * (size_t)(vmeta * msz), vmeta * msz);
    }
}

// One decoded token per (sequence, KV head) without a window: a workgroup of
// D threads, thread d owning channel d of the token's K and V.  Every load
// (the token's K and V, and the value piece it shares with earlier tokens)
// is issued first; the rotation runs as the same butterflies as fwht_rows;
// group statistics are all-reduced across the group's threads (min, max and
// max-magnitude are exact in any order, so they equal the block kernel's),
// then each thread codes its channel, key pieces are OR-reduced over eight
// lanes and each value piece is merged with the bits of earlier tokens.
template <int D>
__device__ __forceinline__ float group_reduce(float v, int g, bool is_max, float* red, int slot)
{
    const int lanes = g < 64 ? g : 64;
    for (int off = 1; off < lanes; off <<= 1) {
        const float o = __shfl_xor(v, off);
        v = is_max ? fmaxf(v, o) : fminf(v, o);
    }
    if (g > 64) {
        // one value per wave, combined over the g / 64 waves of the group
        const int wave = threadIdx.x >> 6;
        if ((threadIdx.x & 63) == 0)
            red[slot * 4 + wave] = v;
        __syncthreads();
        const int w0 = (wave / (g / 64)) * (g / 64);
        v = red[slot * 4 + w0];
        for (int w = 1; w < g / 64; ++w)
            v = is_max ? fmaxf(v, red[slot * 4 + w0 + w]) : fminf(v, red[slot * 4 + w0 + w]);
    }
    return v;
}

template <int D>
__global__ __launch_bounds__(D) void append_token_kernel(AppendParams p)
{
    __shared__ float xs[2][D];
    __shared__ float red[8 * 4];
    const int unit = blockIdx.x, b = unit / p.H, h = unit % p.H, d = threadIdx.x;
    const int t = p.n0, tau = t & 31, j = t & 7;
    const size_t blk = (size_t)unit * (p.T / kBlockTok) + (size_t)(t / kBlockTok);
    const size_t vpi = value_piece<D>(blk, tau >> 3, d);
    const size_t in = ((size_t)b * p.H + h) * D + d;  // n_new == 1
    float x[2] = {bf16_to_f32(p.kin[in]), bf16_to_f32(p.vin[in])};
    const uint64_t old = load_piece(p.vc, vpi, p.v_bits);
    if (p.rotate) {
        xs[0][d] = x[0];
        xs[1][d] = x[1];
        __syncthreads();
        for (int hw = 1; hw < D; hw <<= 1) {
            float nv[2];
#pragma unroll
            for (int w = 0; w < 2; ++w)
                nv[w] = (d & hw) ? xs[w][d - hw] - xs[w][d] : xs[w][d] + xs[w][d + hw];
            __syncthreads();
            xs[0][d] = nv[0];
            xs[1][d] = nv[1];
            __syncthreads();
        }
        x[0] = xs[0][d] * p.rot_c;
        x[1] = xs[1][d] * p.rot_c;
    }
#pragma unroll
    for (int w = 0; w < 2; ++w) {
        const int mode = w ? p.v_mode : p.k_mode, bits = w ? p.v_bits : p.k_bits;
        const int g = w ? p.v_group : p.k_group, gi = d / g, ng = D / g;
        float s, z;
        if (mode == KVQ_AFFINE) {
            const float mn = group_reduce<D>(x[w], g, false, red, 2 * w);
            const float mx = group_reduce<D>(x[w], g, true, red, 2 * w + 1);
            const float top = (float)((1 << bits) - 1);
            s = (mx - mn) / top;
            if (!(s >= 1e-8f))
                s = 1e-8f;
            z = mn + 0.0f;  // canonical +0 for a signed-zero minimum
        } else {
            const float ma = group_reduce<D>(fabsf(x[w]), g, true, red, 2 * w);
            const float qmax = (float)((1 << (bits - 1)) - 1);
            s = ma / qmax;
            if (!(s >= 1e-8f))
                s = 1e-8f;
            z = 0.0f;
        }
        round_meta(p.meta16, &s, &z);
        const uint32_t c = code_one(x[w], s, __builtin_amdgcn_rcpf(s), z, mode, bits);
        if (d % g == 0) {
            const size_t mi = (blk * ng + gi) * kBlockTok + tau;
            store_meta(w ? p.vs : p.ks, mi, s, p.meta16);
            if (mode == KVQ_AFFINE)
                store_meta(w ? p.vz : p.kz, mi, z, p.meta16);
        }
        if (w == 0) {
            // key piece d / 8: codes of channels 8P .. 8P + 7 at bits k_bits e,
            // OR-reduced as two 32-bit halves
            const uint64_t mine = (uint64_t)c << (bits * (d & 7));
            uint32_t lo32 = (uint32_t)mine, hi32 = (uint32_t)(mine >> 32);
#pragma unroll
            for (int off = 1; off < 8; off <<= 1) {
                lo32 |= __shfl_xor(lo32, off);
                hi32 |= __shfl_xor(hi32, off);
            }
            if ((d & 7) == 0)
                store_piece(p.kc, key_piece<D>(blk, tau, d >> 3), bits, ((uint64_t)hi32 << 32) | lo32);
        } else {
            const uint64_t keep = low_codes(bits, j);
            store_piece(p.vc, vpi, bits, (old & keep) | ((uint64_t)c << (bits * j)));
        }
    }
}

// fp16 window: slot t mod (R + F) <- fp16 of token t (rotated first when
// the format rotates), for t in [ring_lo, n0 + n_new).  Runs after the coder
// of the same call, which may still read the slots being replaced.  The
// sink rows are written by the same kernel with ring = sink (slot t).
template <int D>
__global__ __launch_bounds__(kThreads) void append_ring_kernel(AppendParams p)
{
    __shared__ float xs[2 * D];
    __shared__ int use[2];
    const int unit = blockIdx.y;
    const int b = unit / p.H, h = unit % p.H;
    const int t = p.ring_lo + (int)blockIdx.x;
    for (int idx = threadIdx.x; idx < 2 * D; idx += kThreads) {
        int which = idx / D, d = idx % D;
        const uint16_t* in = which ? p.vin : p.kin;
        xs[idx] = bf16_to_f32(in[(((size_t)b * p.n_new + (t - p.n0)) * p.H + h) * D + d]);
    }
    if (threadIdx.x < 2)
        use[threadIdx.x] = 1;
    __syncthreads();
    if (p.rotate)
        fwht_rows<D>(xs, 2, use, p.rot_c);
    for (int idx = threadIdx.x; idx < 2 * D; idx += kThreads) {
        int which = idx / D, d = idx % D;
        uint16_t* ring = which ? p.vr : p.kr;
        ring[(((size_t)b * p.H + h) * p.ring + t % p.ring) * D + d] = f32_to_f16_bits(xs[idx]);
    }
}

template <int D>
hipError_t launch_append_d(const AppendParams& p, hipStream_t stream)
{
    const int units = p.B * p.H;
    if (p.n_new == 1 && p.ring == 0 && p.k_axis == KVQ_PER_TOKEN) {
        launch_kernel(append_token_kernel<D>, dim3(units), dim3(D), 0, stream, p);
        return hipGetLastError();
    }
    if (p.q1 > p.q0) {
        const int nblk = (p.q1 + kBlockTok - 1) / kBlockTok - p.q0 / kBlockTok;
        if (p.k_axis == KVQ_PER_CHANNEL)
            launch_kernel((append_code_kernel<D, true>), dim3(nblk, units), dim3(kThreads), 0, stream, p);
        else
            launch_kernel((append_code_kernel<D, false>), dim3(nblk, units), dim3(kThreads), 0, stream, p);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess)
            return e;
    }
    int n1 = p.n0 + p.n_new;
    if (p.ring && n1 > p.ring_lo) {
        launch_kernel(append_ring_kernel<D>, dim3(n1 - p.ring_lo, units), dim3(kThreads), 0, stream, p);
        return hipGetLastError();
    }
    return hipSuccess;
}

template <int D>
hipError_t launch_rows_d(const AppendParams& p, int hi, hipStream_t stream)
{
    if (hi > p.ring_lo)
        launch_kernel(append_ring_kernel<D>, dim3(hi - p.ring_lo, p.B * p.H), dim3(kThreads), 0, stream, p);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_append_rows(const AppendParams& p, int D, int hi, hipStream_t stream)
{
    switch (D) {
    case 64:
        return launch_rows_d<64>(p, hi, stream);
    case 128:
        return launch_rows_d<128>(p, hi, stream);
    case 256:
        return launch_rows_d<256>(p, hi, stream);
    default:
        return hipErrorInvalidValue;
    }
}

hipError_t launch_append(const AppendParams& p, int D, hipStream_t stream)
{
    switch (D) {
    case 64:
        return launch_append_d<64>(p, stream);
    case 128:
        return launch_append_d<128>(p, stream);
    case 256:
        return launch_append_d<256>(p, stream);
    default:
        return hipErrorInvalidValue;
    }
}

}  // namespace kvq
