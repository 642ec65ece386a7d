// Chunked prefill attention over the packed cache (Sec. 3.1: evaluation
// runs chunk by chunk; the chunk's states are coded and appended, then its
// queries attend causally over the reconstruction of everything stored).
//
// Two launches per group of (sequence, KV head) units:
//   1. dequant_kernel reconstructs every visible 32-token block of a unit
//      once into a workspace "block image" (192 D bytes): k_hat in fp32
//      stored as fp16 hi + lo (hi + lo carries ~22 bits) as [token][D] rows,
//      v_hat as fp16 transposed [D][32 key slots].  A block of per-token
//      key groups whose tokens are all coded (a "code block") keeps the key
//      codes instead, as exact fp16 values, with the groups' scales and
//      offsets in place of the lo half.  A rotating format's value rows are
//      rotated back to the original basis first (an fp32 FWHT per token in
//      LDS), so the outputs need no inverse rotation.  The image is laid
//      out exactly as the attention kernel reads it from LDS (16-byte
//      chunks xor-swizzled by row so that the fragment reads are free of
//      bank conflicts), so it moves to LDS with plain linear copies.
//   2. attn_kernel: one workgroup per (unit, tile of query rows); query rows
//      are the (chunk token, head of the KV group) pairs in token-major
//      order.  Each of the eight waves owns 16 QN query rows (128 / 256 / 512
//      rows per workgroup at D = 256 / 128 / 64).  Block images stream into
//      a ring of LDS stages with global_load_lds_dwordx4 (no registers, no
//      vector work), several blocks ahead, and per block:
//      - scores S^T = K Q^T with v_mfma_f32_16x16x32_f16 (keys as rows,
//        query rows as columns).  A bf16 query of a non-rotating format,
//        scaled by a power of two, is exact in fp16 (K hi x q + K lo x q);
//        a rotated query (rotated in fp32 in LDS) is split into fp16 hi +
//        lo (three products).  The softmax runs in base 2, online per
//        column (the running maximum moves only in steps of more than 2^8);
//        for a code block S = sum_g s_g (c_g . q_g) + z'_g sum q_g with
//        exact products c q and one fp32 scaling of each group's score
//        tile (the offset terms, at D = 256 with four key groups, as one
//        fp32 MFMA per key tile);
//      - O^T += V^T P^T in fp16 (probabilities in [0, 2^8] and values each
//        carry an 11-bit relative rounding; the logits are the
//        precision-critical product).  A lane holds score rows 4 q + i of
//        the block's two 16-key tiles, which are exactly the eight k-slots
//        8 q .. 8 q + 7 its next MFMA operand needs when the keys of slot
//        8 q + e are taken as 4 q + e (e < 4) and 16 + 4 q + e - 4; the
//        image stores V^T in that key order, so probabilities never cross
//        lanes and a value operand is one read.
// Reconstructing once per unit instead of once per query tile is what the
// workspace buys: a 2048-token chunk has 4096 query rows per KV head at
// grouping 2, i.e. 32 tiles that would each rebuild every block.
// Sink tokens (fp16 rows) come first as blocks of their own, so every query
// row holds a finite running maximum before the coded tail; fp16 window
// tokens past the coded ones are copied into the image from the ring.

#include "kvq_internal.h"
#include "kvq_device.h"

namespace kvq {
namespace pre {

constexpr int kDqThreads = 256;

// Waves per attention workgroup: eight (one workgroup per CU, two waves per
// SIMD), four at D = 64, where two workgroups share a CU (each SIMD holds
// one wave of each, with independent per-block barriers) and a tile has
// half the rows, so that the grid divides the work more finely: tiny_b16
// 6.5% faster; at D = 128 the same was 1% slower (llama8b_had) or equal.
template <int D>
constexpr int waves()
{
    return D == 64 ? 4 : 8;
}

template <int D>
constexpr int threads()
{
    return 64 * waves<D>();
}

// query rows per wave (16 QN): the accumulators take D QN / 4 registers
template <int D>
constexpr int qn()
{
    return D == 64 ? 4 : D == 128 ? 2 : 1;
}

template <int D>
constexpr int rows_per_tile()
{
    return waves<D>() * 16 * qn<D>();
}

// One reconstructed 32-token block: K hi [32][D], K lo [32][D] (fp16), then
// V^T [D][32] (fp16), 192 D bytes.  A rotating format's values are rotated
// back (an fp32 FWHT per token) before they are rounded, so the outputs need
// no inverse rotation and every output element carries the rounding of one
// channel's values, as without rotation.
template <int D>
__host__ __device__ constexpr int image_bytes()
{
    return 192 * D;
}

// Byte offsets in an image of the K lo half (or a code block's scales and
// offsets) and of V^T.
template <int D>
__host__ __device__ constexpr int klo_at()
{
    return 64 * D;
}

template <int D>
__host__ __device__ constexpr int vt_at()
{
    return 128 * D;
}

// LDS ring depth (block images in flight)
template <int D>
constexpr int stages()
{
    return D == 128 ? 4 : 3;
}

// LDS: the ring, or the query / output staging [rows][D] fp32 when larger
// (both are used by the same workgroup at different times).
template <int D>
constexpr size_t attn_lds_bytes()
{
    constexpr size_t ring = (size_t)stages<D>() * image_bytes<D>();
    constexpr size_t rows = (size_t)rows_per_tile<D>() * D * 4;
    return ring > rows ? ring : rows;
}

// 16-byte chunk c of K row r sits at chunk c ^ kswz(r): the 16 lanes of a
// fragment read (16 rows, one chunk each) then cover all 64 banks.
template <int D>
__host__ __device__ constexpr int kswz(int r)
{
    return D >= 128 ? (r & 15) : ((r >> 1) & 7);
}

// key-slot chunk q of V^T row d sits at chunk q ^ vswz(d) (64-byte rows):
// free of bank conflicts for the value-operand read (16 rows, four chunks
// each), where (d >> 2) & 3 costs four extra cycles per read (measured with
// the LDS bank-conflict counter)
__host__ __device__ constexpr int vswz(int d)
{
    return (d >> 1) & 3;
}

__device__ __forceinline__ float dq(int mode, int bits, uint32_t c, float s, float z)
{
    return mode == KVQ_AFFINE ? (float)c * s + z : ((float)c - (float)(1 << (bits - 1))) * s;
}

// scale or offset i of a raw metadata range (fp32, or fp16 with meta16)
__device__ __forceinline__ float meta(const uint8_t* sec, size_t i, bool m16)
{
    return m16 ? f16_bits_to_f32(((const uint16_t*)sec)[i]) : ((const float*)sec)[i];
}

typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

// Eight codes of piece idx of a block's code range (8-bit: two u32; 4-bit:
// one u32; 2-bit: one u16), as the words holding codes 0..3 and 4..7 (the
// same word unless the codes are 8-bit).
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

// four consecutive scales or offsets from element i (a multiple of 4)
__device__ __forceinline__ void meta4(const uint8_t* sec, int i, bool m16, float* v)
{
    if (m16) {
        const uint2 h = *(const uint2*)(sec + 2 * i);
        v[0] = f16_bits_to_f32((uint16_t)h.x);
        v[1] = f16_bits_to_f32((uint16_t)(h.x >> 16));
        v[2] = f16_bits_to_f32((uint16_t)h.y);
        v[3] = f16_bits_to_f32((uint16_t)(h.y >> 16));
    } else {
        const floatx4 a = *(const floatx4*)(sec + 4 * i);
#pragma unroll
        for (int e = 0; e < 4; ++e)
            v[e] = a[e];
    }
}

__device__ __forceinline__ float half_bits(const uint16_t* row, size_t i)
{
    return f16_bits_to_f32(row[i]);
}

// In-place unnormalized FWHT of rows [rows][D] fp32 in LDS, then * c, by a
// workgroup of NTH threads.
template <int D, int NTH>
__device__ void fwht_rows(float* x, int rows, float c)
{
    for (int h = 1; h < D; h <<= 1) {
        for (int idx = threadIdx.x; idx < rows * (D / 2); idx += NTH) {
            const int row = idx / (D / 2), k = idx % (D / 2);
            const int j = (k / h) * 2 * h + (k % h);
            const float a = x[row * D + j], b = x[row * D + j + h];
            x[row * D + j] = a + b;
            x[row * D + j + h] = a - b;
        }
        __syncthreads();
    }
    for (int idx = threadIdx.x; idx < rows * D; idx += NTH)
        x[idx] *= c;
    __syncthreads();
}

// Whether workspace block v (sink block when sinkblk, else tail block blk)
// is a code block: per-token key groups and every token of the block coded.
// Its image holds the key codes as exact fp16 values in place of k_hat's hi
// half, and the group scales and offsets in place of the lo half.
template <int D>
__device__ __forceinline__ bool code_block(const AttnParams& p, bool sinkblk, int blk)
{
    return p.k_axis == KVQ_PER_TOKEN && !(D >= 256 && p.k_group == 32) && !sinkblk && 32 * blk + 31 < p.nq;
}

// ---------------------------------------------------------------------------
// 1. Block images.  Grid (blocks per unit, units of the group); workspace
// block v of a unit is sink block v for v < pf_nsb, else tail block
// v - pf_nsb.  Tokens past the end (sink rows beyond n_sink, tail tokens
// beyond n) are zeros: the causal mask removes them, and zero values keep
// 0 * v finite.  W8: both code widths are 8 bits.  A rotating format's
// value rows (coded, window and sink rows alike are stored rotated) pass
// through LDS ([32][D] fp32, dynamic) to be rotated back before they are
// rounded to fp16 (ROT).
template <int D, bool W8, bool ROT>
__global__ __launch_bounds__(kDqThreads) void dequant_kernel(AttnParams p)
{
    extern __shared__ __attribute__((aligned(16))) float vrows[];
    const int v = blockIdx.x;
    const int unit = p.pf_u0 + blockIdx.y;
    uint8_t* img = p.pf_ws + ((size_t)blockIdx.y * p.pf_nvb + v) * (size_t)image_bytes<D>();
    const bool sinkblk = v < p.pf_nsb;
    const int blk = v - p.pf_nsb;

    const int kbits = W8 ? 8 : p.k_bits, vbits = W8 ? 8 : p.v_bits;
    const bool kaff = p.k_mode == KVQ_AFFINE, vaff = p.v_mode == KVQ_AFFINE;
    const bool m16 = p.meta16 != 0;
    const int msz = m16 ? 2 : 4;
    // byte lengths of one block's sections: codes, scales, offsets of K and V
    const int len0 = 4 * D * kbits;
    const int kmeta = p.k_axis == KVQ_PER_TOKEN ? (D / p.k_group) * 32 * msz : D * msz;
    const int len3 = 4 * D * vbits, vmeta = (D / p.v_group) * 32 * msz;
    const size_t ibf = (size_t)unit * (p.T >> 5) + (sinkblk ? 0 : blk);
    const uint8_t* rkc = (const uint8_t*)p.kc + ibf * len0;
    const uint8_t* rks = (const uint8_t*)p.ks + ibf * kmeta;
    const uint8_t* rkz = kaff ? (const uint8_t*)p.kz + ibf * kmeta : nullptr;
    const uint8_t* rvc = (const uint8_t*)p.vc + ibf * len3;
    const uint8_t* rvs = (const uint8_t*)p.vs + ibf * vmeta;
    const uint8_t* rvz = vaff ? (const uint8_t*)p.vz + ibf * vmeta : nullptr;
    const size_t sbase = (size_t)unit * p.sink;
    const size_t rbase = (size_t)unit * p.ring;
    // a wholly coded block of per-token keys keeps its key codes exact (the
    // attention kernel applies the group scales to the score tiles)
    const bool ck = code_block<D>(p, sinkblk, blk);

#pragma unroll
    for (int pc = threadIdx.x; pc < 4 * D; pc += kDqThreads) {
        // K piece: token tau = pc / (D / 8), channels 8 P .. 8 P + 7
        {
            const int tau = pc / (D / 8), P = pc % (D / 8);
            float x[8];
            const uint16_t* row = nullptr;  // fp16 source row (sink or window)
            bool coded = false;
            if (sinkblk) {
                const int ts = 32 * v + tau;
                if (ts < p.n_sink)
                    row = p.kq + (sbase + ts) * D;
            } else {
                const int t = 32 * blk + tau;
                if (t < p.nq)
                    coded = true;
                else if (t < p.n)
                    row = p.kr + (rbase + t % p.ring) * D;
            }
            if (coded) {
                const int r = 4 * (tau / 8) + tau % 4, half = (tau / 4) % 2;
                const int idx = (half * 64 + r + 16 * (P % 4)) * (D / 32) + P / 4;
                const Piece w = piece<W8>(rkc, idx, kbits);
                if (ck) {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        x[e] = (float)code_of(w, kbits, e);
                } else if (p.k_axis == KVQ_PER_TOKEN) {
                    const int mi = ((8 * P) / p.k_group) * 32 + tau;
                    const float sc = meta(rks, mi, m16), z = kaff ? meta(rkz, mi, m16) : 0.0f;
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        x[e] = dq(p.k_mode, kbits, code_of(w, kbits, e), sc, z);
                } else {
                    // per-channel keys: the piece's eight channels' scales
                    // (and offsets) are consecutive, two vector loads each
                    float sc[8], zc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
                    meta4(rks, 8 * P, m16, sc);
                    meta4(rks, 8 * P + 4, m16, sc + 4);
                    if (kaff) {
                        meta4(rkz, 8 * P, m16, zc);
                        meta4(rkz, 8 * P + 4, m16, zc + 4);
                    }
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        x[e] = dq(p.k_mode, kbits, code_of(w, kbits, e), sc[e], zc[e]);
                }
            } else if (row) {
                const u32x4 rw = *(const u32x4*)(row + 8 * P);
                const uint32_t w4[4] = {rw.x, rw.y, rw.z, rw.w};
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    x[e] = f16_bits_to_f32((uint16_t)(w4[e >> 1] >> (16 * (e & 1))));
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    x[e] = 0.0f;
            }
            half8 h, l;
            split_half8(x, &h, &l);  // codes are exact: l = 0
            const size_t off = (size_t)tau * 2 * D + 16 * (P ^ kswz<D>(tau));
            *(u32x4*)(img + off) = __builtin_bit_cast(u32x4, h);
            if (!ck)
                *(u32x4*)(img + klo_at<D>() + off) = __builtin_bit_cast(u32x4, l);
        }
        // V piece: channel d, key-slot chunk q (keys 4 q .. 4 q + 3 and
        // 16 + 4 q .. 16 + 4 q + 3); the four chunks of a row go to four
        // neighbouring lanes, so a wave's stores cover 1 KiB contiguously
        {
            const int d = pc >> 2, q = pc & 3;
            float x[8];
#pragma unroll
            for (int half = 0; half < 2; ++half) {
                const int tk0 = 16 * half + 4 * q;  // first key of the half
                if (!sinkblk && 32 * blk + tk0 < p.nq) {
                    // raw octet tk0 / 8 holds keys tk0 .. tk0 + 3 as its codes
                    // 4 (q & 1) .. + 3; their four scales (and offsets) are
                    // consecutive
                    const Piece w = piece<W8>(rvc, (d % 16 + 16 * (tk0 / 8)) * (D / 16) + d / 16, vbits);
                    const int mi = (d / p.v_group) * 32 + tk0;
                    float sc[4], zc[4] = {0.f, 0.f, 0.f, 0.f};
                    meta4(rvs, mi, m16, sc);
                    if (vaff)
                        meta4(rvz, mi, m16, zc);
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int t = 32 * blk + tk0 + e;
                        x[4 * half + e] = t < p.nq ? dq(p.v_mode, vbits, code_of(w, vbits, 4 * (q & 1) + e), sc[e], zc[e])
                                        : t < p.n  ? half_bits(p.vr, (rbase + t % p.ring) * D + d)
                                                   : 0.0f;
                    }
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int tk = tk0 + e;
                        float val = 0.0f;
                        if (sinkblk) {
                            const int ts = 32 * v + tk;
                            if (ts < p.n_sink)
                                val = half_bits(p.vq, (sbase + ts) * D + d);
                        } else {
                            const int t = 32 * blk + tk;
                            if (t < p.n)
                                val = half_bits(p.vr, (rbase + t % p.ring) * D + d);
                        }
                        x[4 * half + e] = val;
                    }
                }
            }
            if (ROT) {
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    vrows[(16 * (e >> 2) + 4 * q + (e & 3)) * D + d] = x[e];
            } else {
                *(u32x4*)(img + vt_at<D>() + 64 * d + 16 * (q ^ vswz(d))) = __builtin_bit_cast(u32x4, pack_half8(x));
            }
        }
    }
    if (ROT) {
        __syncthreads();
        fwht_rows<D, kDqThreads>(vrows, 32, p.rot_c);
#pragma unroll
        for (int pc = threadIdx.x; pc < 4 * D; pc += kDqThreads) {
            const int d = pc >> 2, q = pc & 3;
            float x[8];
#pragma unroll
            for (int e = 0; e < 8; ++e)
                x[e] = vrows[(16 * (e >> 2) + 4 * q + (e & 3)) * D + d];
            *(u32x4*)(img + vt_at<D>() + 64 * d + 16 * (q ^ vswz(d))) = __builtin_bit_cast(u32x4, pack_half8(x));
        }
    }
    // a code block's key scales s[g][t] and offsets z'[g][t] (fp32, in place
    // of the lo half), with k_hat = c s + z': z' = z for affine codes,
    // -2^(bits-1) s for symmetric ones
    if (ck) {
        const int ng = D / p.k_group;
        float* ms = (float*)(img + klo_at<D>());
        for (int i = threadIdx.x; i < 32 * ng; i += kDqThreads) {
            const float sc = meta(rks, i, m16);
            ms[i] = sc;
            ms[32 * ng + i] = kaff ? meta(rkz, i, m16) : -(float)(1 << (kbits - 1)) * sc;
        }
    }
}

// ---------------------------------------------------------------------------
// 2. Attention over the block images.

// 16 bytes per lane from global memory to LDS address lds_addr + 16 lane
// (lds_addr wave-uniform, held in M0 while the copy issues).  Inline
// assembly, so that the compiler does not make LDS reads wait for every
// outstanding copy; the kernel's own vmcnt waits order them.
__device__ __forceinline__ void copy16(uint64_t base, uint32_t voff, uint32_t lds_addr)
{
    const uint32_t m0v = __builtin_amdgcn_readfirstlane(lds_addr);
    // (the builtin returns int: widen both halves as unsigned, or a low
    // word with bit 31 set would be sign-extended into the high word)
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)base);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(base >> 32));
    const uint64_t sb = ((uint64_t)hi << 32) | (uint64_t)lo;
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2" : : "s"(m0v), "v"(voff), "s"(sb) : "memory");
}

// s_waitcnt vmcnt(n) for a wave-uniform n (expcnt and lgkmcnt not waited)
__device__ __forceinline__ void wait_vm(int n)
{
    switch (n) {
#define KVQ_WAIT_VM(k)                              \
    case k:                                         \
        __builtin_amdgcn_s_waitcnt(0x0F70 | (k)); \
        break;
        KVQ_WAIT_VM(1)
        KVQ_WAIT_VM(2)
        KVQ_WAIT_VM(3)
        KVQ_WAIT_VM(4)
        KVQ_WAIT_VM(5)
        KVQ_WAIT_VM(6)
        KVQ_WAIT_VM(7)
        KVQ_WAIT_VM(8)
        KVQ_WAIT_VM(9)
        KVQ_WAIT_VM(10)
        KVQ_WAIT_VM(11)
        KVQ_WAIT_VM(12)
#undef KVQ_WAIT_VM
    default:
        __builtin_amdgcn_s_waitcnt(0x0F70);
    }
}

// The copies of this wave that precede the newest `after` of its issued
// copies have landed, then every wave is past the same point.
__device__ __forceinline__ void ring_sync(int after)
{
    wait_vm(after);
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
}

// KG: 32-channel score steps per key group when the format's keys have
// per-token groups (code blocks then take exact code operands), 0 otherwise.
// ROT: a rotating format, whose queries (rotated in fp32) carry fp16 lo
// halves; its values come rotated back in the images, so the outputs need
// no inverse rotation.  A bf16 query of a non-rotating format is exact in
// fp16 once scaled by a power of two, so its score steps take one MFMA per
// key tile (code blocks) or two (hi and lo keys).
template <int D, int KG, bool ROT>
__global__ __launch_bounds__(threads<D>(), 2) void attn_kernel(AttnParams p)
{
    constexpr int NW = waves<D>(), kThreads = threads<D>();
    constexpr int QN = qn<D>(), RT = rows_per_tile<D>(), NKS = D / 32, NCT = D / 16;
    constexpr int BI = image_bytes<D>(), NST = stages<D>();
    constexpr int WI = BI / 1024;  // 1 KiB wave copies per image
    extern __shared__ __attribute__((aligned(16))) uint8_t plds[];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int col = lane & 15, qg = lane >> 4;
    // Tiles of one unit run on one XCD (workgroup w goes to XCD w mod 8), so
    // that the unit's block images are read from that XCD's L2 by all of
    // its tiles; the longest (newest) tiles start first.
    const int NT = p.pf_tiles, W = gridDim.x;
    const int L = (W & 7) == 0 ? (blockIdx.x & 7) * (W >> 3) + (blockIdx.x >> 3) : blockIdx.x;
    const int uloc = L / NT, tile = NT - 1 - L % NT;
    const int unit = p.pf_u0 + uloc, b = unit / p.H, h = unit % p.H;
    const int G = p.G, C = p.C;
    const int rows = C * G;
    const int r0 = tile * RT;
    // Positions are tail indices (token minus sink); sink tokens sit at
    // -sink .. -1, so a chunk that starts in the sink has negative positions.
    const int first_pos = p.n - C;  // position of chunk token 0

    // ---- queries: lane's columns are rows r0 + 16 (QN wave + c) + col;
    // for code blocks also the sums of each query over each key group.
    // Rotated queries are scaled by sm_scale log2(e) and split into fp16 hi
    // + lo; others are scaled by qscale, sm_scale log2(e) rounded down to a
    // power of two (exact in fp16 below 65504), and the scores take the
    // rest, sscale.
    constexpr int NG = KG > 0 ? NKS / KG : 1;
    // Offset terms of code blocks as one fp32 MFMA per key tile (ZM) where
    // that measured faster than their FMAs: one 16-row query set per wave,
    // four key groups, no rotation (the rotated path's MFMA pipe is busier)
    constexpr bool ZM = !ROT && QN == 1 && NG == 4;
    half8 qh[QN][NKS], ql[QN][NKS];
    float qsum[QN][NG], qsb[QN];
    const float qscale = ROT ? p.sm_log2 : __uint_as_float(__float_as_uint(p.sm_log2) & 0xFF800000u);
    // (qscale keeps the sign of the scale, so sscale > 0; a zero or
    // subnormal scale gives zero queries, zero scores and sscale 1)
    const float sscale = ROT || qscale == 0.0f ? 1.0f : p.sm_log2 / qscale;
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
        if (ROT)
            fwht_rows<D, kThreads>(xq, RT, p.rot_c);
#pragma unroll
        for (int c = 0; c < QN; ++c) {
            const int rr = 16 * (QN * wave + c) + col;
#pragma unroll
            for (int g = 0; g < NG; ++g)
                qsum[c][g] = 0.0f;
#pragma unroll
            for (int ks = 0; ks < NKS; ++ks) {
                float v[8];
                float part = 0.0f;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    v[e] = xq[rr * D + 32 * ks + 8 * qg + e] * qscale;
                    part += v[e];
                }
                if (ROT)
                    split_half8(v, &qh[c][ks], &ql[c][ks]);
                else
                    qh[c][ks] = pack_half8(v);
                if (KG > 0)
                    qsum[c][ks / (KG > 0 ? KG : 1)] += part;
            }
            // the column's four lanes hold a quarter of every group each
#pragma unroll
            for (int g = 0; g < NG; ++g)
                qsum[c][g] = KG > 0 ? xor_sum16_32(qsum[c][g]) : 0.0f;
            // B operand of the offset product: lane (col, qg) holds the
            // column's sum over group qg (zero beyond NG)
            qsb[c] = 0.0f;
#pragma unroll
            for (int g = 0; g < NG; ++g)
                qsb[c] = ZM && qg == g ? qsum[c][g] : qsb[c];
        }
        __syncthreads();  // the ring overwrites the query rows
    }

    // position of each of this lane's query columns (kNoRow: no such row,
    // every key masked)
    constexpr int kNoRow = -(1 << 30);
    int qpos[QN];
#pragma unroll
    for (int c = 0; c < QN; ++c) {
        const int R = r0 + 16 * (QN * wave + c) + col;
        qpos[c] = R < rows ? first_pos + R / G : kNoRow;
    }
    const int newest = first_pos + (min(r0 + RT, rows) - 1) / G;
    // position of the wave's oldest query when every row of the wave exists
    // (rows are token-major): blocks wholly before it need no causal mask
    const int wrow0 = r0 + 16 * QN * wave;
    const int wave_first = wrow0 + 16 * QN <= rows ? first_pos + wrow0 / G : kNoRow;

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

    const int nkb = newest >= 0 ? newest / 32 + 1 : 0;  // coded-tail blocks
    // sink blocks holding a token no later than the newest query
    const int nsb = min((p.n_sink + 31) >> 5, (newest + p.sink) / 32 + 1);
    const int sb0 = p.sink >> 5;  // sink block j is tail block j - sb0
    const int nvis = nsb + nkb;

    // This wave's copies of an image: wave copies wave, wave + NW, ... < WI
    // (the same count for every wave when WI is a multiple of NW).
    const int cw = WI % NW == 0 ? WI / NW : (WI - wave + NW - 1) / NW;
    const uint32_t lbase = (uint32_t)(uintptr_t)plds;
    const uint8_t* ws_unit = p.pf_ws + (size_t)uloc * p.pf_nvb * BI;
    auto issue = [&](int it) {
        const int vs = it < nsb ? it : p.pf_nsb + (it - nsb);  // workspace block
        const uint64_t base = (uint64_t)(ws_unit + (size_t)vs * BI);
        const uint32_t at = lbase + (uint32_t)((it % NST) * BI);
#pragma unroll
        for (int i = 0; i < (WI + NW - 1) / NW; ++i) {
            const int k = wave + NW * i;
            if (WI % NW == 0 || k < WI)
                copy16(base, (uint32_t)(1024 * k + 16 * lane), at + 1024 * k);
        }
    };

    uint32_t m0_saved;
    asm volatile("s_mov_b32 %0, m0" : "=s"(m0_saved));
    // prologue: images 0 .. NST - 2 in flight, image 0 landed
    for (int it = 0; it < NST - 1 && it < nvis; ++it)
        issue(it);
    ring_sync(NST - 1 <= nvis ? cw * (NST - 2) : 0);

    int stg = 0;  // stage of image it (it mod NST)
    for (int it = 0; it < nvis; ++it) {
        const int blk = it < nsb ? it - sb0 : it - nsb;
        const uint8_t* kh = plds + stg * BI;
        const uint8_t* kl = kh + klo_at<D>();
        const bool codeb = KG > 0 && code_block<D>(p, it < nsb, blk);
        const uint8_t* vt = kh + vt_at<D>();
        // copies of image it + NST - 1 (into the stage image it - 1 used),
        // one per score step so that the wave never waits on a burst of them
        const bool more = it + NST - 1 < nvis;
        const int pstg = stg == 0 ? NST - 1 : stg - 1;
        uint64_t cbase = 0;
        uint32_t cat = 0;
        if (more) {
            const int nvs = it + NST - 1;
            const int vs = nvs < nsb ? nvs : p.pf_nsb + (nvs - nsb);
            cbase = (uint64_t)(ws_unit + (size_t)vs * BI);
            cat = lbase + (uint32_t)(pstg * BI);
        }
        stg = stg + 1 == NST ? 0 : stg + 1;

        // ---- scores S^T (keys x query rows), two 16-key tiles; the next
        // step's K fragments are read while this step's MFMAs run
        floatx4 s[QN][2];
#pragma unroll
        for (int c = 0; c < QN; ++c)
            s[c][0] = s[c][1] = floatx4{0.f, 0.f, 0.f, 0.f};
        auto copy_step = [&](int ks) {
            if (ks < (WI + NW - 1) / NW && more && (WI % NW == 0 || wave + NW * ks < WI))
                copy16(cbase, (uint32_t)(1024 * (wave + NW * ks) + 16 * lane), cat + 1024 * (wave + NW * ks));
        };
        if (codeb) {
            // exact codes c: S = sum_g s_g (c_g . q_g) + z'_g (sum q_g), the
            // products c q over a group in one MFMA per step and key tile
            // (two, q hi and lo, when rotating), then one scaling per group;
            // with ZM the offset terms are one fp32 product [16 keys x 4
            // groups] x [4 groups x 16 queries] per key tile (A: lane (col,
            // qg) holds z'[qg][key col])
            const float* ms = (const float*)kl;
            const float* mz = ms + 32 * NG;
            if (ZM) {
#pragma unroll
                for (int kt = 0; kt < 2; ++kt) {
                    const float za = mz[32 * qg + 16 * kt + col];
#pragma unroll
                    for (int c = 0; c < QN; ++c)
                        s[c][kt] = __builtin_amdgcn_mfma_f32_16x16x4f32(za, qsb[c], s[c][kt], 0, 0, 0);
                }
            }
            half8 fc[2][2];  // [buffer][kt]
            auto cread = [&](int ks, half8 (&f)[2]) {
#pragma unroll
                for (int kt = 0; kt < 2; ++kt) {
                    const int row = 16 * kt + col;
                    f[kt] = __builtin_bit_cast(half8, *(const u32x4*)(kh + row * 2 * D + 16 * ((4 * ks + qg) ^ kswz<D>(row))));
                }
            };
            cread(0, fc[0]);
#pragma unroll
            for (int g = 0; g < NG; ++g) {
                floatx4 sg[QN][2];
#pragma unroll
                for (int c = 0; c < QN; ++c)
                    sg[c][0] = sg[c][1] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int j = 0; j < (KG > 0 ? KG : 1); ++j) {
                    const int ks = g * (KG > 0 ? KG : 1) + j;
                    if (ks + 1 < NKS)
                        cread(ks + 1, fc[(ks + 1) & 1]);
                    copy_step(ks);
#pragma unroll
                    for (int kt = 0; kt < 2; ++kt) {
                        const half8 a = fc[ks & 1][kt];
#pragma unroll
                        for (int c = 0; c < QN; ++c) {
                            sg[c][kt] = mfma16(a, qh[c][ks], sg[c][kt]);
                            if (ROT)
                                sg[c][kt] = mfma16(a, ql[c][ks], sg[c][kt]);
                        }
                    }
                }
                const floatx4 s0 = *(const floatx4*)(ms + 32 * g + 4 * qg);
                const floatx4 s1 = *(const floatx4*)(ms + 32 * g + 16 + 4 * qg);
                floatx4 z0 = {0.f, 0.f, 0.f, 0.f}, z1 = z0;
                if (!ZM) {
                    z0 = *(const floatx4*)(mz + 32 * g + 4 * qg);
                    z1 = *(const floatx4*)(mz + 32 * g + 16 + 4 * qg);
                }
#pragma unroll
                for (int c = 0; c < QN; ++c)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const float o0 = ZM ? s[c][0][i] : fmaf(z0[i], qsum[c][g], s[c][0][i]);
                        const float o1 = ZM ? s[c][1][i] : fmaf(z1[i], qsum[c][g], s[c][1][i]);
                        s[c][0][i] = fmaf(s0[i], sg[c][0][i], o0);
                        s[c][1][i] = fmaf(s1[i], sg[c][1][i], o1);
                    }
            }
        } else {
            half8 fa[2][2][2];  // [buffer][kt][hi, lo]
            auto kread = [&](int ks, half8 (&f)[2][2]) {
#pragma unroll
                for (int kt = 0; kt < 2; ++kt) {
                    const int row = 16 * kt + col;
                    const int off = row * 2 * D + 16 * ((4 * ks + qg) ^ kswz<D>(row));
                    f[kt][0] = __builtin_bit_cast(half8, *(const u32x4*)(kh + off));
                    f[kt][1] = __builtin_bit_cast(half8, *(const u32x4*)(kl + off));
                }
            };
            kread(0, fa[0]);
#pragma unroll
            for (int ks = 0; ks < NKS; ++ks) {
                if (ks + 1 < NKS)
                    kread(ks + 1, fa[(ks + 1) & 1]);
                copy_step(ks);
#pragma unroll
                for (int kt = 0; kt < 2; ++kt) {
                    const half8 ah = fa[ks & 1][kt][0], al = fa[ks & 1][kt][1];
#pragma unroll
                    for (int c = 0; c < QN; ++c) {
                        s[c][kt] = mfma16(ah, qh[c][ks], s[c][kt]);
                        if (ROT)
                            s[c][kt] = mfma16(ah, ql[c][ks], s[c][kt]);
                        s[c][kt] = mfma16(al, qh[c][ks], s[c][kt]);
                    }
                }
            }
        }
        // copies left over when an image needs more than NKS per wave
#pragma unroll
        for (int i = NKS; i < (WI + NW - 1) / NW; ++i)
            if (more && (WI % NW == 0 || wave + NW * i < WI))
                copy16(cbase, (uint32_t)(1024 * (wave + NW * i) + 16 * lane), cat + 1024 * (wave + NW * i));

        // the first value fragments, read while the softmax runs
        constexpr int NVP = D == 256 ? 1 : 2;  // value fragments read ahead
        half8 vf[NVP];
#pragma unroll
        for (int t = 0; t < NVP; ++t) {
            const int d = 16 * t + col;
            vf[t] = __builtin_bit_cast(half8, *(const u32x4*)(vt + 64 * d + 16 * (qg ^ vswz(d))));
        }

        // ---- online softmax per query column; P^T operands
        // The running maximum of a column is raised only when the block's
        // maximum exceeds it by more than 8 (log2 units): probabilities stay
        // below 2^8, and the accumulators are rescaled a few times per row,
        // not per block.  The column maximum needs the column's four lanes;
        // it is gathered only when some lane of the wave holds a score
        // beyond its running maximum + 8 (otherwise no column is raised).
        const bool nomask = 32 * blk + 31 <= wave_first;  // wave-uniform
        // scores x are in the units of the MFMA sums; x sscale is the
        // exponent (sscale > 0), and m is kept in exponent units
        float x[QN][8], lm[QN];
        bool up = false;
#pragma unroll
        for (int c = 0; c < QN; ++c) {
            lm[c] = -INFINITY;
            if (nomask) {
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    x[c][e] = s[c][e >> 2][e & 3];
                    lm[c] = fmaxf(lm[c], x[c][e]);
                }
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int key = 32 * blk + (e < 4 ? 4 * qg + e : 16 + 4 * qg + e - 4);
                    x[c][e] = key <= qpos[c] ? s[c][e >> 2][e & 3] : -INFINITY;
                    lm[c] = fmaxf(lm[c], x[c][e]);
                }
            }
            lm[c] *= sscale;
            up = up || lm[c] > m[c] + 8.0f;
        }
        if (__any(up)) {
#pragma unroll
            for (int c = 0; c < QN; ++c) {
                const float bm = xor_max16_32(lm[c]);
                if (bm > m[c] + 8.0f) {
                    const float alpha = m[c] == -INFINITY ? 0.0f : fast_exp2(m[c] - bm);
                    m[c] = bm;
                    lsum[c] *= alpha;
#pragma unroll
                    for (int t = 0; t < NCT; ++t)
                        acc[c][t] *= alpha;
                }
            }
        }
        half8 ph[QN];
#pragma unroll
        for (int c = 0; c < QN; ++c) {
            // m is finite once a column has seen a key (every existing query
            // row sees a key of the first block); a column that has not
            // takes 0, so that its masked -inf scores give 0, not NaN
            const float mn = m[c] == -INFINITY ? 0.0f : m[c];
            float pv[8];
            float ps = 0.0f;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                pv[e] = fast_exp2(fmaf(x[c][e], sscale, -mn));
                ps += pv[e];
            }
            lsum[c] += ps;
            ph[c] = pack_half8(pv);
        }

        // ---- O^T += V^T P^T, 16 channels per tile, keys in the slot order
        // above; fragment t + NVP is read while tile t's MFMAs run
#pragma unroll
        for (int t = 0; t < NCT; ++t) {
            const half8 av = vf[t % NVP];
            if (t + NVP < NCT) {
                const int d = 16 * (t + NVP) + col;
                vf[t % NVP] = __builtin_bit_cast(half8, *(const u32x4*)(vt + 64 * d + 16 * (qg ^ vswz(d))));
            }
#pragma unroll
            for (int c = 0; c < QN; ++c)
                acc[c][t] = mfma16(av, ph[c], acc[c][t]);
        }
        // image it + 1 has landed (all of this wave's copies but those of
        // the images after it), and no wave reads stage it any more
        ring_sync(it + NST - 1 < nvis ? cw * (NST - 2) : 0);
    }
    asm volatile("s_mov_b32 m0, %0" ::"s"(m0_saved));

    // ---- normalize and write: lane holds O[row][16 t + 4 qg + i]
    float inv[QN];
#pragma unroll
    for (int c = 0; c < QN; ++c) {
        const float l = xor_sum16_32(lsum[c]);
        inv[c] = l > 0.0f ? 1.0f / l : 0.0f;
    }
    // (values were rotated back in the images: outputs are in the original
    // basis for every format)
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
}

template <int D, bool ROT>
void (*pick(int kg))(AttnParams)
{
    return kg == 1   ? attn_kernel<D, (D >= 256 ? 0 : 1), ROT>
           : kg == 2 ? attn_kernel<D, 2, ROT>
           : kg == 4 ? attn_kernel<D, (D >= 128 ? 4 : 1), ROT>
           : kg == 8 ? attn_kernel<D, (D >= 256 ? 8 : 1), ROT>
                     : attn_kernel<D, 0, ROT>;
}

template <int D>
hipError_t launch(const AttnParams& p0, size_t ws_bytes, hipStream_t stream)
{
    constexpr int RT = rows_per_tile<D>();
    const int units = p0.B * p0.H;
    const bool rot = p0.rotate != 0;
    const size_t per_unit = (size_t)p0.pf_nvb * image_bytes<D>();
    const int group = (int)(ws_bytes / per_unit < (size_t)units ? ws_bytes / per_unit : (size_t)units);
    if (group < 1)
        return hipErrorInvalidValue;
    const int tiles = (p0.C * p0.G + RT - 1) / RT;
    const bool w8 = p0.k_bits == 8;  // 8-bit codes come as K and V both 8-bit
    void (*deq)(AttnParams) = w8 ? (rot ? dequant_kernel<D, true, true> : dequant_kernel<D, true, false>)
                                 : (rot ? dequant_kernel<D, false, true> : dequant_kernel<D, false, false>);
    // per-token key groups of 32 KG channels (a power of two from 32 to D);
    // groups of 32 at D = 256 keep the hi + lo path (the code path's eight
    // group sums per query would spill)
    const int kg = p0.k_axis == KVQ_PER_TOKEN ? p0.k_group / 32 : 0;
    void (*att)(AttnParams) = rot ? pick<D, true>(kg) : pick<D, false>(kg);
    if (kg != 0 && kg != 1 && kg != 2 && !(kg == 4 && D >= 128) && !(kg == 8 && D >= 256))
        return hipErrorInvalidValue;
    for (int u0 = 0; u0 < units; u0 += group) {
        AttnParams p = p0;
        p.pf_u0 = u0;
        p.pf_tiles = tiles;
        const int nu = units - u0 < group ? units - u0 : group;
        launch_kernel(deq, dim3(p.pf_nvb, nu), dim3(kDqThreads), rot ? (size_t)32 * D * 4 : 0, stream, p);
        launch_kernel(att, dim3(tiles * nu), dim3(threads<D>()), attn_lds_bytes<D>(), stream, p);
    }
    return hipGetLastError();
}

}  // namespace pre

size_t prefill_image_bytes(int D)
{
    return (size_t)192 * D;
}

hipError_t launch_prefill(const AttnParams& p, int D, size_t ws_bytes, hipStream_t stream)
{
    switch (D) {
    case 64:
        return pre::launch<64>(p, ws_bytes, stream);
    case 128:
        return pre::launch<128>(p, ws_bytes, stream);
    case 256:
        return pre::launch<256>(p, ws_bytes, stream);
    default:
        return hipErrorInvalidValue;
    }
}

}  // namespace kvq
