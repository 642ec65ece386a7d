// The quantizer shared by the append kernels and the fused projection
// epilogue (Sec. 3.1, Eq. (3) and the symmetric control): group statistics,
// fp16 rounding of metadata, codes and packed pieces.  Codes and metadata
// must equal the CPU reference bit for bit, so every function here takes
// exactly the reference's IEEE binary32 steps with contraction off.
#pragma once

#include <stdint.h>

#include "kvq_device.h"
#include "kvq_internal.h"

namespace kvq {

// A piece holds eight codes of `bits` bits: 16, 32 or 64 bits wide.
__device__ __forceinline__ void store_piece(void* base, size_t i, int bits, uint64_t v)
{
#pragma clang fp contract(off)
    if (bits == 8)
        ((uint64_t*)base)[i] = v;
    else if (bits == 4)
        ((uint32_t*)base)[i] = (uint32_t)v;
    else
        ((uint16_t*)base)[i] = (uint16_t)v;
}

__device__ __forceinline__ uint64_t load_piece(const void* base, size_t i, int bits)
{
#pragma clang fp contract(off)
    if (bits == 8)
        return ((const uint64_t*)base)[i];
    return bits == 4 ? ((const uint32_t*)base)[i] : ((const uint16_t*)base)[i];
}

// Mask of the low `n` codes of a piece (n < 8).
__device__ __forceinline__ uint64_t low_codes(int bits, int n)
{
#pragma clang fp contract(off)
    return (1ull << (bits * n)) - 1ull;
}

// rint(fl(d / s)), the correctly rounded quotient rounded half to even,
// with r the hardware reciprocal of s (within 1 ulp).  d r is within about
// 1.5 2^-23 relative of d / s, so for |d / s| <= 256 (every code here) it
// is within 2^-14 of fl(d / s); rint can differ only if that interval
// contains a half-integer, so the exact division runs only where d r lies
// within 2^-10 of one.
__device__ __forceinline__ float rint_quotient(float d, float s, float r)
{
#pragma clang fp contract(off)
    const float q = d * r;
    float c = __builtin_rintf(q);
    const float f = q - floorf(q);
    if (fabsf(f - 0.5f) < 0x1p-10f)
        c = __builtin_rintf(d / s);
    return c;
}

__device__ __forceinline__ uint32_t code_affine(float x, float mn, float s, float r, float top)
{
#pragma clang fp contract(off)
    float c = rint_quotient(x - mn, s, r);
    c = fminf(fmaxf(c, 0.0f), top);
    return (uint32_t)c;
}

__device__ __forceinline__ uint32_t code_sym(float x, float s, float r, float qmax, float half)
{
#pragma clang fp contract(off)
    float q = rint_quotient(x, s, r);
    q = fminf(fmaxf(q, -qmax), qmax);
    return (uint32_t)(int)(q + half);
}

// Scale (and offset) of one group, Eq. (3) / symmetric control.
__device__ __forceinline__ void group_stats(const float* x, int stride, int g, int mode, int bits,
                                            float* s_out, float* z_out)
{
#pragma clang fp contract(off)
    if (mode == KVQ_AFFINE) {
        float mn = x[0], mx = x[0];
        for (int i = 1; i < g; ++i) {
            float v = x[i * stride];
            mn = fminf(mn, v);
            mx = fmaxf(mx, v);
        }
        const float top = (float)((1 << bits) - 1);
        float s = (mx - mn) / top;
        if (!(s >= 1e-8f))
            s = 1e-8f;
        *s_out = s;
        *z_out = mn + 0.0f;  // canonical +0 for a signed-zero minimum
    } else {
        float ma = 0.0f;
        for (int i = 0; i < g; ++i)
            ma = fmaxf(ma, fabsf(x[i * stride]));
        const float qmax = (float)((1 << (bits - 1)) - 1);
        float s = ma / qmax;
        if (!(s >= 1e-8f))
            s = 1e-8f;
        *s_out = s;
        *z_out = 0.0f;
    }
}

// fp16 metadata: the scale and offset as stored, i.e. rounded to nearest
// fp16 (scale clamped to [2^-24, 65504], offset to +-65504); the codes are
// then computed from these values.
__device__ __forceinline__ void round_meta(int meta16, float* s, float* z)
{
#pragma clang fp contract(off)
    if (!meta16)
        return;
    const float sc = fminf(fmaxf(*s, 0x1p-24f), 65504.0f);
    const float zc = fminf(fmaxf(*z, -65504.0f), 65504.0f);
    *s = f16_bits_to_f32(f32_to_f16_bits(sc));
    *z = f16_bits_to_f32(f32_to_f16_bits(zc)) + 0.0f;
}

// Scale or offset i of a metadata section: fp32, or fp16 (an exact value).
__device__ __forceinline__ void store_meta(float* base, size_t i, float v, int meta16)
{
#pragma clang fp contract(off)
    if (meta16)
        ((uint16_t*)base)[i] = f32_to_f16_bits(v);
    else
        base[i] = v;
}

// Code of x in a group with scale s (r = its hardware reciprocal) and offset z.
__device__ __forceinline__ uint32_t code_one(float x, float s, float r, float z, int mode, int bits)
{
#pragma clang fp contract(off)
    if (mode == KVQ_AFFINE)
        return code_affine(x, z, s, r, (float)((1 << bits) - 1));
    return code_sym(x, s, r, (float)((1 << (bits - 1)) - 1), (float)(1 << (bits - 1)));
}

// Statistics of one per-token group held by `lanes` consecutive lanes,
// eight values each (lanes = group size / 8: a power of two, at most 32, so
// a group never straddles a wave).  min, max and max-magnitude are exact in
// any order, so the shuffle tree gives the serial loop's values.
__device__ __forceinline__ void piece_group_stats(const float* x, int lanes, int mode, int bits, float* s_out,
                                                  float* z_out)
{
#pragma clang fp contract(off)
    if (mode == KVQ_AFFINE) {
        float mn = x[0], mx = x[0];
#pragma unroll
        for (int e = 1; e < 8; ++e) {
            mn = fminf(mn, x[e]);
            mx = fmaxf(mx, x[e]);
        }
        for (int off = 1; off < lanes; off <<= 1) {
            mn = fminf(mn, __shfl_xor(mn, off));
            mx = fmaxf(mx, __shfl_xor(mx, off));
        }
        const float top = (float)((1 << bits) - 1);
        float s = (mx - mn) / top;
        if (!(s >= 1e-8f))
            s = 1e-8f;
        *s_out = s;
        *z_out = mn + 0.0f;  // canonical +0 for a signed-zero minimum
    } else {
        float ma = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e)
            ma = fmaxf(ma, fabsf(x[e]));
        for (int off = 1; off < lanes; off <<= 1)
            ma = fmaxf(ma, __shfl_xor(ma, off));
        const float qmax = (float)((1 << (bits - 1)) - 1);
        float s = ma / qmax;
        if (!(s >= 1e-8f))
            s = 1e-8f;
        *s_out = s;
        *z_out = 0.0f;
    }
}

}  // namespace kvq
