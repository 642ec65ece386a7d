// Device helpers for the gfx950 kernels: MFMA fragment types, conversions
// between packed codes and fp16 MFMA operands, and exact rounding helpers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kvq {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// v_mfma_f32_16x16x32_{f16,bf16}: D[16x16] += A[16x32] B[32x16].  Lane l
// supplies A[l % 16][8 (l / 16) + e] and B[8 (l / 16) + e][l % 16] for
// e = 0..7, and receives D[4 (l / 16) + i][l % 16] for i = 0..3.
__device__ __forceinline__ floatx4 mfma16(half8 a, half8 b, floatx4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ floatx4 mfma16_bf16(bf16x8 a, bf16x8 b, floatx4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h)
{
    return __uint_as_float((uint32_t)h << 16);
}

// binary32 -> bfloat16, round to nearest even (finite inputs).
__device__ __forceinline__ uint16_t f32_to_bf16(float f)
{
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

__device__ __forceinline__ uint16_t f32_to_f16_bits(float f)
{
    _Float16 h = (_Float16)f;  // v_cvt_f16_f32: round to nearest even
    return __builtin_bit_cast(uint16_t, h);
}

__device__ __forceinline__ float f16_bits_to_f32(uint16_t h)
{
    return (float)__builtin_bit_cast(_Float16, h);
}

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));

// Eight packed codes -> eight exact fp16 MFMA operand values c - offset, in
// the element order (c0, c4, c1, c5, c2, c6, c3, c7).  For 4-bit codes `w`
// is a whole word; for 2-bit codes the eight codes are the low 16 bits of
// `w`.  0x6400 is binary16 1024.0, whose unit in the last place is 1, so
// OR-ing a code c < 1024 into the mantissa gives exactly 1024 + c; one packed
// fp16 subtract per pair (exact: the result is a small integer) removes
// 1024 + offset.  offset is 0 for affine codes and 2^(bits-1) for symmetric
// codes, whose stored value is q + 2^(bits-1).
template <int BITS>
__device__ __forceinline__ half8 codes_to_half8(uint32_t w, half2_t bias)
{
    uint32_t y;
    uint32_t mask;
    if (BITS == 4) {
        y = w;
        mask = 0x000F000Fu;
    } else {
        y = (w & 0xFFFFu) | ((w & 0xFFFFu) << 8);  // codes 4..7 land at bits 16..23
        mask = 0x00030003u;
    }
    half2_t h0 = __builtin_bit_cast(half2_t, ((y >> (0 * BITS)) & mask) | 0x64006400u) - bias;
    half2_t h1 = __builtin_bit_cast(half2_t, ((y >> (1 * BITS)) & mask) | 0x64006400u) - bias;
    half2_t h2 = __builtin_bit_cast(half2_t, ((y >> (2 * BITS)) & mask) | 0x64006400u) - bias;
    half2_t h3 = __builtin_bit_cast(half2_t, ((y >> (3 * BITS)) & mask) | 0x64006400u) - bias;
    u32x4 v;
    v.x = __builtin_bit_cast(uint32_t, h0);
    v.y = __builtin_bit_cast(uint32_t, h1);
    v.z = __builtin_bit_cast(uint32_t, h2);
    v.w = __builtin_bit_cast(uint32_t, h3);
    return __builtin_bit_cast(half8, v);
}

// Position e of an MFMA operand built by codes_to_half8 holds code PERM4[e].
__device__ constexpr int perm4(int e)
{
    return (e & 1) ? 4 + (e >> 1) : (e >> 1);
}

__device__ __forceinline__ half8 pack_half8(const float* v)
{
    half8 h;
#pragma unroll
    for (int e = 0; e < 8; ++e)
        h[e] = (_Float16)v[e];
    return h;
}

// fp32 -> fp16 hi + lo with hi + lo = v to about 22 significant bits, so an
// MFMA pair over (hi, lo) carries nearly fp32 precision.
__device__ __forceinline__ void split_half8(const float* v, half8* hi, half8* lo)
{
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        _Float16 h = (_Float16)v[e];
        (*hi)[e] = h;
        (*lo)[e] = (_Float16)(v[e] - (float)h);
    }
}

__device__ __forceinline__ float xor_sum16_32(float v)
{
    v += __shfl_xor(v, 16);
    v += __shfl_xor(v, 32);
    return v;
}

__device__ __forceinline__ float xor_max16_32(float v)
{
    v = fmaxf(v, __shfl_xor(v, 16));
    v = fmaxf(v, __shfl_xor(v, 32));
    return v;
}

__device__ __forceinline__ float fast_exp2(float x)
{
    return __builtin_amdgcn_exp2f(x);
}

}  // namespace kvq
