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

// Position e of a code operand holds code perm4(e) of its piece: dword j of
// the operand carries codes j and j + 4.
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
