// Device-side helpers shared by the libfo kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fo {

typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

template <typename To, typename From>
__device__ __forceinline__ To bit_cast(const From& f) {
    static_assert(sizeof(To) == sizeof(From), "size mismatch");
    To t;
    __builtin_memcpy(&t, &f, sizeof(To));
    return t;
}

// fp32 -> fp16 bits, round to nearest even (v_cvt_f16_f32 in the default
// rounding mode).
__device__ __forceinline__ uint32_t f32_to_f16_bits(float x) {
    return (uint32_t)bit_cast<uint16_t>((_Float16)x);
}

// fp32 -> bf16 bits, round to nearest even; NaN stays a (quiet) NaN. The
// conversion is gfx950's v_cvt_pk_bf16_f32: no per-element branch.
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float x) {
    return (uint32_t)bit_cast<uint16_t>((__bf16)x);
}

__device__ __forceinline__ float f16_bits_to_f32(uint32_t h) {
    return (float)bit_cast<_Float16>((uint16_t)h);
}

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b) {
    return bit_cast<float>(b << 16);
}

template <int DT>
__device__ __forceinline__ float to_f32(uint32_t bits) {
    if constexpr (DT == 0) return f16_bits_to_f32(bits);
    else return bf16_bits_to_f32(bits);
}

template <int DT>
__device__ __forceinline__ uint32_t from_f32(float x) {
    if constexpr (DT == 0) return f32_to_f16_bits(x);
    else return f32_to_bf16_bits(x);
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));

// Two fp32 values rounded (to nearest even) and packed into one 32-bit word
// (low = a): one v_cvt_pk_f16_f32 or v_cvt_pk_bf16_f32.
template <int DT>
__device__ __forceinline__ uint32_t pack2(float a, float b) {
    const f32x2_t v = {a, b};
    if constexpr (DT == 0) return bit_cast<uint32_t>(__builtin_convertvector(v, f16x2_t));
    else return bit_cast<uint32_t>(__builtin_convertvector(v, bf16x2_t));
}

}  // namespace fo
