// 16-bit MFMA element types (bf16 and IEEE half) for the union-path GEMMs: one 16x16x32
// v_mfma with float32 accumulation, the 8-element operand vector, and rounding to / widening
// from the 16-bit storage format. Storage is always the raw 16-bit pattern (uint16_t).
#pragma once

#include "common.h"

namespace si {

typedef __attribute__((ext_vector_type(4))) float f32x4_t;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4_t;

template <typename ET>
struct Mfma;

template <>
struct Mfma<bf16_t> {
    typedef __attribute__((ext_vector_type(8))) __bf16 vec8;
    __device__ __forceinline__ static vec8 vec(const V16& v) {
        const u32x4_t t = {v.w[0], v.w[1], v.w[2], v.w[3]};
        return __builtin_bit_cast(vec8, t);
    }
    __device__ __forceinline__ static f32x4_t mma(const vec8& a, const vec8& b, const f32x4_t& c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
    __device__ __forceinline__ static uint32_t rne(float f) { return f32_to_bf16_rne(f); }
    __device__ __forceinline__ static float widen(uint32_t b) { return bf16_to_f32(b); }
};

template <>
struct Mfma<f16_t> {
    typedef __attribute__((ext_vector_type(8))) _Float16 vec8;
    __device__ __forceinline__ static vec8 vec(const V16& v) {
        const u32x4_t t = {v.w[0], v.w[1], v.w[2], v.w[3]};
        return __builtin_bit_cast(vec8, t);
    }
    __device__ __forceinline__ static f32x4_t mma(const vec8& a, const vec8& b, const f32x4_t& c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
    }
    __device__ __forceinline__ static uint32_t rne(float f) { return f32_to_f16_rne(f); }
    __device__ __forceinline__ static float widen(uint32_t b) { return f16_to_f32(b); }
};

}  // namespace si
