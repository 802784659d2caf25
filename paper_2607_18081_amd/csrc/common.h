// Device helpers shared by the selective-FFN kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace si {

constexpr int kWave = 64;

typedef uint16_t bf16_t;  // bfloat16 bit pattern
typedef _Float16 f16_t;   // IEEE half precision

// Error word layout written by device-side checks (first nonzero code wins).
struct ErrWord {
    int code;
    int detail;
};

__device__ __forceinline__ void set_err(int* err, int code, int detail) {
    // integer compare-and-swap on a status word; never on the decode hot path
    if (atomicCAS(err, 0, code) == 0) err[1] = detail;
}

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
    return __uint_as_float(bits16 << 16);
}

// low / high halves of a 32-bit word holding two bf16 values
__device__ __forceinline__ float bf16lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// float -> bf16 bits, round to nearest even (inputs here are finite)
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}

// half precision <-> float32 (hardware conversion, round to nearest even)
__device__ __forceinline__ float f16_to_f32(uint32_t bits16) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)bits16);
}
__device__ __forceinline__ uint32_t f32_to_f16_rne(float f) {
    return __builtin_bit_cast(uint16_t, (_Float16)f);
}

// 16-byte vector types
struct alignas(16) V16 {
    uint32_t w[4];
};

__device__ __forceinline__ V16 ld16(const void* p) {
    return *reinterpret_cast<const V16*>(p);
}
__device__ __forceinline__ void st16(void* p, const V16& v) {
    *reinterpret_cast<V16*>(p) = v;
}

// Raw buffer loads (gfx9 buffer descriptors). The descriptor's range check returns zeros, and
// reads no memory, for a byte offset outside the buffer: kernels pass kOOB for rows or columns
// that must contribute nothing, so loads need no branches. Offsets are 32-bit, so a buffer
// read this way must be smaller than 2 GiB.
typedef __attribute__((ext_vector_type(4))) int i32x4_t;
constexpr int kOOB = (int)0x80000000;

// 16-byte store with the non-temporal hint: for data written once and read once by the next
// kernel (partial sums), which need not stay in this XCD's L2
__device__ __forceinline__ void st16_nt(void* p, const V16& v) {
    const i32x4_t t = {(int)v.w[0], (int)v.w[1], (int)v.w[2], (int)v.w[3]};
    __builtin_nontemporal_store(t, reinterpret_cast<i32x4_t*>(p));
}
constexpr int kBufWord3 = 0x00020000;  // dword 3 of a raw gfx9 descriptor: 32-bit data format

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, kBufWord3);
}

__device__ __forceinline__ V16 bload16(__amdgpu_buffer_rsrc_t r, int off) {
    const i32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
    V16 o;
    o.w[0] = (uint32_t)v[0];
    o.w[1] = (uint32_t)v[1];
    o.w[2] = (uint32_t)v[2];
    o.w[3] = (uint32_t)v[3];
    return o;
}

// The same load with the non-temporal cache policy: for weight rows that a launch reads once
// (a decode step's active rows). Measured on a 54 MB gather of 24 KB rows: 10.4 us against
// 11.3 us with the default policy.
constexpr int kNonTemporal = 2;  // cache-policy word of a gfx950 buffer access: nt
__device__ __forceinline__ V16 bload16nt(__amdgpu_buffer_rsrc_t r, int off) {
    const i32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kNonTemporal);
    V16 o;
    o.w[0] = (uint32_t)v[0];
    o.w[1] = (uint32_t)v[1];
    o.w[2] = (uint32_t)v[2];
    o.w[3] = (uint32_t)v[3];
    return o;
}

// Buffer load at a per-lane offset plus a wave-uniform (scalar-register) offset. The row base
// of a gather goes in the scalar offset, so addressing a row costs no vector instructions.
__device__ __forceinline__ V16 bload16s(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
    const i32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
    V16 o;
    o.w[0] = (uint32_t)v[0];
    o.w[1] = (uint32_t)v[1];
    o.w[2] = (uint32_t)v[2];
    o.w[3] = (uint32_t)v[3];
    return o;
}

// Unpack a 16-byte vector into V floats (V = 8 for bf16, 4 for f32).
template <typename T>
struct Elem;
template <>
struct Elem<float> {
    static constexpr int V = 4;
    __device__ __forceinline__ static void unpack(const V16& v, float* f) {
#pragma unroll
        for (int e = 0; e < 4; ++e) f[e] = __uint_as_float(v.w[e]);
    }
};
template <>
struct Elem<f16_t> {
    static constexpr int V = 8;
    __device__ __forceinline__ static void unpack(const V16& v, float* f) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            f[2 * e] = f16_to_f32(v.w[e] & 0xffffu);
            f[2 * e + 1] = f16_to_f32(v.w[e] >> 16);
        }
    }
};
template <>
struct Elem<bf16_t> {
    static constexpr int V = 8;
    __device__ __forceinline__ static void unpack(const V16& v, float* f) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            f[2 * e] = bf16lo(v.w[e]);
            f[2 * e + 1] = bf16hi(v.w[e]);
        }
    }
};

// Float32 partial sums of the two-level reductions are stored column-chunked: for token b,
// partial p and column c, element ((b * nch + c / 16) * P + p) * 16 + c % 16, with
// nch = ceil(d / 16). The P partials of 16 columns are then one contiguous block of P * 64
// bytes, which the reducer reads in full 128-byte lines, and a writer's 16 columns are 64
// contiguous bytes.
constexpr int kChunk = 16;
__host__ __device__ __forceinline__ int64_t part_chunks(int64_t d) { return (d + kChunk - 1) / kChunk; }
__host__ __device__ __forceinline__ int64_t part_off(int64_t b, int64_t p, int64_t col, int64_t P,
                                                     int64_t nch) {
    return ((b * nch + col / kChunk) * P + p) * kChunk + col % kChunk;
}

// SiLU(g) = g * sigmoid(g), float32
// Inclusive prefix sum over the 64 lanes of a wave (lane order): DPP row shifts scan each row
// of 16 lanes, then two row broadcasts carry the totals of rows 0 and 0-1 upward.
__device__ __forceinline__ int wave_incl_scan(int v) {
    v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, false);  // row_shr:1
    v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, false);  // row_shr:2
    v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, false);  // row_shr:4
    v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, false);  // row_shr:8
    v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xa, 0xf, false);  // row_bcast:15 -> rows 1, 3
    v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xc, 0xf, false);  // row_bcast:31 -> rows 2, 3
    return v;
}

__device__ __forceinline__ float silu_f32(float g) { return __fdividef(g, 1.0f + __expf(-g)); }

// Sum over the 64 lanes of a wave; every lane receives the total.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
    return v;
}

// Reduce NVAL per-lane values across the wave at once. On return, lane l holds the wave total
// of value index l / (64 / NVAL). NVAL is a power of two, 1 <= NVAL <= 64. Each step pairs the
// lanes that differ in one lane-id bit: the lower lane keeps the lower half of its values, the
// upper lane the upper half, and each adds its partner's copy of the half it keeps. Costs
// NVAL - 1 + log2(64 / NVAL) shuffles instead of 6 * NVAL. All indices are compile-time.
template <int CNT, int MASK>
struct TransposeSum {
    __device__ __forceinline__ static void run(float* v, int lane) {
        constexpr int half = CNT / 2;
        const bool upper = (lane & MASK) != 0;
#pragma unroll
        for (int m = 0; m < half; ++m) {
            const float send = upper ? v[m] : v[m + half];
            const float keep = upper ? v[m + half] : v[m];
            v[m] = keep + __shfl_xor(send, MASK, kWave);
        }
        TransposeSum<half, MASK / 2>::run(v, lane);
    }
};
template <int MASK>
struct TransposeSum<1, MASK> {
    __device__ __forceinline__ static void run(float* v, int lane) {
        v[0] += __shfl_xor(v[0], MASK, kWave);
        TransposeSum<1, MASK / 2>::run(v, lane);
    }
};
template <>
struct TransposeSum<1, 0> {
    __device__ __forceinline__ static void run(float*, int) {}
};

template <int NVAL>
__device__ __forceinline__ float wave_transpose_sum(float (&v)[NVAL], int lane) {
    static_assert((NVAL & (NVAL - 1)) == 0 && NVAL >= 1 && NVAL <= 64, "NVAL");
    TransposeSum<NVAL, 32>::run(v, lane);
    return v[0];
}

}  // namespace si
