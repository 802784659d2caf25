// Small kernels around the selective FFN: original id -> slot remap, device-side validation
// of a CSR active-set list, and the residual + RMSNorm step of an FFN stack.
#include "common.h"
#include "launch.h"

namespace si {

namespace {

constexpr int kErrInvalid = 1;
constexpr int kErrRange = 2;
constexpr int kErrDuplicate = 3;
constexpr int kErrNotLoaded = 4;

// Only loaded neurons are computed (Selective Computation section): an original id maps to its
// compacted slot, or to -1 when it is out of range or was not loaded.
__global__ void remap_ids(const int32_t* __restrict__ o2s, int64_t N,
                          const int32_t* __restrict__ ids, int64_t n,
                          int32_t* __restrict__ slots, int* err) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const int32_t v = ids[i];
    int32_t s = -1;
    if (v < 0 || v >= N) {
        if (err) set_err(err, kErrRange, (int)i);
    } else {
        s = o2s[v];
        if (s < 0 && err) set_err(err, kErrNotLoaded, (int)i);
    }
    slots[i] = s;
}

// One work-group per token: offsets in range and non-decreasing, slots in [0, L), no slot
// twice (an LDS bitmap of L bits); with `sorted`, each slot above the one before it.
__global__ __launch_bounds__(256) void check_csr(const int32_t* __restrict__ offsets,
                                                 const int32_t* __restrict__ idx, int64_t nnz,
                                                 int64_t L, int sorted, int* err) {
    extern __shared__ uint32_t bits[];
    const int64_t b = blockIdx.x;
    const int64_t lo = offsets[b], hi = offsets[b + 1];
    if (lo < 0 || hi < lo || hi > nnz) {
        if (threadIdx.x == 0) set_err(err, kErrRange, (int)b);
        return;
    }
    const int64_t words = (L + 31) / 32;
    for (int64_t q = threadIdx.x; q < words; q += blockDim.x) bits[q] = 0u;
    __syncthreads();
    for (int64_t r = lo + threadIdx.x; r < hi; r += blockDim.x) {
        const int32_t s = idx[r];
        if (s < 0 || s >= L) {
            set_err(err, kErrRange, (int)r);
            continue;
        }
        const uint32_t bit = 1u << (s & 31);
        const uint32_t old = atomicOr(&bits[s >> 5], bit);
        if (old & bit) set_err(err, kErrDuplicate, (int)r);
        if (sorted && r > lo && idx[r - 1] > s) set_err(err, kErrInvalid, (int)r);
    }
}

// x_out = RMSNorm(x + y), unit gain, float32 math; one work-group per token, fixed-order sums.

template <typename XT>
__device__ __forceinline__ float xval(const XT* p, int64_t i);
template <>
__device__ __forceinline__ float xval<float>(const float* p, int64_t i) { return p[i]; }
template <>
__device__ __forceinline__ float xval<bf16_t>(const bf16_t* p, int64_t i) {
    return bf16_to_f32(p[i]);
}
__device__ __forceinline__ void xstore(float* p, int64_t i, float v) { p[i] = v; }
__device__ __forceinline__ void xstore(bf16_t* p, int64_t i, float v) {
    p[i] = (bf16_t)f32_to_bf16_rne(v);
}

// One work-group of 1024 threads per token. Thread t owns the groups of four elements
// 4 t + 4096 j: the first pass reads them (up to 16384 elements stay in registers, all loads
// issued together), the sum of squares goes through a fixed shuffle tree in each wave and a
// fixed-order sum of the 16 wave totals, and the second pass scales and stores.
constexpr int kRmsThreads = 1024;
constexpr int kRmsChunk = 4 * kRmsThreads;  // elements per chunk
constexpr int kRmsHold = 4;                 // chunks held in registers

template <typename XT>
__global__ __launch_bounds__(kRmsThreads) void residual_rmsnorm(const XT* x,
                                                               const float* __restrict__ y,
                                                               int64_t d, float eps, XT* xo) {
    // x and xo may alias: each element is read and then written by the same thread
    const int64_t b = blockIdx.x;
    const XT* xb = x + b * d;
    const float* yb = y + b * d;
    XT* ob = xo + b * d;
    const int t = threadIdx.x;
    const int64_t nch = (d + kRmsChunk - 1) / kRmsChunk;
    // d is a multiple of 4 (residual_rmsnorm_any takes the others), so a group of four is
    // all in or all out
    auto load_r = [&](int64_t i, float (&r)[4]) {
        if (i < d) {
#pragma unroll
            for (int e = 0; e < 4; ++e) r[e] = xval<XT>(xb, i + e) + yb[i + e];
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) r[e] = 0.0f;
        }
    };
    float r[kRmsHold][4];
    float ss = 0.0f;
    for (int64_t c0 = 0; c0 < nch; c0 += kRmsHold) {
#pragma unroll
        for (int h = 0; h < kRmsHold; ++h) load_r((c0 + h) * kRmsChunk + 4 * t, r[h]);
#pragma unroll
        for (int h = 0; h < kRmsHold; ++h)
#pragma unroll
            for (int e = 0; e < 4; ++e) ss = fmaf(r[h][e], r[h][e], ss);
    }
#pragma unroll
    for (int m = 1; m < kWave; m <<= 1) ss += __shfl_xor(ss, m, kWave);
    __shared__ float red[kRmsThreads / kWave];
    if ((t & (kWave - 1)) == 0) red[t / kWave] = ss;
    __syncthreads();
    float tot = 0.0f;
#pragma unroll
    for (int q = 0; q < kRmsThreads / kWave; ++q) tot += red[q];
    const float scale = 1.0f / sqrtf(tot / (float)d + eps);
    if (nch <= kRmsHold) {
#pragma unroll
        for (int h = 0; h < kRmsHold; ++h) {
            const int64_t i = h * kRmsChunk + 4 * t;
            if (i < d) {
#pragma unroll
                for (int e = 0; e < 4; ++e) xstore(ob, i + e, r[h][e] * scale);
            }
        }
    } else {
        for (int64_t i = 4 * t; i < d; i += kRmsChunk) {
            float q[4];
            load_r(i, q);
#pragma unroll
            for (int e = 0; e < 4; ++e) xstore(ob, i + e, q[e] * scale);
        }
    }
}

// Any d (d not a multiple of 4): 256 threads, strided loops, the same fixed-order reduction
// shape per work-group.
template <typename XT>
__global__ __launch_bounds__(256) void residual_rmsnorm_any(const XT* x,
                                                            const float* __restrict__ y,
                                                            int64_t d, float eps, XT* xo) {
    const int64_t b = blockIdx.x;
    const XT* xb = x + b * d;
    const float* yb = y + b * d;
    XT* ob = xo + b * d;
    float ss = 0.0f;
    for (int64_t i = threadIdx.x; i < d; i += 256) {
        const float r = xval<XT>(xb, i) + yb[i];
        ss = fmaf(r, r, ss);
    }
    __shared__ float red[256];
    red[threadIdx.x] = ss;
    __syncthreads();
    for (int st = 128; st >= 1; st >>= 1) {
        if ((int)threadIdx.x < st) red[threadIdx.x] += red[threadIdx.x + st];
        __syncthreads();
    }
    const float scale = 1.0f / sqrtf(red[0] / (float)d + eps);
    for (int64_t i = threadIdx.x; i < d; i += 256) {
        const float r = xval<XT>(xb, i) + yb[i];
        xstore(ob, i, r * scale);
    }
}

}  // namespace

hipError_t launch_remap(const int32_t* orig_to_slot, int64_t N, const int32_t* ids, int64_t n,
                        int32_t* slots, int* err, hipStream_t s) {
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(remap_ids, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                       orig_to_slot, N, ids, n, slots, err);
    return hipGetLastError();
}

hipError_t launch_check_csr(const int32_t* offsets, const int32_t* idx, int64_t B, int64_t nnz,
                            int64_t L, bool sorted, int* err, hipStream_t s) {
    if (B == 0) return hipSuccess;
    const size_t lds = (size_t)((L + 31) / 32) * 4;
    hipLaunchKernelGGL(check_csr, dim3((unsigned)B), dim3(256), lds, s, offsets, idx, nnz, L,
                       sorted ? 1 : 0, err);
    return hipGetLastError();
}

hipError_t launch_residual_rmsnorm(const void* x, int xdt, const float* y, int64_t B, int64_t d,
                                   float eps, void* x_out, hipStream_t s) {
    if (B == 0) return hipSuccess;
    const bool v4 = d % 4 == 0;
    if (xdt == 1) {
        const bf16_t* xi = static_cast<const bf16_t*>(x);
        bf16_t* xo = static_cast<bf16_t*>(x_out);
        if (v4)
            hipLaunchKernelGGL(residual_rmsnorm<bf16_t>, dim3((unsigned)B), dim3(kRmsThreads), 0,
                               s, xi, y, d, eps, xo);
        else
            hipLaunchKernelGGL(residual_rmsnorm_any<bf16_t>, dim3((unsigned)B), dim3(256), 0, s,
                               xi, y, d, eps, xo);
    } else {
        const float* xi = static_cast<const float*>(x);
        float* xo = static_cast<float*>(x_out);
        if (v4)
            hipLaunchKernelGGL(residual_rmsnorm<float>, dim3((unsigned)B), dim3(kRmsThreads), 0,
                               s, xi, y, d, eps, xo);
        else
            hipLaunchKernelGGL(residual_rmsnorm_any<float>, dim3((unsigned)B), dim3(256), 0, s,
                               xi, y, d, eps, xo);
    }
    return hipGetLastError();
}

}  // namespace si
