// Memory-system references for the per-token path (measurement only, not part of the method).
//
// Both kernels only load and fold the loaded words into one value per lane, which they store,
// so the loads stay live; they do no arithmetic of the FFN.
//
//  - ceiling_stream: a contiguous read of a buffer, 16-byte non-temporal loads, eight in flight
//    per lane, each work-group reading one contiguous part;
//  - ceiling_gather: the per-token path's access pattern without its arithmetic: P work-groups
//    of 512 threads deal a token's k active slots as the gather-GEMV kernel does (work-group p
//    takes rows [floor(k p / P), floor(k (p + 1) / P))), and for each batch of up to 16 rows
//    issue every gate and up row load, then every down row load, 16 bytes per lane per row,
//    non-temporal; a batch issues loads for the rows it has only. Its time is the floor of
//    that kernel's on the same rows.
#include <hip/hip_ext.h>

#include "common.h"
#include "launch.h"

namespace si {

namespace {

constexpr int kCeilThreads = 512;
constexpr int kCeilRows = 16;

__global__ __launch_bounds__(kCeilThreads) void ceiling_stream(const void* __restrict__ buf,
                                                               int64_t bytes,
                                                               uint32_t* __restrict__ sink) {
    const __amdgpu_buffer_rsrc_t r = make_rsrc(buf, bytes);
    constexpr int64_t kStep = (int64_t)kCeilThreads * 16;
    const int64_t per = (bytes + gridDim.x - 1) / gridDim.x;
    const int64_t lo = (int64_t)blockIdx.x * per;
    const int64_t hi = lo + per < bytes ? lo + per : bytes;
    uint32_t acc = 0;
    int64_t o = lo + threadIdx.x * 16;
    for (; o + 7 * kStep < hi; o += 8 * kStep) {
        V16 v[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) v[q] = bload16nt(r, (int)(o + q * kStep));
#pragma unroll
        for (int q = 0; q < 8; ++q) acc ^= v[q].w[0] + v[q].w[1] + v[q].w[2] + v[q].w[3];
    }
    for (; o < hi; o += kStep) {  // the buffer's own bounds check zeroes a partial last group
        const V16 v = bload16nt(r, (int)o);
        acc ^= v.w[0] + v.w[1] + v.w[2] + v.w[3];
    }
    sink[(int64_t)blockIdx.x * kCeilThreads + threadIdx.x] = acc;
}

// One batch of N rows (N a compile-time constant, as in the gather-GEMV kernel): every gate and
// up load of the N rows, then every down load, then the fold. Only the N rows issue loads, so
// a work-group whose share ends inside a batch spends no load issue slots on rows it does not
// have.
template <int N>
__device__ __forceinline__ void gather_batch(__amdgpu_buffer_rsrc_t rg, __amdgpu_buffer_rsrc_t rd,
                                             const int32_t (&sl)[kCeilRows], int64_t L,
                                             int64_t row_bytes, uint32_t& acc) {
    for (int64_t c = (int64_t)threadIdx.x * 16; c < row_bytes + 15; c += kCeilThreads * 16) {
        const int col = c < row_bytes ? (int)c : kOOB;
        V16 g[N], u[N], dn[N];
#pragma unroll
        for (int q = 0; q < N; ++q) {
            const bool ok = sl[q] >= 0 && sl[q] < L && col != kOOB;
            const int og = ok ? (int)(sl[q] * 2 * row_bytes) + col : kOOB;
            g[q] = bload16nt(rg, og);
            u[q] = bload16nt(rg, ok ? og + (int)row_bytes : kOOB);
        }
#pragma unroll
        for (int q = 0; q < N; ++q) {
            const bool ok = sl[q] >= 0 && sl[q] < L && col != kOOB;
            dn[q] = bload16nt(rd, ok ? (int)(sl[q] * row_bytes) + col : kOOB);
        }
#pragma unroll
        for (int q = 0; q < N; ++q)
#pragma unroll
            for (int e = 0; e < 4; ++e) acc ^= g[q].w[e] + 3u * u[q].w[e] + 7u * dn[q].w[e];
    }
}

// gather_batch<n> for a run-time n in [N, kCeilRows], through a chain of uniform compares
template <int N>
__device__ __forceinline__ void gather_rows(int n, __amdgpu_buffer_rsrc_t rg,
                                            __amdgpu_buffer_rsrc_t rd,
                                            const int32_t (&sl)[kCeilRows], int64_t L,
                                            int64_t row_bytes, uint32_t& acc) {
    if constexpr (N <= kCeilRows) {
        if (n == N)
            gather_batch<N>(rg, rd, sl, L, row_bytes, acc);
        else
            gather_rows<N + 1>(n, rg, rd, sl, L, row_bytes, acc);
    }
}

__global__ __launch_bounds__(kCeilThreads) void ceiling_gather(
    const void* __restrict__ gate_up_c, const void* __restrict__ down_c, int64_t L,
    int64_t row_bytes, const int32_t* __restrict__ idx, int64_t k,
    uint32_t* __restrict__ sink) {
    const int p = blockIdx.x;
    const int P = gridDim.x;
    const __amdgpu_buffer_rsrc_t rg = make_rsrc(gate_up_c, L * 2 * row_bytes);
    const __amdgpu_buffer_rsrc_t rd = make_rsrc(down_c, L * row_bytes);
    const int64_t r0 = (int64_t)((uint32_t)k * (uint32_t)p / (uint32_t)P);
    const int64_t r1 = (int64_t)((uint32_t)k * (uint32_t)(p + 1) / (uint32_t)P);
    uint32_t acc = 0;
    for (int64_t rb = r0; rb < r1; rb += kCeilRows) {
        const int n = (int)(r1 - rb < kCeilRows ? r1 - rb : kCeilRows);
        int32_t sl[kCeilRows];
#pragma unroll
        for (int q = 0; q < kCeilRows; ++q) sl[q] = q < n ? idx[rb + q] : -1;
        gather_rows<1>(n, rg, rd, sl, L, row_bytes, acc);
    }
    sink[(int64_t)p * kCeilThreads + threadIdx.x] = acc;
}

}  // namespace

hipError_t launch_ceiling_stream(const void* buf, int64_t bytes, int blocks, uint32_t* sink,
                                 hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
    hipExtLaunchKernelGGL(ceiling_stream, dim3((unsigned)blocks), dim3(kCeilThreads), 0, s, ev0,
                          ev1, 0, buf, bytes, sink);
    return hipGetLastError();
}

hipError_t launch_ceiling_gather(const void* gate_up_c, const void* down_c, int64_t L,
                                 int64_t row_bytes, const int32_t* idx, int64_t k, int P,
                                 uint32_t* sink, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
    hipExtLaunchKernelGGL(ceiling_gather, dim3((unsigned)P), dim3(kCeilThreads), 0, s, ev0, ev1,
                          0, gate_up_c, down_c, L, row_bytes, idx, k, sink);
    return hipGetLastError();
}

}  // namespace si
