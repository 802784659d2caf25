// Selective loading (Selective Loading section): keep only the loaded neurons' slices of
// gate_proj, up_proj and down_proj, laid out neuron-major.
//
// Maps: counts of each id are taken in orig_to_slot (integer atomics, load-time only); one
// work-group then scans the N counts in id order, so slot s is the s-th smallest loaded id,
// and flags duplicates. Gathers: gate/up rows are copied with 16-byte moves into
// gate_up_c [L][2][d]; the down_proj columns are gathered through a 64x64 LDS tile so that
// both the column reads (ascending ids within a row of W_down) and the row writes of
// down_c [L][d] stay contiguous.
#include "common.h"
#include "launch.h"

namespace si {

namespace {

constexpr int kErrRange = 2;
constexpr int kErrDuplicate = 3;

__global__ void fill_i32(int32_t* __restrict__ p, int64_t n, int32_t v) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = v;
}

__global__ void count_ids(const int32_t* __restrict__ loaded, int64_t L, int64_t N,
                          int32_t* __restrict__ counts, int* err) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= L) return;
    const int32_t v = loaded[i];
    if (v < 0 || v >= N) {
        set_err(err, kErrRange, (int)i);
        return;
    }
    atomicAdd(&counts[v], 1);
}

constexpr int kScanThreads = 1024;

__global__ __launch_bounds__(kScanThreads) void assign_slots(int64_t N, int64_t L,
                                                             int32_t* __restrict__ o2s,
                                                             int32_t* __restrict__ s2o,
                                                             int* err) {
    __shared__ int wave_cnt[kScanThreads / kWave];
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    int64_t run = 0;
    for (int64_t base = 0; base < N; base += kScanThreads) {
        const int64_t n = base + threadIdx.x;
        const int32_t c = n < N ? o2s[n] : 0;
        if (c > 1) set_err(err, kErrDuplicate, (int)n);
        const bool f = c >= 1;
        const unsigned long long m = __ballot(f);
        const unsigned long long below = lane == 0 ? 0ull : (m & ((~0ull) >> (64 - lane)));
        if (lane == 0) wave_cnt[w] = __popcll(m);
        __syncthreads();
        int before = 0, all = 0;
        for (int q = 0; q < kScanThreads / kWave; ++q) {
            before += q < w ? wave_cnt[q] : 0;
            all += wave_cnt[q];
        }
        __syncthreads();
        const int64_t slot = run + before + __popcll(below);
        if (n < N) {
            o2s[n] = f ? (int32_t)slot : -1;
            if (f && slot < L) s2o[slot] = (int32_t)n;
        }
        run += all;
    }
}

__global__ void gather_rows16(const uint8_t* __restrict__ wg, const uint8_t* __restrict__ wu,
                              int64_t row_bytes, const int32_t* __restrict__ s2o,
                              uint8_t* __restrict__ gu) {
    const int64_t s = blockIdx.x;
    const int64_t n = s2o[s];
    const uint8_t* g = wg + n * row_bytes;
    const uint8_t* u = wu + n * row_bytes;
    uint8_t* o = gu + s * 2 * row_bytes;
    for (int64_t c = (int64_t)threadIdx.x * 16; c < row_bytes; c += (int64_t)blockDim.x * 16) {
        st16(o + c, ld16(g + c));
        st16(o + row_bytes + c, ld16(u + c));
    }
}

template <typename T>
__global__ __launch_bounds__(256) void gather_cols(const T* __restrict__ wd, int64_t N, int64_t d,
                                                   const int32_t* __restrict__ s2o, int64_t L,
                                                   T* __restrict__ dc) {
    __shared__ T tile[64][65];
    __shared__ int32_t ids[64];
    const int64_t s0 = (int64_t)blockIdx.x * 64;
    const int64_t i0 = (int64_t)blockIdx.y * 64;
    const int tx = threadIdx.x & 63;
    const int ty = threadIdx.x >> 6;
    // no s2o: the identity (a transpose of [d][L] into [L][d])
    if (threadIdx.x < 64) ids[tx] = (s0 + tx < L) ? (s2o ? s2o[s0 + tx] : (int32_t)(s0 + tx)) : 0;
    __syncthreads();
    for (int r = ty; r < 64; r += 4) {
        const int64_t i = i0 + r;
        if (i < d && s0 + tx < L) tile[r][tx] = wd[i * N + ids[tx]];
    }
    __syncthreads();
    for (int r = ty; r < 64; r += 4) {
        const int64_t s = s0 + r;
        const int64_t i = i0 + tx;
        if (s < L && i < d) dc[s * d + i] = tile[tx][r];
    }
}

}  // namespace

hipError_t launch_compact_maps(const int32_t* loaded, int64_t L, int64_t N,
                               int32_t* slot_to_orig, int32_t* orig_to_slot, int* err,
                               hipStream_t s) {
    hipLaunchKernelGGL(fill_i32, dim3((unsigned)((N + 255) / 256)), dim3(256), 0, s,
                       orig_to_slot, N, 0);
    hipLaunchKernelGGL(count_ids, dim3((unsigned)((L + 255) / 256)), dim3(256), 0, s, loaded,
                       L, N, orig_to_slot, err);
    hipLaunchKernelGGL(assign_slots, dim3(1), dim3(kScanThreads), 0, s, N, L, orig_to_slot,
                       slot_to_orig, err);
    return hipGetLastError();
}

hipError_t launch_compact_gather(const void* w_gate, const void* w_up, const void* w_down,
                                 int64_t N, int64_t d, int esize, const int32_t* slot_to_orig,
                                 int64_t L, void* gate_up_c, void* down_c, hipStream_t s) {
    const int64_t row_bytes = d * esize;
    hipLaunchKernelGGL(gather_rows16, dim3((unsigned)L), dim3(256), 0, s,
                       static_cast<const uint8_t*>(w_gate), static_cast<const uint8_t*>(w_up),
                       row_bytes, slot_to_orig, static_cast<uint8_t*>(gate_up_c));
    dim3 grid((unsigned)((L + 63) / 64), (unsigned)((d + 63) / 64));
    if (esize == 2)
        hipLaunchKernelGGL(gather_cols<uint16_t>, grid, dim3(256), 0, s,
                           static_cast<const uint16_t*>(w_down), N, d, slot_to_orig, L,
                           static_cast<uint16_t*>(down_c));
    else
        hipLaunchKernelGGL(gather_cols<uint32_t>, grid, dim3(256), 0, s,
                           static_cast<const uint32_t*>(w_down), N, d, slot_to_orig, L,
                           static_cast<uint32_t*>(down_c));
    return hipGetLastError();
}

hipError_t launch_transpose_cols(const void* src, int64_t d, int64_t L, int esize, void* dst,
                                 hipStream_t s) {
    dim3 grid((unsigned)((L + 63) / 64), (unsigned)((d + 63) / 64));
    if (esize == 2)
        hipLaunchKernelGGL(gather_cols<uint16_t>, grid, dim3(256), 0, s,
                           static_cast<const uint16_t*>(src), L, d, (const int32_t*)nullptr, L,
                           static_cast<uint16_t*>(dst));
    else
        hipLaunchKernelGGL(gather_cols<uint32_t>, grid, dim3(256), 0, s,
                           static_cast<const uint32_t*>(src), L, d, (const int32_t*)nullptr, L,
                           static_cast<uint32_t*>(dst));
    return hipGetLastError();
}

}  // namespace si
