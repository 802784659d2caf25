// Per-token top-k over the loaded neurons (dynamic-neuron selection, Selective Computation
// section): for each score row, the k slots with the largest key, returned in ascending order.
//
// Order: key = |s| (ABS) or s (RAW); larger key first; equal keys -> lower index first;
// -0 == +0; NaN after every number. Each float key is mapped to a uint32 whose unsigned order
// is that order (NaN -> 0). One 1024-thread work-group per row:
//   1. radix select, 4 passes of 8 bits from the top: a histogram of the candidates that
//      match the prefix found so far gives the next byte of the k-th largest key T and how
//      many keys equal to T must still be taken (take_eq);
//   2. selection in index order: an element is selected iff key > T, or key == T and fewer
//      than take_eq equal keys precede it; block-wide prefix counts give each selected element
//      its output position, so the output is ascending without a sort.
// Rows of up to 16384 keys (topk_rows_reg): thread t holds the C contiguous keys t*C .. in
// registers, read once; each wave counts into its own LDS histogram (16 x 256 bins), the bins
// are added in wave order and searched with a wave-wide suffix scan; the selection takes two
// block-wide scans of per-thread counts. Longer rows (topk_rows) re-read the row from memory
// in each pass.
#include "common.h"
#include "launch.h"

namespace si {

namespace {

constexpr int kTopkThreads = 1024;
constexpr int kTopkWaves = kTopkThreads / kWave;

// Integer-only mapping, so no floating-point mode can change how -0 or NaN are treated.
__device__ __forceinline__ uint32_t order_key(float v, int mode) {
    uint32_t u = __float_as_uint(v);
    if (mode == 0) u &= 0x7fffffffu;                 // |v|
    const uint32_t mag = u & 0x7fffffffu;
    if (mag > 0x7f800000u) return 0u;                // NaN: below every number
    if (mag == 0u) u = 0u;                           // -0 -> +0
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Exclusive prefix count of `flag` over the block in thread order; returns the prefix and
// writes the block total to *total. Uses wave ballots and a scan of the 16 wave counts.
__device__ __forceinline__ int block_prefix(bool flag, int* wave_cnt, int* total) {
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    const unsigned long long m = __ballot(flag);
    const unsigned long long below = lane == 0 ? 0ull : (m & ((~0ull) >> (64 - lane)));
    const int in_wave = __popcll(below);
    if (lane == 0) wave_cnt[w] = __popcll(m);
    __syncthreads();
    int before = 0, all = 0;
#pragma unroll
    for (int q = 0; q < kTopkWaves; ++q) {
        const int c = wave_cnt[q];
        before += q < w ? c : 0;
        all += c;
    }
    __syncthreads();
    *total = all;
    return before + in_wave;
}

__global__ __launch_bounds__(kTopkThreads) void topk_rows(const float* __restrict__ scores,
                                                         int64_t L, int64_t ld, int64_t k,
                                                         int mode, int32_t* __restrict__ out) {
    const int64_t b = blockIdx.x;
    const float* row = scores + b * ld;
    int32_t* orow = out + b * k;
    __shared__ int hist[256];
    __shared__ int wave_cnt[kTopkWaves];
    __shared__ uint32_t s_prefix;
    __shared__ int64_t s_take;

    uint32_t prefix = 0u, pmask = 0u;
    int64_t take = k;  // how many still to take among candidates matching the prefix
#pragma unroll 1
    for (int shift = 24; shift >= 0; shift -= 8) {
        for (int i = threadIdx.x; i < 256; i += kTopkThreads) hist[i] = 0;
        __syncthreads();
        for (int64_t i = threadIdx.x; i < L; i += kTopkThreads) {
            const uint32_t key = order_key(row[i], mode);
            if ((key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1);
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            int64_t above = 0;
            int dsel = 0;
            for (int dg = 255; dg >= 0; --dg) {
                const int64_t c = hist[dg];
                if (above + c >= take) {
                    dsel = dg;
                    break;
                }
                above += c;
            }
            s_prefix = prefix | ((uint32_t)dsel << shift);
            s_take = take - above;
        }
        __syncthreads();
        prefix = s_prefix;
        take = s_take;
        pmask |= 255u << shift;
        __syncthreads();
    }
    const uint32_t T = prefix;

    int64_t run_eq = 0, run_sel = 0;
    for (int64_t base = 0; base < L; base += kTopkThreads) {
        const int64_t i = base + threadIdx.x;
        const uint32_t key = i < L ? order_key(row[i], mode) : 0u;
        const bool gt = i < L && key > T;
        const bool eq = i < L && key == T;
        int eq_total;
        const int eq_rank = block_prefix(eq, wave_cnt, &eq_total);
        const bool sel = gt || (eq && run_eq + eq_rank < take);
        int sel_total;
        const int pos = block_prefix(sel, wave_cnt, &sel_total);
        if (sel && run_sel + pos < k) orow[run_sel + pos] = (int32_t)i;
        run_eq += eq_total;
        run_sel += sel_total;
    }
}

// Inclusive prefix sum over the lanes of a wave (lane order).
__device__ __forceinline__ int wave_incl_scan(int v) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int m = 1; m < kWave; m <<= 1) {
        const int o = __shfl_up(v, m, kWave);
        v += lane >= m ? o : 0;
    }
    return v;
}

// Exclusive prefix sum of v over the block in thread order; *total = block sum. Two barriers.
__device__ __forceinline__ int block_excl_scan(int v, int* wave_tot, int* total) {
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    const int incl = wave_incl_scan(v);
    if (lane == kWave - 1) wave_tot[w] = incl;
    __syncthreads();
    int before = 0, all = 0;
#pragma unroll
    for (int q = 0; q < kTopkWaves; ++q) {
        const int c = wave_tot[q];
        before += q < w ? c : 0;
        all += c;
    }
    __syncthreads();
    *total = all;
    return before + incl - v;
}

template <int C>
__global__ __launch_bounds__(kTopkThreads) void topk_rows_reg(const float* __restrict__ scores,
                                                             int64_t L, int64_t ld, int64_t k,
                                                             int mode,
                                                             int32_t* __restrict__ out) {
    const int64_t b = blockIdx.x;
    const float* row = scores + b * ld;
    int32_t* orow = out + b * k;
    const int t = threadIdx.x;
    const int lane = t & 63;
    const int w = t >> 6;
    __shared__ int hist[kTopkWaves][256];
    __shared__ int tot[256];
    __shared__ int wave_tot[kTopkWaves];
    __shared__ uint32_t s_prefix;
    __shared__ int s_take;

    // keys t*C .. t*C + C - 1; past L: never a candidate (valid = false)
    uint32_t key[C];
#pragma unroll
    for (int j = 0; j < C; ++j) {
        const int64_t i = (int64_t)t * C + j;
        key[j] = i < L ? order_key(row[i], mode) : 0u;
    }
    const int64_t rest = L - (int64_t)t * C;  // keys of the row from this thread's first on
    const int nvalid = rest <= 0 ? 0 : (rest < C ? (int)rest : C);

    uint32_t prefix = 0u, pmask = 0u;
    int take = (int)k;  // how many still to take among the keys matching the prefix
#pragma unroll 1
    for (int shift = 24; shift >= 0; shift -= 8) {
        for (int q = t; q < kTopkWaves * 256; q += kTopkThreads) (&hist[0][0])[q] = 0;
        __syncthreads();
#pragma unroll
        for (int j = 0; j < C; ++j)
            if (j < nvalid && (key[j] & pmask) == prefix)
                atomicAdd(&hist[w][(key[j] >> shift) & 255u], 1);
        __syncthreads();
        if (t < 256) {
            int c = 0;
#pragma unroll
            for (int q = 0; q < kTopkWaves; ++q) c += hist[q][t];
            tot[t] = c;
        }
        __syncthreads();
        if (w == 0) {
            // lane l owns digits 255 - 4l .. 252 - 4l (descending); `above` = keys with a
            // larger digit
            int c4[4], sum = 0;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                c4[e] = tot[255 - 4 * lane - e];
                sum += c4[e];
            }
            int above = wave_incl_scan(sum) - sum;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                if (above < take && above + c4[e] >= take) {  // exactly one digit qualifies
                    s_prefix = prefix | ((uint32_t)(255 - 4 * lane - e) << shift);
                    s_take = take - above;
                }
                above += c4[e];
            }
        }
        __syncthreads();
        prefix = s_prefix;
        take = s_take;
        pmask |= 255u << shift;
    }
    const uint32_t T = prefix;

    int n_eq = 0;
#pragma unroll
    for (int j = 0; j < C; ++j) n_eq += (j < nvalid && key[j] == T) ? 1 : 0;
    int eq_all;
    int eq_before = block_excl_scan(n_eq, wave_tot, &eq_all);
    bool sel[C];
    int n_sel = 0;
#pragma unroll
    for (int j = 0; j < C; ++j) {
        const bool ok = j < nvalid;
        const bool eq = ok && key[j] == T;
        sel[j] = ok && (key[j] > T || (eq && eq_before < take));
        eq_before += eq ? 1 : 0;
        n_sel += sel[j] ? 1 : 0;
    }
    int sel_all;
    int pos = block_excl_scan(n_sel, wave_tot, &sel_all);
#pragma unroll
    for (int j = 0; j < C; ++j) {
        if (sel[j] && pos < k) orow[pos] = (int32_t)((int64_t)t * C + j);
        pos += sel[j] ? 1 : 0;
    }
}

}  // namespace

hipError_t launch_topk_strided(const float* scores, int64_t B, int64_t L, int64_t ld, int64_t k,
                               int mode, int32_t* out, hipStream_t s) {
    if (B == 0 || k == 0) return hipSuccess;
    const int64_t per = (L + kTopkThreads - 1) / kTopkThreads;  // keys per thread
#define SI_TOPK_REG(C)                                                                          \
    hipLaunchKernelGGL(topk_rows_reg<C>, dim3((unsigned)B), dim3(kTopkThreads), 0, s, scores, L, \
                       ld, k, mode, out)
    if (per <= 1)
        SI_TOPK_REG(1);
    else if (per <= 2)
        SI_TOPK_REG(2);
    else if (per <= 4)
        SI_TOPK_REG(4);
    else if (per <= 8)
        SI_TOPK_REG(8);
    else if (per <= 16)
        SI_TOPK_REG(16);
    else
        hipLaunchKernelGGL(topk_rows, dim3((unsigned)B), dim3(kTopkThreads), 0, s, scores, L, ld,
                           k, mode, out);
#undef SI_TOPK_REG
    return hipGetLastError();
}

hipError_t launch_topk(const float* scores, int64_t B, int64_t L, int64_t k, int mode,
                       int32_t* out, hipStream_t s) {
    return launch_topk_strided(scores, B, L, L, k, mode, out, s);
}

}  // namespace si
