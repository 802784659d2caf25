// Neuron selection around the hot path: dynamic-set construction (Selective Computation
// section) and the profiler's scores (LLM Profiler section, Eq. 1).
//
//  - act_rows: the activation a[t][j] = SiLU(gate_j . x_t) * (up_j . x_t) of every loaded slot
//    for any storage type (one wave per (token, slot)); bf16 data use the MFMA tiles of
//    k_tiled.hip instead;
//  - col_abs_sum / add_rows: Eq. 1 sums |a| over tokens (float32 over at most 256 tokens) and
//    the partial rows of the token tiles in float64, in ascending order, into float64 scores;
//  - count_bits: how many tokens select each slot, from the tokens' top-alpha bitmaps (up to
//    32768 slots): one work-group per 32-slot word, wave ballots and a fixed-order sum, so the
//    count is exact and free of atomics; it also writes the counts as the keys of the pick;
//  - count_slots: the same from the tokens' top-alpha lists (more slots), one integer atomic
//    per id, so the result does not depend on their order;
//  - freq_keys: the frequency of each slot as a float key (exact below 2^24), static slots
//    (set in the bitmap) below every frequency;
//  - set_bits: a slot list as a bitmap (then listed in ascending order by the union scan);
//  - merge_file: out += s / tokens for one score file, file by file (float64);
//  - rank_scores: the position of each neuron in decreasing score (ties to the lower index,
//    NaN last), by counting the neurons ranked before it; exact and order-free.
#include "common.h"
#include "launch.h"

namespace si {

namespace {

template <typename T>
__device__ __forceinline__ float ldf(const T* p);
template <>
__device__ __forceinline__ float ldf<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float ldf<bf16_t>(const bf16_t* p) { return bf16_to_f32(*p); }
template <>
__device__ __forceinline__ float ldf<f16_t>(const f16_t* p) { return (float)*p; }

// Grid (ceil(L / 4), T), 256 threads: wave w takes slot 4 blockIdx.x + w of token blockIdx.y.
template <typename WT, typename XT>
__global__ __launch_bounds__(256) void act_rows(const XT* __restrict__ x, int64_t d,
                                                const WT* __restrict__ gu, int64_t L,
                                                float* __restrict__ out, int64_t ldo) {
    const int lane = threadIdx.x & 63;
    const int64_t j = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int64_t t = blockIdx.y;
    if (j >= L) return;
    const XT* xr = x + t * d;
    const WT* gr = gu + j * 2 * d;
    float g = 0.0f, u = 0.0f;
    for (int64_t c = lane; c < d; c += kWave) {
        const float xv = ldf(xr + c);
        g = fmaf(ldf(gr + c), xv, g);
        u = fmaf(ldf(gr + d + c), xv, u);
    }
    g = wave_sum(g);
    u = wave_sum(u);
    if (lane == 0) out[t * ldo + j] = silu_f32(g) * u;
}

// s[n] += sum over t = 0 .. T-1 of |A[t][n]| (A with row stride lda): float32 sums over
// blocks of 256 tokens, as the MFMA tiles form them, added in float64
__global__ __launch_bounds__(256) void col_abs_sum(const float* __restrict__ A, int64_t T,
                                                   int64_t N, int64_t lda,
                                                   double* __restrict__ s) {
    const int64_t n = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (n >= N) return;
    double tot = 0.0;
    for (int64_t t0 = 0; t0 < T; t0 += 256) {
        const int64_t t1 = (T - t0) < 256 ? T : t0 + 256;
        float v = 0.0f;
        for (int64_t t = t0; t < t1; ++t) v += fabsf(A[t * lda + n]);
        tot += (double)v;
    }
    s[n] += tot;
}

// s[n] += sum over r = 0 .. R-1 of P[r][n] (P with row stride ldp), in float64
__global__ __launch_bounds__(256) void add_rows(const float* __restrict__ P, int64_t R, int64_t N,
                                                int64_t ldp, double* __restrict__ s) {
    const int64_t n = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (n >= N) return;
    double v = 0.0;
    for (int64_t r = 0; r < R; ++r) v += (double)P[r * ldp + n];
    s[n] += v;
}

__global__ __launch_bounds__(256) void count_slots(const int32_t* __restrict__ ids, int64_t n,
                                                   int64_t L, int* __restrict__ counts) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    const int32_t v = ids[i];
    if (v >= 0 && v < L) atomicAdd(&counts[v], 1);
}

// Grid W, 256 threads. tb: T token bitmaps of W words each (row stride W). Work-group w sets,
// for slot i = 32 w + j < L, counts[i] = how many tokens have bit j of word w set, and keys[i]
// the same count as an unsigned key. Each wave counts a bit over its 64 tokens with a ballot;
// the four wave counts are added in wave order.
__global__ __launch_bounds__(256) void count_bits(const uint32_t* __restrict__ tb, int64_t T,
                                                  int64_t W, int64_t L, int* __restrict__ counts,
                                                  uint32_t* __restrict__ keys) {
    __shared__ int part[4][32];
    const int64_t w = blockIdx.x;
    const int lane = threadIdx.x & 63;
    const int wv = threadIdx.x >> 6;
    int mine = 0;  // lane j < 32: this wave's count of bit j
    for (int64_t t0 = 0; t0 < T; t0 += 256) {
        const int64_t t = t0 + threadIdx.x;
        const uint32_t v = t < T ? tb[t * W + w] : 0u;
#pragma unroll
        for (int j = 0; j < 32; ++j) {
            const int c = __popcll(__ballot((v >> j) & 1u));
            mine += lane == j ? c : 0;
        }
    }
    if (lane < 32) part[wv][lane] = mine;
    __syncthreads();
    if (threadIdx.x < 32) {
        const int64_t i = w * 32 + threadIdx.x;
        const int c = part[0][threadIdx.x] + part[1][threadIdx.x] + part[2][threadIdx.x] +
                      part[3][threadIdx.x];
        if (i < L) {
            counts[i] = c;
            keys[i] = (uint32_t)c;
        }
    }
}

// keys[i] = counts[i], or -1 for a static slot (bit i of the bitmap set): below every
// frequency, so the dynamic pick never takes it
__global__ __launch_bounds__(256) void freq_keys(const int* __restrict__ counts,
                                                 const uint32_t* __restrict__ static_bits,
                                                 int64_t L, float* __restrict__ keys) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < L) keys[i] = ((static_bits[i / 32] >> (i % 32)) & 1u) ? -1.0f : (float)counts[i];
}

// p[0 .. n) = v and q[0 .. m) = v
__global__ __launch_bounds__(256) void fill2_u32(uint32_t* __restrict__ p, int64_t n,
                                                 uint32_t* __restrict__ q, int64_t m,
                                                 uint32_t v) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n) p[i] = v;
    if (i < m) q[i] = v;
}

__global__ __launch_bounds__(256) void set_bits(const int32_t* __restrict__ ids, int64_t n,
                                                int64_t L, uint32_t* __restrict__ bits) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    const int32_t v = ids[i];
    if (v >= 0 && v < L) atomicOr(&bits[v >> 5], 1u << (v & 31));
}

__global__ __launch_bounds__(256) void merge_file(const double* __restrict__ s, int64_t N,
                                                  double tokens, int first,
                                                  double* __restrict__ out) {
    const int64_t n = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (n >= N) return;
    const double v = s[n] / tokens;
    out[n] = first ? v : out[n] + v;
}

// Order key of a float64 score, larger first: -0 and +0 equal, NaN below every number.
__device__ __forceinline__ uint64_t desc_key(double f) {
    if (f != f) return 0ull;
    uint64_t u = (uint64_t)__double_as_longlong(f);
    if ((u << 1) == 0ull) u = 0ull;
    return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}

// Grid ceil(N / 256): thread n counts the neurons ranked before n over LDS tiles of keys.
__global__ __launch_bounds__(256) void rank_scores(const double* __restrict__ s, int64_t N,
                                                   int32_t* __restrict__ order) {
    __shared__ uint64_t tk[256];
    const int64_t n = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const uint64_t kn = n < N ? desc_key(s[n]) : 0ull;
    int64_t before = 0;
    for (int64_t m0 = 0; m0 < N; m0 += 256) {
        __syncthreads();
        const int64_t m = m0 + threadIdx.x;
        tk[threadIdx.x] = m < N ? desc_key(s[m]) : 0ull;
        __syncthreads();
        const int64_t lim = (N - m0) < 256 ? (N - m0) : 256;
        for (int q = 0; q < lim; ++q) {
            const uint64_t km = tk[q];
            before += (km > kn) || (km == kn && m0 + q < n);
        }
    }
    if (n < N) order[before] = (int32_t)n;
}

inline unsigned blocks(int64_t n) { return (unsigned)((n + 255) / 256); }

// 16-bit data (bf16 or half, x and weights alike) with whole 16-byte K chunks and 32-bit
// buffer offsets take the MFMA tiles
inline bool mfma_ok(int xdt, int wdt, int64_t T, int64_t L, int64_t d) {
    return xdt == wdt && (wdt == 1 || wdt == 2) && d % 8 == 0 && tiled_supported(T, L, d);
}

}  // namespace

hipError_t launch_activations(const void* x, int xdt, int64_t T, int64_t d, const void* gate_up_c,
                              int64_t L, int wdt, float* out, int64_t ldo, hipStream_t s,
                              hipEvent_t ev0, hipEvent_t ev1) {
    if (T == 0 || L == 0) return hipSuccess;
    if (mfma_ok(xdt, wdt, T, L, d))
        return launch_activations_mfma(x, T, d, gate_up_c, L, wdt, out, ldo, 0, s, ev0, ev1);
    // grid y holds the tokens: at most 65535 per launch
    for (int64_t t0 = 0; t0 < T; t0 += 65535) {
        const int64_t nt = (T - t0) < 65535 ? (T - t0) : 65535;
        const dim3 grid((unsigned)((L + 3) / 4), (unsigned)nt);
        const int64_t xo = t0 * d;
        float* o = out + t0 * ldo;
#define SI_ACT(WT, XT)                                                                          \
    hipLaunchKernelGGL((act_rows<WT, XT>), grid, dim3(256), 0, s,                              \
                       static_cast<const XT*>(x) + xo, d, static_cast<const WT*>(gate_up_c), L, \
                       o, ldo)
        if (wdt == 1 && xdt == 1)
            SI_ACT(bf16_t, bf16_t);
        else if (wdt == 1 && xdt == 0)
            SI_ACT(bf16_t, float);
        else if (wdt == 0 && xdt == 1)
            SI_ACT(float, bf16_t);
        else if (wdt == 2 && xdt == 2)
            SI_ACT(f16_t, f16_t);
        else if (wdt == 2 && xdt == 0)
            SI_ACT(f16_t, float);
        else if (wdt == 0 && xdt == 2)
            SI_ACT(float, f16_t);
        else if (wdt == 0 && xdt == 0)
            SI_ACT(float, float);
        else
            return hipErrorInvalidValue;  // bf16 with half: not a supported pair
    }
#undef SI_ACT
    return hipGetLastError();
}

size_t score_workspace(int64_t T, int64_t N, int64_t d, int xdt, int wdt) {
    const int64_t ldo = (N + 63) / 64 * 64;
    if (mfma_ok(xdt, wdt, T, N, d)) return (size_t)activation_tiles_max(T) * ldo * 4;  // per tile
    return (size_t)T * ldo * 4;                         // the activations themselves
}

hipError_t launch_scores(const void* x, int xdt, int64_t T, int64_t d, const void* gate_up,
                         int64_t N, int wdt, double* scores, void* ws, hipStream_t s,
                         hipEvent_t ev0, hipEvent_t ev1) {
    if (T == 0 || N == 0) return hipSuccess;
    const int64_t ldo = (N + 63) / 64 * 64;
    float* buf = static_cast<float*>(ws);
    hipError_t e;
    if (mfma_ok(xdt, wdt, T, N, d)) {
        e = launch_activations_mfma(x, T, d, gate_up, N, wdt, buf, ldo, 1, s, ev0, ev1);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(add_rows, dim3(blocks(N)), dim3(256), 0, s, buf,
                           (int64_t)activation_tiles(T, N), N, ldo, scores);
    } else {
        e = launch_activations(x, xdt, T, d, gate_up, N, wdt, buf, ldo, s);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(col_abs_sum, dim3(blocks(N)), dim3(256), 0, s, buf, T, N, ldo, scores);
    }
    return hipGetLastError();
}

DynPlan dyn_plan(int64_t T, int64_t L, int64_t alpha, int64_t n_total) {
    DynPlan p;
    auto al = [](size_t v) { return (v + 255) & ~(size_t)255; };
    p.lda = (L + 63) / 64 * 64;
    p.W = (L + 31) / 32;
    size_t o = 0;
    p.off_act = o;
    o = al(o + (size_t)T * p.lda * 4);
    // the tokens' top-alpha choices: bitmaps of W words up to 32768 slots, else lists
    p.token_bits = L <= kTokenBitsMaxL;
    p.off_lists = o;
    o = al(o + (size_t)T * (p.token_bits ? p.W : alpha) * 4);
    p.off_counts = o;
    o = al(o + (size_t)L * 4);
    p.off_keys = o;
    o = al(o + (size_t)L * 4);
    p.off_dyn = o;
    o = al(o + (size_t)(n_total > 0 ? n_total : 1) * 4);
    p.off_bits = o;
    o = al(o + (size_t)p.W * 4);
    p.off_count = o;
    o = al(o + 4);
    p.total = o;
    return p;
}

hipError_t launch_dynamic_set(const void* x, int xdt, int64_t T, int64_t d, const void* gate_up_c,
                              int64_t L, int wdt, const int32_t* static_slots, int64_t n_static,
                              int64_t alpha, int64_t n_total, int key, int32_t* out,
                              int32_t* counts_out, void* ws, hipStream_t s, hipEvent_t ev0,
                              hipEvent_t ev1) {
    const DynPlan p = dyn_plan(T, L, alpha, n_total);
    uint8_t* base = static_cast<uint8_t*>(ws);
    float* act = reinterpret_cast<float*>(base + p.off_act);
    int32_t* lists = reinterpret_cast<int32_t*>(base + p.off_lists);
    int* counts = counts_out ? counts_out : reinterpret_cast<int*>(base + p.off_counts);
    float* keys = reinterpret_cast<float*>(base + p.off_keys);
    int32_t* dyn = reinterpret_cast<int32_t*>(base + p.off_dyn);
    uint32_t* bits = reinterpret_cast<uint32_t*>(base + p.off_bits);
    int* cnt = reinterpret_cast<int*>(base + p.off_count);
    hipError_t e;
    const int64_t kd = n_total - n_static;  // dynamic slots to add to the static ones
    // 1. activations of every loaded slot, per token
    if (alpha > 0) {
        e = launch_activations(x, xdt, T, d, gate_up_c, L, wdt, act, p.lda, s, ev0, ev1);
        if (e != hipSuccess) return e;
    }
    if (p.token_bits) {
        // 2. each token's top alpha by |a| or a (key) as a bitmap; 3. counts (the keys of the
        //    pick) per 32-slot word; 4. the static slots joined with the dynamic pick among the
        //    others, ascending
        uint32_t* tbits = reinterpret_cast<uint32_t*>(lists);
        const int64_t Tr = alpha > 0 ? T : 0;
        e = launch_topk_bitmap(act, Tr, L, p.lda, alpha, key, tbits, p.W, s);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(count_bits, dim3((unsigned)p.W), dim3(256), 0, s, tbits, Tr, p.W, L,
                           counts, reinterpret_cast<uint32_t*>(keys));
        // the static slots are not candidates of the pick (mode 2: the keys are counts)
        return launch_topk_join(keys, L, kd, 2, static_slots, n_static, out, n_total, cnt, s);
    }
    // counts and the bitmap start at zero; the bitmap takes the static slots
    hipLaunchKernelGGL(fill2_u32, dim3(blocks(L > p.W ? L : p.W)), dim3(256), 0, s,
                       reinterpret_cast<uint32_t*>(counts), L, bits, p.W, 0u);
    if (n_static > 0)
        hipLaunchKernelGGL(set_bits, dim3(blocks(n_static)), dim3(256), 0, s, static_slots,
                           n_static, L, bits);
    // 2. each token's top alpha by |a| or a (key); 3. how often each slot is chosen (atomics
    //    on the ids)
    if (T > 0 && alpha > 0) {
        e = launch_topk_strided(act, T, L, p.lda, alpha, key, lists, s);
        if (e != hipSuccess) return e;
        const int64_t n = T * alpha;
        hipLaunchKernelGGL(count_slots, dim3(blocks(n)), dim3(256), 0, s, lists, n, L, counts);
    }
    hipLaunchKernelGGL(freq_keys, dim3(blocks(L)), dim3(256), 0, s, counts, bits, L, keys);
    // 4. the most frequent non-static slots, n_total - n_static of them
    if (kd > 0) {
        e = launch_topk(keys, 1, L, kd, 1, dyn, s);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(set_bits, dim3(blocks(kd)), dim3(256), 0, s, dyn, kd, L, bits);
    }
    // 5. static u dynamic, ascending
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_bits_to_list(bits, p.W, out, cnt, s);
}

hipError_t launch_merge_file(const double* sc, int64_t N, double tokens, int first, double* out,
                             hipStream_t s) {
    hipLaunchKernelGGL(merge_file, dim3(blocks(N)), dim3(256), 0, s, sc, N, tokens, first, out);
    return hipGetLastError();
}

hipError_t launch_rank(const double* sc, int64_t N, int32_t* order, hipStream_t s) {
    if (N == 0) return hipSuccess;
    hipLaunchKernelGGL(rank_scores, dim3(blocks(N)), dim3(256), 0, s, sc, N, order);
    return hipGetLastError();
}

}  // namespace si
