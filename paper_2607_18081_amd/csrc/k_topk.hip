// Per-token top-k over the loaded neurons (dynamic-neuron selection, Selective Computation
// section): for each score row, the k slots with the largest key, returned in ascending order.
//
// Order: key = |s| (ABS) or s (RAW); larger key first; equal keys -> lower index first;
// -0 == +0; NaN after every number. Each float key is mapped to a uint32 whose unsigned order
// is that order (NaN -> 0); counts are taken as unsigned integers directly. One 1024-thread
// work-group per row:
//   1. radix select over 8-bit digits from the top: a histogram of the candidates that match
//      the prefix found so far gives the next digit of the k-th largest key T and how many
//      keys equal to T must still be taken (take_eq);
//   2. selection in index order: an element is selected iff key > T, or key == T and fewer
//      than take_eq equal keys precede it; block-wide prefix counts give each selected element
//      its output position, so the output is ascending without a sort.
// Rows of up to 32768 keys (topk_rows_reg): thread t holds the C contiguous keys t*C .. in
// registers, read once; each wave counts into its own LDS histogram (16 x 256 bins), the bins
// are added in wave order and every wave searches them with a DPP scan (two barriers a pass).
// The digits start below the bits all candidates share, the search stops once the whole
// bucket of T's prefix is taken (the lower bits cannot change the choice), and then the
// selection needs no scan of equal keys. The choice can also be written as a bitmap per row,
// or joined with a given set. Longer rows (topk_rows) re-read the row in each of 4 passes.
#include "common.h"
#include "launch.h"

namespace si {

namespace {

constexpr int kTopkThreads = 1024;
constexpr int kTopkWaves = kTopkThreads / kWave;

// Integer-only mapping, so no floating-point mode can change how -0 or NaN are treated.
// mode 0: |v|, 1: v, 2: the 32 bits as an unsigned integer (counts).
__device__ __forceinline__ uint32_t order_key(float v, int mode) {
    uint32_t u = __float_as_uint(v);
    if (mode == 2) return u;
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

// What a register-resident launch writes (exactly one of idx, bmp, ulist is set):
struct TopkOut {
    int32_t* idx;  // [B][k] the chosen indices, ascending
    uint32_t* bmp;  // [B][bW] a bitmap per row: bit j of word w set iff slot 32 w + j is chosen
    int64_t bW;
    // one row: the set join_ids[0 .. n_join) (ids outside [0, L) ignored) joined with the k
    // chosen among the other keys, ascending, at most ucap of them -> ulist, their number ->
    // *ucount
    const int32_t* join_ids;
    int64_t n_join;
    int32_t* ulist;
    int64_t ucap;
    int* ucount;
};

constexpr int kMaxRegKeys = 32 * kTopkThreads;  // the register-resident kernel's longest row

// vec: the rows are 16-byte aligned, so a thread's C keys are read as float4s.
template <int C>
__global__ __launch_bounds__(kTopkThreads) void topk_rows_reg(const float* __restrict__ scores,
                                                             int64_t L, int64_t ld, int64_t k,
                                                             int mode, int vec, TopkOut o) {
    static_assert(32 % C == 0, "a thread's keys lie in one bitmap word");
    constexpr int kStride = 257;  // one histogram per wave, a bank apart
    const int64_t b = blockIdx.x;
    const int t = threadIdx.x;
    const int lane = t & 63;
    const int w = t >> 6;
    __shared__ int hist[kTopkWaves * kStride];
    __shared__ int tot[256];
    __shared__ int wave_tot[kTopkWaves];
    __shared__ uint32_t s_or[kTopkWaves], s_and[kTopkWaves];
    __shared__ uint32_t jbits[kMaxRegKeys / 32];
    if (o.ulist) {  // the joined set as a bitmap
        for (int q = t; q < kMaxRegKeys / 32; q += kTopkThreads) jbits[q] = 0u;
        __syncthreads();
        for (int64_t i = t; i < o.n_join; i += kTopkThreads) {
            const int32_t v = o.join_ids[i];
            if (v >= 0 && v < L) atomicOr(&jbits[v >> 5], 1u << (v & 31));
        }
        __syncthreads();
    }
    const float* row = scores + b * ld;
    // keys t*C .. t*C + C - 1 (the first nvalid of them lie in the row)
    uint32_t key[C];
    const int64_t rest = L - (int64_t)t * C;
    const int nvalid = rest <= 0 ? 0 : (rest < C ? (int)rest : C);
    if (C % 4 == 0 && vec && nvalid == C) {
        const float4* r4 = reinterpret_cast<const float4*>(row + (int64_t)t * C);
#pragma unroll
        for (int q = 0; q < C / 4; ++q) {
            const float4 v = r4[q];
            key[4 * q] = order_key(v.x, mode);
            key[4 * q + 1] = order_key(v.y, mode);
            key[4 * q + 2] = order_key(v.z, mode);
            key[4 * q + 3] = order_key(v.w, mode);
        }
    } else {
#pragma unroll
        for (int j = 0; j < C; ++j)
            key[j] = j < nvalid ? order_key(row[(int64_t)t * C + j], mode) : 0u;
    }
    // candidates: the keys in the row, less (join mode) the slots of the joined set
    const uint32_t vmask = nvalid >= 32 ? ~0u : (1u << nvalid) - 1u;  // keys in the row
    uint32_t cand = k > 0 ? vmask : 0u;
    const uint32_t jw = (o.ulist && nvalid > 0) ? jbits[(t * C) / 32] >> ((t * C) & 31) : 0u;
    cand &= ~jw;
    // bits common to every candidate need no pass: the search starts at the highest bit in
    // which two candidates differ
    uint32_t kor = 0u, kand = ~0u;
#pragma unroll
    for (int j = 0; j < C; ++j)
        if ((cand >> j) & 1u) {
            kor |= key[j];
            kand &= key[j];
        }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
        kor |= (uint32_t)__shfl_xor((int)kor, m, kWave);
        kand &= (uint32_t)__shfl_xor((int)kand, m, kWave);
    }
    if (lane == 0) {
        s_or[w] = kor;
        s_and[w] = kand;
    }
    for (int q = t; q < kTopkWaves * kStride; q += kTopkThreads) hist[q] = 0;
    __syncthreads();
#pragma unroll
    for (int q = 0; q < kTopkWaves; ++q) {
        kor |= s_or[q];
        kand &= s_and[q];
    }
    const uint32_t diff = kor ^ kand;
    const int top = diff ? 31 - __clz((int)diff) : -1;  // -1: all candidates equal (or none)
    // the bits above `top`, decided before the first pass
    uint32_t pmask = top < 0 ? ~0u : (top >= 31 ? 0u : ~((2u << top) - 1u));
    uint32_t prefix = kand & pmask;
    int* my_hist = hist + w * kStride;
    int take = (int)k;   // how many still to take among the candidates matching the prefix
    bool done = k == 0;  // every candidate matching the prefix is taken: no further pass
#pragma unroll 1
    for (int hi = top; hi >= 0 && !done; hi -= 8) {
        // this pass decides bits lo .. hi (8 of them, fewer at the bottom)
        const int lo = hi >= 7 ? hi - 7 : 0;
        const uint32_t dmask = (1u << (hi - lo + 1)) - 1u;
        // 1. count the candidates by digit into the wave's histogram; a run of equal digits
        //    in a thread's keys is added at once (few distinct digits would serialise the
        //    atomics on one bin)
        int cur = -1, cnt = 0;
#pragma unroll
        for (int j = 0; j < C; ++j) {
            if (((cand >> j) & 1u) && (key[j] & pmask) == prefix) {
                const int dg = (int)((key[j] >> lo) & dmask);
                if (dg != cur) {
                    if (cnt) atomicAdd(&my_hist[cur], cnt);
                    cur = dg;
                    cnt = 0;
                }
                ++cnt;
            }
        }
        if (cnt) atomicAdd(&my_hist[cur], cnt);
        __syncthreads();
        // 2. bins added in wave order; the histograms are cleared for the next pass
        if (t < 256) {
            int c = 0;
#pragma unroll
            for (int q = 0; q < kTopkWaves; ++q) {
                c += hist[q * kStride + t];
                hist[q * kStride + t] = 0;
            }
            tot[t] = c;
        }
        __syncthreads();
        // 3. every wave finds the digit of the k-th key itself (the same result in each, so
        //    no third barrier): lane l owns digits 255 - 4l .. 252 - 4l, `above` counts the
        //    keys with a larger digit, exactly one digit qualifies. tot is rewritten only after
        //    the next pass's first barrier, which every wave reaches after reading it.
        int c4[4], sum = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            c4[e] = tot[255 - 4 * lane - e];
            sum += c4[e];
        }
        int above = wave_incl_scan(sum) - sum;
        int found = 0, dsel = 0, tsel = 0, dn = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if (above < take && above + c4[e] >= take) {
                found = 1;
                dsel = 255 - 4 * lane - e;
                tsel = take - above;
                dn = tsel == c4[e];
            }
            above += c4[e];
        }
        const unsigned long long fm = __ballot(found);
        if (fm == 0ull) {  // k above the number of candidates: every candidate is taken
            done = true;
            break;
        }
        const int src = __ffsll((long long)fm) - 1;
        prefix |= (uint32_t)__builtin_amdgcn_readlane(dsel, src) << lo;
        take = __builtin_amdgcn_readlane(tsel, src);
        done = __builtin_amdgcn_readlane(dn, src) != 0;
        pmask |= dmask << lo;
    }
    // keys compare on the bits decided
    const uint32_t T = prefix;
#pragma unroll
    for (int j = 0; j < C; ++j) key[j] &= pmask;
    uint32_t sel = 0u;  // bit j: key t*C + j is chosen
    if (done) {  // every candidate equal to T is taken
#pragma unroll
        for (int j = 0; j < C; ++j) sel |= (((cand >> j) & 1u) && key[j] >= T) ? 1u << j : 0u;
    } else {  // the first `take` candidates equal to T in index order
        int n_eq = 0;
#pragma unroll
        for (int j = 0; j < C; ++j) n_eq += (((cand >> j) & 1u) && key[j] == T) ? 1 : 0;
        int eq_all;
        int eq_before = block_excl_scan(n_eq, wave_tot, &eq_all);
#pragma unroll
        for (int j = 0; j < C; ++j) {
            const bool ok = (cand >> j) & 1u;
            const bool eq = ok && key[j] == T;
            sel |= (ok && (key[j] > T || (eq && eq_before < take))) ? 1u << j : 0u;
            eq_before += eq ? 1 : 0;
        }
    }
    if (o.bmp) {
        // the 32 / C threads of one word (consecutive lanes) OR their bits together
        uint32_t m = C == 32 ? sel : sel << ((t * C) & 31);
#pragma unroll
        for (int q = 1; q < 32 / C; q <<= 1) m |= (uint32_t)__shfl_xor((int)m, q, kWave);
        const int64_t wd = ((int64_t)t * C) / 32;
        if (((t * C) & 31) == 0 && wd < o.bW) o.bmp[b * o.bW + wd] = m;
        return;
    }
    int64_t cap = k;
    int32_t* orow = o.ulist;
    if (!o.ulist) {
        orow = o.idx + b * k;
    } else {
        sel |= jw & vmask;  // join the bits of o.join (none of them a candidate)
        cap = o.ucap;
    }
    int sel_all;
    int pos = block_excl_scan(__popc(sel), wave_tot, &sel_all);
#pragma unroll
    for (int j = 0; j < C; ++j) {
        const bool on = (sel >> j) & 1u;
        if (on && pos < cap) orow[pos] = (int32_t)((int64_t)t * C + j);
        pos += on ? 1 : 0;
    }
    if (o.ulist && t == 0) *o.ucount = sel_all < cap ? sel_all : (int)cap;
}

}  // namespace

namespace {

// One register-resident launch: C keys per thread (L <= 1024 C), one work-group per row.
template <int C>
void launch_reg_c(const float* scores, int64_t B, int64_t L, int64_t ld, int64_t k, int mode,
                  const TopkOut& o, hipStream_t s) {
    const bool al = reinterpret_cast<uintptr_t>(scores) % 16 == 0;
    const int vec = (al && (B <= 1 || ld % 4 == 0)) ? 1 : 0;
    hipLaunchKernelGGL(topk_rows_reg<C>, dim3((unsigned)B), dim3(kTopkThreads), 0, s, scores, L,
                       ld, k, mode, vec, o);
}

// false when a row has more than 32768 keys
bool launch_reg(const float* scores, int64_t B, int64_t L, int64_t ld, int64_t k, int mode,
                const TopkOut& o, hipStream_t s) {
    const int64_t per = (L + kTopkThreads - 1) / kTopkThreads;  // keys per thread
    if (per <= 1)
        launch_reg_c<1>(scores, B, L, ld, k, mode, o, s);
    else if (per <= 2)
        launch_reg_c<2>(scores, B, L, ld, k, mode, o, s);
    else if (per <= 4)
        launch_reg_c<4>(scores, B, L, ld, k, mode, o, s);
    else if (per <= 8)
        launch_reg_c<8>(scores, B, L, ld, k, mode, o, s);
    else if (per <= 16)
        launch_reg_c<16>(scores, B, L, ld, k, mode, o, s);
    else if (per <= 32)
        launch_reg_c<32>(scores, B, L, ld, k, mode, o, s);
    else
        return false;
    return true;
}

}  // namespace

hipError_t launch_topk_strided(const float* scores, int64_t B, int64_t L, int64_t ld, int64_t k,
                               int mode, int32_t* out, hipStream_t s) {
    if (B == 0 || k == 0) return hipSuccess;
    TopkOut o{};
    o.idx = out;
    if (!launch_reg(scores, B, L, ld, k, mode, o, s))
        hipLaunchKernelGGL(topk_rows, dim3((unsigned)B), dim3(kTopkThreads), 0, s, scores, L, ld,
                           k, mode, out);
    return hipGetLastError();
}

hipError_t launch_topk_bitmap(const float* scores, int64_t B, int64_t L, int64_t ld, int64_t k,
                              int mode, uint32_t* bits, int64_t W, hipStream_t s) {
    if (B == 0) return hipSuccess;
    TopkOut o{};
    o.bmp = bits;
    o.bW = W;
    // every word of a row is written by the kernel: W must be exactly the row's word count
    if (W != (L + 31) / 32 || !launch_reg(scores, B, L, ld, k, mode, o, s))
        return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t launch_topk_join(const float* scores, int64_t L, int64_t k, int mode,
                            const int32_t* join_ids, int64_t n_join, int32_t* list, int64_t cap,
                            int* count, hipStream_t s) {
    TopkOut o{};
    o.join_ids = join_ids;
    o.n_join = n_join;
    o.ulist = list;
    o.ucap = cap;
    o.ucount = count;
    if (!launch_reg(scores, 1, L, L, k, mode, o, s)) return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t launch_topk(const float* scores, int64_t B, int64_t L, int64_t k, int mode,
                       int32_t* out, hipStream_t s) {
    return launch_topk_strided(scores, B, L, L, k, mode, out, s);
}

}  // namespace si
