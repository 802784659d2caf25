// Per-token path of the selective SwiGLU FFN (Selective Computation section).
//
// For one token with active slots A and compacted weights gate_up_c [L][2][d], down_c [L][d]:
//     h_j = SiLU(gate_j . x) * (up_j . x),   y = sum_{j in A} h_j * down_j.
//
// Kernel 1 (sffn_rows): work-group (p, b) takes chunk p of token b's active list. Its 8 waves
// split the d columns: wave w, lane l own the 16-byte column groups ((i*8 + w)*64 + l), so a
// row is read as one fully coalesced sweep of the work-group. For a batch of up to R rows the
// work-group issues every gate and up load of the batch, then every down load (the down rows
// do not depend on h, so they stream in while the dot products complete), reduces each row's two dot
// products across the wave with a transposing shuffle reduction and across the 8 waves through
// LDS, applies SiLU*up, and accumulates h_j * down_j into per-lane float32 registers. The
// work-group's partial sum over its rows is written to the workspace in the column-chunked
// partial layout (common.h).
//
// Kernel 2 (reduce_chunks) adds the P partials of each token in a fixed order, so the result
// is deterministic and no global atomics are used.
#include <hip/hip_ext.h>

#include <type_traits>

#include "common.h"
#include "launch.h"

namespace si {

namespace {

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * kWave;

// Rows whose loads a work-group issues together: 3 * R * NI 16-byte loads per lane stay in
// registers. A stacked-layer instance (RN) also holds the residual r until the normalisation,
// so beyond the one-group bf16 case it takes smaller batches and never spills.
template <typename XT, int NI, bool RN>
struct RowsPerBatch {
    static constexpr bool lean = RN && !(sizeof(XT) == 2 && NI == 1);
    static constexpr int value = lean ? (NI == 1 ? 8 : NI == 2 ? 4 : NI == 3 ? 2 : 1)
                                      : (NI == 1 ? 16 : NI == 2 ? 8 : NI == 3 ? 4 : 2);
};

typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;

// The token's x restricted to one lane's 16-byte column group, in the form its dot products
// use: packed bf16 pairs when both x and the weights are bf16 (v_dot2_f32_bf16), else float.
// Loaded through a buffer descriptor over the token's row, so a lane outside the row passes
// kOOB and gets zeros without a branch: a conditional load would make the compiler wait for it
// at the branch join, ahead of the row loads, and add a memory round trip to the kernel start.
typedef __attribute__((ext_vector_type(2))) int i32x2_t;

template <typename WT, typename XT>
struct XSlice {
    static constexpr int V = Elem<WT>::V;
    static constexpr int WORDS = V * (int)sizeof(XT) / 4;  // 2, 4 or 8
    float v[V];
    __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t r, int off) {
        uint32_t wd[WORDS];
        if (WORDS == 2) {
            const i32x2_t t = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
            wd[0] = (uint32_t)t[0];
            wd[1] = (uint32_t)t[1];
        } else {
#pragma unroll
            for (int q = 0; q < WORDS / 4; ++q) {
                const V16 t = bload16(r, off == kOOB ? kOOB : off + 16 * q);
#pragma unroll
                for (int e = 0; e < 4; ++e) wd[4 * q + e] = t.w[e];
            }
        }
#pragma unroll
        for (int e = 0; e < V; ++e) v[e] = xval(wd, e, (const XT*)nullptr);
    }
    template <int N>
    __device__ __forceinline__ static float xval(const uint32_t (&wd)[N], int e, const float*) {
        return __uint_as_float(wd[e]);
    }
    template <int N>
    __device__ __forceinline__ static float xval(const uint32_t (&wd)[N], int e, const bf16_t*) {
        return (e & 1) ? bf16hi(wd[e >> 1]) : bf16lo(wd[e >> 1]);
    }
    template <int N>
    __device__ __forceinline__ static float xval(const uint32_t (&wd)[N], int e, const f16_t*) {
        return f16_to_f32((e & 1) ? (wd[e >> 1] >> 16) : (wd[e >> 1] & 0xffffu));
    }
    // v = f: values already rounded to XT
    __device__ __forceinline__ void set(const float (&f)[V]) {
#pragma unroll
        for (int e = 0; e < V; ++e) v[e] = f[e];
    }
    __device__ __forceinline__ float dot(const V16& w, float acc) const {
        float f[V];
        Elem<WT>::unpack(w, f);
#pragma unroll
        for (int e = 0; e < V; ++e) acc = fmaf(f[e], v[e], acc);
        return acc;
    }
};

template <>
struct XSlice<bf16_t, bf16_t> {
    uint32_t v[4];
    __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t r, int off) {
        const V16 t = bload16(r, off);
#pragma unroll
        for (int q = 0; q < 4; ++q) v[q] = t.w[q];
    }
    // f: 8 values already rounded to bf16, packed back into pairs
    __device__ __forceinline__ void set(const float (&f)[8]) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
            v[q] = (__float_as_uint(f[2 * q]) >> 16) | (__float_as_uint(f[2 * q + 1]) & 0xffff0000u);
    }
    __device__ __forceinline__ float dot(const V16& w, float acc) const {
#pragma unroll
        for (int q = 0; q < 4; ++q)
            acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w.w[q]),
                                                  __builtin_bit_cast(bf16x2_t, v[q]), acc, false);
        return acc;
    }
};

typedef __attribute__((ext_vector_type(2))) _Float16 f16x2_t;

template <>
struct XSlice<f16_t, f16_t> {
    uint32_t v[4];
    __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t r, int off) {
        const V16 t = bload16(r, off);
#pragma unroll
        for (int q = 0; q < 4; ++q) v[q] = t.w[q];
    }
    __device__ __forceinline__ float dot(const V16& w, float acc) const {
#pragma unroll
        for (int q = 0; q < 4; ++q)
            acc = __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2_t, w.w[q]),
                                         __builtin_bit_cast(f16x2_t, v[q]), acc, false);
        return acc;
    }
};

// Residual RMSNorm prologue: V consecutive elements of a row of type T (float or bf16) as
// float32, through a buffer descriptor (kOOB: zeros, no access).
template <typename T, int V>
__device__ __forceinline__ void load_elems(__amdgpu_buffer_rsrc_t r, int off, float (&f)[V]) {
    if constexpr (sizeof(T) == 4) {
#pragma unroll
        for (int q = 0; q < V / 4; ++q) {
            const V16 t = bload16(r, off == kOOB ? kOOB : off + 16 * q);
#pragma unroll
            for (int e = 0; e < 4; ++e) f[4 * q + e] = __uint_as_float(t.w[e]);
        }
    } else if constexpr (V == 8) {
        const V16 t = bload16(r, off);
        Elem<bf16_t>::unpack(t, f);
    } else {
        const i32x2_t t = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
#pragma unroll
        for (int e = 0; e < 2; ++e) {
            f[2 * e] = bf16lo((uint32_t)t[e]);
            f[2 * e + 1] = bf16hi((uint32_t)t[e]);
        }
    }
}
// a float32 value rounded to the storage type T and widened back (bf16: round to nearest even)
template <typename T>
__device__ __forceinline__ float round_to(float f) {
    if constexpr (sizeof(T) == 4) return f;
    else return bf16_to_f32(f32_to_bf16_rne(f));
}
// V values (already rounded to T) stored as T at p
template <typename T, int V>
__device__ __forceinline__ void store_elems(T* p, const float (&f)[V]) {
    if constexpr (sizeof(T) == 4) {
#pragma unroll
        for (int q = 0; q < V / 4; ++q)
            st16(p + 4 * q, V16{{__float_as_uint(f[4 * q]), __float_as_uint(f[4 * q + 1]),
                                 __float_as_uint(f[4 * q + 2]), __float_as_uint(f[4 * q + 3])}});
    } else {
        uint32_t wd[V / 2];
#pragma unroll
        for (int q = 0; q < V / 2; ++q)
            wd[q] = (__float_as_uint(f[2 * q]) >> 16) | (__float_as_uint(f[2 * q + 1]) & 0xffff0000u);
        if constexpr (V == 8)
            st16(p, V16{{wd[0], wd[1], wd[2], wd[3]}});
        else
            *reinterpret_cast<uint2*>(p) = make_uint2(wd[0], wd[1]);
    }
}

// Row loads of the gather-GEMV; lane column group i of row j, for a wave-uniform slot id j and
// validity flag ok. A step reads each of its rows once, so the loads are non-temporal.
// BUF: buffer loads with 32-bit offsets (the compacted tensors must be smaller than 2 GiB); a
// row or column that must read nothing gets an offset past the end of the buffer, so the access
// reads no memory and returns zeros, without a branch. Otherwise guarded global loads.
template <typename WT, bool BUF, int NI>
struct RowLoader;

template <typename WT, int NI>
struct RowLoader<WT, true, NI> {
    __amdgpu_buffer_rsrc_t rg, rd;
    int rowg, rowd;    // bytes per row of gate_up_c and down_c
    int vcol[NI];      // lane column byte offset, or kOOB outside the row
    __device__ __forceinline__ RowLoader(const WT* gu, const WT* dc, int64_t L, int64_t d,
                                         const int64_t (&col)[NI], const bool (&cok)[NI]) {
        rg = make_rsrc(gu, L * 2 * d * (int64_t)sizeof(WT));
        rd = make_rsrc(dc, L * d * (int64_t)sizeof(WT));
        rowg = (int)(2 * d * (int64_t)sizeof(WT));
        rowd = (int)(d * (int64_t)sizeof(WT));
#pragma unroll
        for (int i = 0; i < NI; ++i) vcol[i] = cok[i] ? (int)(col[i] * (int64_t)sizeof(WT)) : kOOB;
    }
    // kOOB + a row offset (< 2^31) stays out of range without wrapping
    __device__ __forceinline__ void load_gu(bool ok, int32_t j, int i, V16& g, V16& u) const {
        const int og = ok ? vcol[i] + j * rowg : kOOB;
        g = bload16nt(rg, og);
        u = bload16nt(rg, og + rowd);
    }
    __device__ __forceinline__ void load_dn(bool ok, int32_t j, int i, V16& dn) const {
        dn = bload16nt(rd, ok ? vcol[i] + j * rowd : kOOB);
    }
};

template <typename WT, int NI>
struct RowLoader<WT, false, NI> {
    const WT* gu;
    const WT* dc;
    int64_t d;
    int64_t col[NI];
    bool cok[NI];
    __device__ __forceinline__ RowLoader(const WT* gu_, const WT* dc_, int64_t, int64_t d_,
                                         const int64_t (&col_)[NI], const bool (&cok_)[NI])
        : gu(gu_), dc(dc_), d(d_) {
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            col[i] = col_[i];
            cok[i] = cok_[i];
        }
    }
    __device__ __forceinline__ void load_gu(bool ok, int32_t j, int i, V16& g, V16& u) const {
        if (ok && cok[i]) {
            const WT* gp = gu + (int64_t)j * 2 * d + col[i];
            g = ld16(gp);
            u = ld16(gp + d);
        } else {
            g = V16{{0u, 0u, 0u, 0u}};
            u = g;
        }
    }
    __device__ __forceinline__ void load_dn(bool ok, int32_t j, int i, V16& dn) const {
        dn = (ok && cok[i]) ? ld16(dc + (int64_t)j * d + col[i]) : V16{{0u, 0u, 0u, 0u}};
    }
};

// f(std::integral_constant<int, n>) for a run-time n in [N, R]: code that must know a row
// count at compile time, reached through a chain of uniform compares
template <int N, int R, class F>
__device__ __forceinline__ void with_rows(int n, F& f) {
    if constexpr (N <= R) {
        if (n == N)
            f(std::integral_constant<int, N>());
        else
            with_rows<N + 1, R>(n, f);
    }
}

// floor(n * p / P) for 0 <= n, 0 <= p <= P: the first row of chunk p when n rows are dealt to
// P chunks. The host keeps nnz * P below 2^32 (decode_chunks), so 32-bit arithmetic is exact;
// the GPU has no integer divide instruction and a 64-bit emulation is several times longer.
__device__ __forceinline__ int64_t split(int64_t n, int p, int P) {
    return (int64_t)((uint32_t)n * (uint32_t)p / (uint32_t)P);
}

// RN: x is not read; the token's input is RMSNorm(xprev + yprev) (unit gain, eps), computed by
// every work-group of the token for its lanes' columns, and work-group 0 stores it to xout.
template <typename WT, typename XT, int NI, bool BUF, bool RN>
__global__ __launch_bounds__(kThreads) void sffn_rows(
    const XT* __restrict__ x, int64_t d, const int32_t* __restrict__ offsets,
    const int32_t* __restrict__ idx, int64_t nnz, const WT* __restrict__ gate_up_c,
    const WT* __restrict__ down_c, int64_t L, float* __restrict__ partials, int P,
    const XT* __restrict__ xprev, const float* __restrict__ yprev, float eps,
    XT* __restrict__ xout) {
    constexpr int V = Elem<WT>::V;
    constexpr int R = RowsPerBatch<XT, NI, RN>::value;
    constexpr int NVAL = 2 * R;
    constexpr int PER = kWave / NVAL;

    const int p = blockIdx.x;
    const int b = blockIdx.y;
    const int lane = threadIdx.x & (kWave - 1);
    const int w = threadIdx.x >> 6;

    int64_t col[NI];
    bool cok[NI];
    float acc[NI][V];
#pragma unroll
    for (int i = 0; i < NI; ++i) {
        col[i] = ((int64_t)(i * kWaves + w) * kWave + lane) * V;
        cok[i] = col[i] < d;
#pragma unroll
        for (int e = 0; e < V; ++e) acc[i][e] = 0.0f;
    }
    const RowLoader<WT, BUF, NI> ldr(gate_up_c, down_c, L, d, col, cok);

    // x first: vector loads complete in issue order, so the dot products of the first rows
    // wait only for x and their own rows
    XSlice<WT, XT> xs[NI];
    // RN: r = xprev + yprev for the lane's columns (zeros outside the row), then normalise()
    float rr[NI][RN ? V : 1];
    if constexpr (RN) {
        const __amdgpu_buffer_rsrc_t rxp =
            make_rsrc(xprev + (int64_t)b * d, d * (int64_t)sizeof(XT));
        const __amdgpu_buffer_rsrc_t ryp = make_rsrc(yprev + (int64_t)b * d, d * 4);
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            float xf[V], yf[V];
            load_elems<XT, V>(rxp, cok[i] ? (int)(col[i] * (int64_t)sizeof(XT)) : kOOB, xf);
            load_elems<float, V>(ryp, cok[i] ? (int)(col[i] * 4) : kOOB, yf);
#pragma unroll
            for (int e = 0; e < V; ++e) rr[i][e] = xf[e] + yf[e];
        }
    } else {
        const __amdgpu_buffer_rsrc_t rx = make_rsrc(x + (int64_t)b * d, d * (int64_t)sizeof(XT));
#pragma unroll
        for (int i = 0; i < NI; ++i)
            xs[i].load(rx, cok[i] ? (int)(col[i] * (int64_t)sizeof(XT)) : kOOB);
    }
    // RN: x = r / sqrt(mean(r^2) + eps), rounded to XT. The sum of squares is reduced over the
    // work-group in a fixed order (lane tree, then the waves in order), the same in every
    // work-group of the token. Called once, after the first batch's row loads are issued, so
    // its wait for xprev / yprev and its barrier overlap the row loads.
    bool pending = RN;
    auto normalise = [&]() {
        if constexpr (RN) {
            float ss = 0.0f;
#pragma unroll
            for (int i = 0; i < NI; ++i)
#pragma unroll
                for (int e = 0; e < V; ++e) ss = fmaf(rr[i][e], rr[i][e], ss);
            ss = wave_sum(ss);
            __shared__ float nred[kWaves];
            if (lane == 0) nred[w] = ss;
            __syncthreads();
            float tot = 0.0f;
#pragma unroll
            for (int q = 0; q < kWaves; ++q) tot += nred[q];
            const float scale = 1.0f / sqrtf(tot / (float)d + eps);
#pragma unroll
            for (int i = 0; i < NI; ++i) {
#pragma unroll
                for (int e = 0; e < V; ++e) rr[i][e] = round_to<XT>(rr[i][e] * scale);
                xs[i].set(rr[i]);
                // the token's first work-group keeps x for the next layer's residual
                if (p == 0 && cok[i]) store_elems<XT, V>(xout + (int64_t)b * d + col[i], rr[i]);
            }
            pending = false;
        }
    };

    // Slot ids of batch [rb, rb + nr): a batch that lies inside idx is read with unconditional
    // scalar loads, which the compiler merges into one wide load (separate conditional loads
    // would each wait for the previous one). Rows past nr get -1.
    auto fetch_ids = [&](int64_t rb, int nr, int32_t (&sl)[R]) {
        if (rb + R <= nnz) {
#pragma unroll
            for (int r = 0; r < R; ++r) sl[r] = idx[rb + r];
        } else {
#pragma unroll
            for (int r = 0; r < R; ++r) sl[r] = rb + r < nnz ? idx[rb + r] : -1;
        }
#pragma unroll
        for (int r = 0; r < R; ++r) sl[r] = r < nr ? sl[r] : -1;
    };
    // A batch of N rows (N <= R, a constant in each instance, see with_rows), start to end:
    // every gate/up load, then every down load, the gate/up dot products, their exchange
    // across the waves, SiLU * up, and the down-row FMAs. The memory system returns the
    // gate/up rows first, so the dot products and the exchange finish while the down rows are
    // still streaming in. Ids are wave-uniform, so the row bases stay in scalar registers.
    // Each of the N rows issues its loads whatever its id (an invalid id loads nothing through
    // an out-of-range offset), and rows past N issue none: the number of loads still in
    // flight at each use is then known when the kernel is compiled, and each use waits for
    // its own row only. (Loads behind a run-time condition make the compiler wait for every
    // load, down rows included, before the first dot product; and out-of-range loads for the
    // rows past N would still take issue slots in the load pipeline, the bottleneck while a
    // batch is being issued.)
    // okr[r]: row r exists and has a valid slot id (wave-uniform)
    V16 gv[R][NI], uv[R][NI], dv[R][NI];
    bool okr[R];
    int32_t sl[R];
    __shared__ float red[2][NVAL][kWaves];
    int buf = 0;
    auto batch = [&](auto ncst) {
        constexpr int N = decltype(ncst)::value;
#pragma unroll
        for (int r = 0; r < R; ++r) okr[r] = r < N && sl[r] >= 0 && sl[r] < L;
#pragma unroll
        for (int r = 0; r < N; ++r)
#pragma unroll
            for (int i = 0; i < NI; ++i) ldr.load_gu(okr[r], sl[r], i, gv[r][i], uv[r][i]);
#pragma unroll
        for (int r = 0; r < N; ++r)
#pragma unroll
            for (int i = 0; i < NI; ++i) ldr.load_dn(okr[r], sl[r], i, dv[r][i]);
        if (pending) normalise();  // uniform; RN only
        // all N rows, without a branch (a load used only inside a branch is moved into it,
        // behind the other loads); a row with an invalid id gives a value nobody uses
        float vals[NVAL];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            float g = 0.0f, u = 0.0f;
            if (r < N) {
#pragma unroll
                for (int i = 0; i < NI; ++i) {
                    g = xs[i].dot(gv[r][i], g);
                    u = xs[i].dot(uv[r][i], u);
                }
            }
            vals[r] = g;
            vals[R + r] = u;
        }
        // lane l: this wave's total of value l / PER; then the 8 waves meet in LDS
        const float tot = wave_transpose_sum<NVAL>(vals, lane);
        if ((lane % PER) == 0) red[buf][lane / PER][w] = tot;
        __syncthreads();
        // lane r < R holds g_r, lane R + r holds u_r (summed over waves in a fixed order)
        float t = 0.0f;
        if (lane < NVAL) {
#pragma unroll
            for (int q = 0; q < kWaves; ++q) t += red[buf][lane][q];
        }
        const float uu = __shfl_down(t, R, kWave);
        const float hv = silu_f32(t) * uu;  // valid in lanes 0 .. R-1
        // h_r * down_r for the N rows, again without a branch: a row with an invalid id has
        // h = 0 and a zero down row, and adds exactly nothing. Every load of the batch is
        // consumed here, so none is in flight where the instances of this code meet.
#pragma unroll
        for (int r = 0; r < N; ++r) {
            float h = __builtin_bit_cast(
                float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, hv), r));
            h = okr[r] ? h : 0.0f;
#pragma unroll
            for (int i = 0; i < NI; ++i) {
                float df[V];
                Elem<WT>::unpack(dv[r][i], df);
#pragma unroll
                for (int e = 0; e < V; ++e) acc[i][e] = fmaf(h, df[e], acc[i][e]);
            }
        }
    };

    // The first batch's slot ids are fetched together with the token's offsets, from the
    // range this work-group gets when the B tokens hold nnz / B rows each from index 0 (a
    // top-k output, or one token with offsets {0, nnz}): the row loads then wait for one
    // memory round trip instead of two (offsets, then ids). The guess is checked before the
    // ids are used; a wrong guess fetches them again and costs only that round trip.
    const int64_t per = split(nnz, 1, (int)gridDim.y);
    const int64_t g0 = (int64_t)b * per + split(per, p, P);
    fetch_ids(g0, R, sl);

    int64_t lo = offsets[b], hi = offsets[b + 1];
    lo = lo < 0 ? 0 : (lo > nnz ? nnz : lo);
    hi = hi < lo ? lo : (hi > nnz ? nnz : hi);
    const int64_t n = hi - lo;
    int64_t rb = lo + split(n, p, P);
    const int64_t r1 = lo + split(n, p + 1, P);
    int nr = (int)((r1 - rb) < R ? (r1 - rb) : R);
    if (rb == g0) {
#pragma unroll
        for (int r = 0; r < R; ++r) sl[r] = r < nr ? sl[r] : -1;
    } else {
        fetch_ids(rb, nr, sl);
    }

    while (nr > 0) {
        with_rows<1, R>(nr, batch);
        buf ^= 1;
        rb += R;
        if (rb >= r1) break;
        nr = (int)((r1 - rb) < R ? (r1 - rb) : R);
        fetch_ids(rb, nr, sl);
    }

    if constexpr (RN) {
        if (pending) normalise();  // a work-group without rows
    }

    const int64_t nch = part_chunks(d);
#pragma unroll
    for (int i = 0; i < NI; ++i) {
        if (cok[i]) {
            // V <= 16 consecutive columns starting at a multiple of V stay inside one chunk
            float* out = partials + part_off(b, p, col[i], P, nch);
#pragma unroll
            for (int e = 0; e < V; e += 4) {
                V16 o;
                o.w[0] = __float_as_uint(acc[i][e]);
                o.w[1] = __float_as_uint(acc[i][e + 1]);
                o.w[2] = __float_as_uint(acc[i][e + 2]);
                o.w[3] = __float_as_uint(acc[i][e + 3]);
                st16_nt(out + e, o);
            }
        }
    }
}

// y[b][c] = sum_{p = 0..P-1} of the partials of column c, in a fixed order. One (token, chunk)
// pair per WPP waves: its P x kChunk floats are contiguous; thread t adds the float4 groups
// t, t + 64 WPP, ... (all of column group t % kG, kG = kChunk / 4) in ascending order, then a
// fixed shuffle tree over the lanes of one group and, for WPP = 4, a fixed-order sum of the
// waves through LDS.
constexpr int kG = kChunk / 4;  // float4 groups of a chunk
template <int WPP>
__global__ __launch_bounds__(256) void reduce_chunks(const float* __restrict__ partials, int P,
                                                     int64_t pairs, int64_t nch, int64_t d,
                                                     float* __restrict__ y) {
    constexpr int NT = WPP * kWave;
    const int lane = threadIdx.x & (kWave - 1);
    const int w = threadIdx.x >> 6;
    const int64_t pair = (int64_t)blockIdx.x * (4 / WPP) + w / WPP;
    if (pair >= pairs) return;  // uniform per work-group when WPP = 4
    const int t = (w % WPP) * kWave + lane;
    const float4* base = reinterpret_cast<const float4*>(partials + pair * (int64_t)P * kChunk);
    const int n4 = P * kG;
    float s[4] = {0.f, 0.f, 0.f, 0.f};
    int i = t;
    for (; i + 3 * NT < n4; i += 4 * NT) {
        float4 v[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) v[q] = base[i + q * NT];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            s[0] += v[q].x;
            s[1] += v[q].y;
            s[2] += v[q].z;
            s[3] += v[q].w;
        }
    }
    for (; i < n4; i += NT) {
        const float4 v = base[i];
        s[0] += v.x;
        s[1] += v.y;
        s[2] += v.z;
        s[3] += v.w;
    }
#pragma unroll
    for (int m = kG; m < kWave; m <<= 1)
#pragma unroll
        for (int e = 0; e < 4; ++e) s[e] += __shfl_xor(s[e], m, kWave);
    const int64_t b = pair / nch;
    const int64_t c0 = (pair % nch) * kChunk;
    if (WPP == 1) {
        const int64_t c = c0 + 4 * lane;
        if (lane < kG && c < d)  // d is a multiple of 4: the float4 is all in range
            *reinterpret_cast<float4*>(y + b * d + c) = make_float4(s[0], s[1], s[2], s[3]);
    } else {
        __shared__ float red[WPP][kChunk];
        if (lane < kG) {
#pragma unroll
            for (int e = 0; e < 4; ++e) red[w][lane * 4 + e] = s[e];
        }
        __syncthreads();
        if (t < kChunk && c0 + t < d) {
            float a = 0.f;
#pragma unroll
            for (int q = 0; q < WPP; ++q) a += red[q][t];
            y[b * d + c0 + t] = a;
        }
    }
}

// The same sum for few partials (P < 16): thread i owns float4 group i % kG of chunk i / kG
// (over tokens and chunks) and adds its P float4 values in ascending p.
__global__ __launch_bounds__(256) void reduce_few(const float* __restrict__ partials, int P,
                                                  int64_t n4, int64_t nch, int64_t d,
                                                  float* __restrict__ y) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n4) return;
    const int64_t pair = i / kG;  // (token, chunk)
    const int q = (int)(i % kG);
    const float4* base = reinterpret_cast<const float4*>(partials + pair * (int64_t)P * kChunk) + q;
    float4 s = base[0];
    for (int p = 1; p < P; ++p) {
        const float4 v = base[p * kG];
        s.x += v.x;
        s.y += v.y;
        s.z += v.z;
        s.w += v.w;
    }
    const int64_t b = pair / nch;
    const int64_t c = (pair % nch) * kChunk + 4 * q;
    if (c < d) *reinterpret_cast<float4*>(y + b * d + c) = s;  // d % 4 == 0
}

// ev0/ev1 (optional): stamped from the kernel's own dispatch (hipExtLaunchKernelGGL), so
// their elapsed time is the kernel's device time without queueing or marker overheads.
template <typename WT, typename XT, bool BUF>
hipError_t launch_rows_t(const void* x, int64_t B, int64_t d, const int32_t* offsets,
                         const int32_t* idx, int64_t nnz, const void* gu, const void* dc,
                         int64_t L, float* partials, int P, hipStream_t s, hipEvent_t ev0,
                         hipEvent_t ev1, const ResNormIn* rn) {
    constexpr int V = Elem<WT>::V;
    const int64_t span = (int64_t)kThreads * V;
    const int ni = (int)((d + span - 1) / span);
    dim3 grid((unsigned)P, (unsigned)B);
    dim3 block(kThreads);
    const XT* xx = static_cast<const XT*>(x);
    const WT* g = static_cast<const WT*>(gu);
    const WT* dn = static_cast<const WT*>(dc);
    // the prologue stores x as float32 or bf16 only
    constexpr bool kRN = !std::is_same<XT, f16_t>::value;
    if (rn && !kRN) return hipErrorInvalidValue;
    const XT* xp = rn ? static_cast<const XT*>(rn->x_prev) : nullptr;
    const float* yp = rn ? rn->y_prev : nullptr;
    const float eps = rn ? rn->eps : 0.0f;
    XT* xo = rn ? static_cast<XT*>(rn->x_out) : nullptr;
#define SI_ROWS_CASE(N)                                                                        \
    case N:                                                                                    \
        if (rn) {                                                                              \
            if constexpr (kRN)                                                                 \
                hipExtLaunchKernelGGL((sffn_rows<WT, XT, N, BUF, kRN>), grid, block, 0, s, ev0, \
                                      ev1, 0, xx, d, offsets, idx, nnz, g, dn, L, partials, P, \
                                      xp, yp, eps, xo);                                        \
        } else                                                                                 \
            hipExtLaunchKernelGGL((sffn_rows<WT, XT, N, BUF, false>), grid, block, 0, s, ev0,  \
                                  ev1, 0, xx, d, offsets, idx, nnz, g, dn, L, partials, P, xp, \
                                  yp, eps, xo);                                                \
        break;
    switch (ni) {
        SI_ROWS_CASE(1)
        SI_ROWS_CASE(2)
        SI_ROWS_CASE(3)
        SI_ROWS_CASE(4)
        default:
            return hipErrorInvalidValue;
    }
#undef SI_ROWS_CASE
    return hipGetLastError();
}

}  // namespace

int decode_supported(int xdt, int wdt, int64_t d) {
    // x is float32 or has the weights' type; half-precision weights pair with half or f32 x,
    // bf16 weights with bf16 or f32 x, f32 weights with f32 or bf16 x
    if (wdt == 2 && xdt != 2 && xdt != 0) return 1;
    if (xdt == 2 && wdt != 2) return 1;
    const int V = wdt == 0 ? 4 : 8;
    if (d <= 0 || d % V != 0) return 1;
    if (xdt != 0 && d % 8 != 0) return 1;
    if (d > (int64_t)4 * kThreads * V) return 1;
    return 0;
}

int decode_chunks(int64_t B, int64_t nnz, int num_cu) {
    if (B <= 0) return 1;
    const int64_t per_tok = (nnz + B - 1) / B;
    int64_t target = num_cu / B;
    if (target < 1) target = 1;
    int64_t P = per_tok < target ? per_tok : target;
    // the kernel's row split uses 32-bit products: nnz * P < 2^32 (nnz itself is below 2^31)
    const int64_t cap = nnz > 0 ? (int64_t)0xffffffff / nnz : P;
    if (P > cap) P = cap;
    if (P < 1) P = 1;
    return (int)P;
}

hipError_t launch_decode(const void* x, int xdt, int64_t B, int64_t d, const int32_t* offsets,
                         const int32_t* idx, int64_t nnz, const void* gate_up_c,
                         const void* down_c, int64_t L, int wdt, float* partials, int P,
                         float* y, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1,
                         const ResNormIn* rn) {
    if (B == 0) return hipSuccess;
    hipError_t e;
    // buffer loads take 32-bit byte offsets: both compacted tensors must stay below 2 GiB
    const int64_t es = wdt == 0 ? 4 : 2;
    const bool buf = L * 2 * d * es < ((int64_t)1 << 31);
#define SI_DEC(WT, XT)                                                                        \
    (buf ? launch_rows_t<WT, XT, true>(x, B, d, offsets, idx, nnz, gate_up_c, down_c, L,      \
                                       partials, P, s, ev0, ev1, rn)                          \
         : launch_rows_t<WT, XT, false>(x, B, d, offsets, idx, nnz, gate_up_c, down_c, L,     \
                                        partials, P, s, ev0, ev1, rn))
    if (wdt == 1 && xdt == 1)
        e = SI_DEC(bf16_t, bf16_t);
    else if (wdt == 1 && xdt == 0)
        e = SI_DEC(bf16_t, float);
    else if (wdt == 0 && xdt == 1)
        e = SI_DEC(float, bf16_t);
    else if (wdt == 2 && xdt == 2)
        e = SI_DEC(f16_t, f16_t);
    else if (wdt == 2 && xdt == 0)
        e = SI_DEC(f16_t, float);
    else if (wdt == 0 && xdt == 0)
        e = SI_DEC(float, float);
    else
        return hipErrorInvalidValue;  // excluded by decode_supported
#undef SI_DEC
    if (e != hipSuccess) return e;
    return launch_reduce_partials(partials, P, B, d, y, s);
}

hipError_t launch_reduce_partials(const float* partials, int P, int64_t B, int64_t d, float* y,
                                  hipStream_t s) {
    if (B == 0) return hipSuccess;
    const int64_t nch = part_chunks(d);
    const int64_t pairs = B * nch;
    if (P < 16) {  // one thread per float4 of y: a wave reads 16 chunks' partials contiguously
        const int64_t n4 = B * nch * kG;
        hipLaunchKernelGGL(reduce_few, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, s,
                           partials, P, n4, nch, d, y);
    } else if (P >= 64) {  // four waves per (token, chunk) pair
        hipLaunchKernelGGL(reduce_chunks<4>, dim3((unsigned)pairs), dim3(256), 0, s, partials, P,
                           pairs, nch, d, y);
    } else {        // one wave per pair, four pairs per work-group
        hipLaunchKernelGGL(reduce_chunks<1>, dim3((unsigned)((pairs + 3) / 4)), dim3(256), 0, s,
                           partials, P, pairs, nch, d, y);
    }
    return hipGetLastError();
}

size_t decode_workspace(int64_t B, int64_t nnz, int64_t d, int num_cu) {
    return (size_t)B * decode_chunks(B, nnz, num_cu) * part_chunks(d) * kChunk * sizeof(float);
}

}  // namespace si
