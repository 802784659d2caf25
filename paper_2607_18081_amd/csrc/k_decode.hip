// Per-token path of the selective SwiGLU FFN (Selective Computation section).
//
// For one token with active slots A and compacted weights gate_up_c [L][2][d], down_c [L][d]:
//     h_j = SiLU(gate_j . x) * (up_j . x),   y = sum_{j in A} h_j * down_j.
//
// Kernel 1 (sffn_rows): work-group (p, b) takes chunk p of token b's active list. Its 8 waves
// split the d columns: wave w, lane l own the 16-byte column groups ((i*8 + w)*64 + l), so a
// row is read as one fully coalesced sweep of the work-group. For a batch of up to R rows the
// work-group issues every gate, up and down load of the batch at once (the down rows do not
// depend on h, so they stream in while the dot products complete), reduces each row's two dot
// products across the wave with a transposing shuffle reduction and across the 8 waves through
// LDS, applies SiLU*up, and accumulates h_j * down_j into per-lane float32 registers. The
// work-group's partial sum over its rows is written as one float32 row of the workspace.
//
// Kernel 2 (reduce_partials) adds the P partial rows of each token in a fixed order, so the
// result is deterministic and no global atomics are used.
#include <hip/hip_ext.h>

#include "common.h"
#include "launch.h"

namespace si {

namespace {

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * kWave;

template <int NI>
struct RowsPerBatch {
    static constexpr int value = NI == 1 ? 16 : NI == 2 ? 8 : NI == 3 ? 4 : 2;
};

typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;

// The token's x restricted to one lane's 16-byte column group, in the form its dot products
// use: packed bf16 pairs when both x and the weights are bf16 (v_dot2_f32_bf16), else float.
template <typename WT, typename XT>
struct XSlice {
    static constexpr int V = Elem<WT>::V;
    float v[V];
    __device__ __forceinline__ void load(const XT* p, bool ok) {
#pragma unroll
        for (int e = 0; e < V; ++e) v[e] = ok ? xval(p + e) : 0.0f;
    }
    __device__ __forceinline__ static float xval(const float* p) { return *p; }
    __device__ __forceinline__ static float xval(const bf16_t* p) { return bf16_to_f32(*p); }
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
    __device__ __forceinline__ void load(const bf16_t* p, bool ok) {
        const V16 t = ok ? ld16(p) : V16{{0u, 0u, 0u, 0u}};
#pragma unroll
        for (int q = 0; q < 4; ++q) v[q] = t.w[q];
    }
    __device__ __forceinline__ float dot(const V16& w, float acc) const {
#pragma unroll
        for (int q = 0; q < 4; ++q)
            acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w.w[q]),
                                                  __builtin_bit_cast(bf16x2_t, v[q]), acc, false);
        return acc;
    }
};

// Row loads of the gather-GEMV. BUF: buffer loads with range-checked 32-bit offsets (no
// branches; the compacted tensors must be smaller than 2 GiB); else guarded global loads.
template <typename WT, bool BUF>
struct RowLoader;

template <typename WT>
struct RowLoader<WT, true> {
    __amdgpu_buffer_rsrc_t rg, rd;
    int64_t d;
    __device__ __forceinline__ RowLoader(const WT* gu, const WT* dc, int64_t L, int64_t d_)
        : d(d_) {
        rg = make_rsrc(gu, L * 2 * d_ * (int64_t)sizeof(WT));
        rd = make_rsrc(dc, L * d_ * (int64_t)sizeof(WT));
    }
    __device__ __forceinline__ void load(bool ok, int32_t j, int64_t col, V16& g, V16& u,
                                         V16& dn) const {
        const int og = ok ? (int)(((int64_t)j * 2 * d + col) * sizeof(WT)) : kOOB;
        const int od = ok ? (int)(((int64_t)j * d + col) * sizeof(WT)) : kOOB;
        g = bload16(rg, og);
        u = bload16(rg, ok ? og + (int)(d * sizeof(WT)) : kOOB);
        dn = bload16(rd, od);
    }
};

template <typename WT>
struct RowLoader<WT, false> {
    const WT* gu;
    const WT* dc;
    int64_t d;
    __device__ __forceinline__ RowLoader(const WT* gu_, const WT* dc_, int64_t, int64_t d_)
        : gu(gu_), dc(dc_), d(d_) {}
    __device__ __forceinline__ void load(bool ok, int32_t j, int64_t col, V16& g, V16& u,
                                         V16& dn) const {
        const V16 z = V16{{0u, 0u, 0u, 0u}};
        if (ok) {
            const WT* gp = gu + (int64_t)j * 2 * d + col;
            g = ld16(gp);
            u = ld16(gp + d);
            dn = ld16(dc + (int64_t)j * d + col);
        } else {
            g = z;
            u = z;
            dn = z;
        }
    }
};

template <typename WT, typename XT, int NI, bool BUF>
__global__ __launch_bounds__(kThreads) void sffn_rows(
    const XT* __restrict__ x, int64_t d, const int32_t* __restrict__ offsets,
    const int32_t* __restrict__ idx, int64_t nnz, const WT* __restrict__ gate_up_c,
    const WT* __restrict__ down_c, int64_t L, float* __restrict__ partials, int P) {
    constexpr int V = Elem<WT>::V;
    constexpr int R = RowsPerBatch<NI>::value;
    constexpr int NVAL = 2 * R;
    constexpr int PER = kWave / NVAL;

    const int p = blockIdx.x;
    const int b = blockIdx.y;
    const int lane = threadIdx.x & (kWave - 1);
    const int w = threadIdx.x >> 6;

    int64_t lo = offsets[b], hi = offsets[b + 1];
    lo = lo < 0 ? 0 : (lo > nnz ? nnz : lo);
    hi = hi < lo ? lo : (hi > nnz ? nnz : hi);
    const int64_t n = hi - lo;
    const int64_t r0 = lo + (n * p) / P;
    const int64_t r1 = lo + (n * (p + 1)) / P;

    int64_t col[NI];
    bool cok[NI];
    XSlice<WT, XT> xs[NI];
    float acc[NI][V];
    const XT* xb = x + (int64_t)b * d;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
        col[i] = ((int64_t)(i * kWaves + w) * kWave + lane) * V;
        cok[i] = col[i] < d;
        xs[i].load(xb + (cok[i] ? col[i] : 0), cok[i]);
#pragma unroll
        for (int e = 0; e < V; ++e) acc[i][e] = 0.0f;
    }
    const RowLoader<WT, BUF> ldr(gate_up_c, down_c, L, d);

    __shared__ float red[2][NVAL][kWaves];
    int buf = 0;
    for (int64_t rb = r0; rb < r1; rb += R) {
        const int nr = (int)((r1 - rb) < R ? (r1 - rb) : R);
        V16 gv[R][NI], uv[R][NI], dv[R][NI];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            // wave-uniform slot id: the row base stays in scalar registers
            const int32_t s = __builtin_amdgcn_readfirstlane(r < nr ? idx[rb + r] : -1);
            const bool ok = (s >= 0) && (s < L);
#pragma unroll
            for (int i = 0; i < NI; ++i) ldr.load(ok && cok[i], s, col[i], gv[r][i], uv[r][i], dv[r][i]);
        }
        float vals[NVAL];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            float g = 0.0f, u = 0.0f;
#pragma unroll
            for (int i = 0; i < NI; ++i) {
                g = xs[i].dot(gv[r][i], g);
                u = xs[i].dot(uv[r][i], u);
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
#pragma unroll
        for (int r = 0; r < R; ++r) {
            if (r < nr) {
                const float h = __builtin_bit_cast(
                    float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, hv), r));
#pragma unroll
                for (int i = 0; i < NI; ++i) {
                    float df[V];
                    Elem<WT>::unpack(dv[r][i], df);
#pragma unroll
                    for (int e = 0; e < V; ++e) acc[i][e] = fmaf(h, df[e], acc[i][e]);
                }
            }
        }
        buf ^= 1;
    }

    float* out = partials + ((int64_t)b * P + p) * d;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
        if (cok[i]) {
#pragma unroll
            for (int e = 0; e < V; e += 4) {
                V16 o;
                o.w[0] = __float_as_uint(acc[i][e]);
                o.w[1] = __float_as_uint(acc[i][e + 1]);
                o.w[2] = __float_as_uint(acc[i][e + 2]);
                o.w[3] = __float_as_uint(acc[i][e + 3]);
                st16(out + col[i] + e, o);
            }
        }
    }
}

// y[b][c] = sum_{p = 0..P-1} partials[b][p][c] in a fixed order. One wave per 4 columns (a
// float4 group): lane l adds p = l, l + 64, ... in order, then a fixed transposing shuffle tree
// leaves column c + l/16 in lanes 16*(l/16). No LDS, no barrier.
__global__ __launch_bounds__(256) void reduce_partials(const float* __restrict__ partials, int P,
                                                       int64_t d, float* __restrict__ y) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t c = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * 4;
    const int b = blockIdx.y;
    if (c >= d) return;
    const float* base = partials + (int64_t)b * P * d + c;
    float4 v[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int pp = lane + kWave * q;
        v[q] = pp < P ? *reinterpret_cast<const float4*>(base + (int64_t)pp * d)
                      : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    float s[4] = {v[0].x, v[0].y, v[0].z, v[0].w};
#pragma unroll
    for (int q = 1; q < 4; ++q) {
        s[0] += v[q].x;
        s[1] += v[q].y;
        s[2] += v[q].z;
        s[3] += v[q].w;
    }
    for (int pp = lane + 4 * kWave; pp < P; pp += kWave) {
        const float4 t = *reinterpret_cast<const float4*>(base + (int64_t)pp * d);
        s[0] += t.x;
        s[1] += t.y;
        s[2] += t.z;
        s[3] += t.w;
    }
    const float tot = wave_transpose_sum<4>(s, lane);
    if ((lane & 15) == 0) y[(int64_t)b * d + c + (lane >> 4)] = tot;
}

// ev0/ev1 (optional): stamped from the kernel's own dispatch (hipExtLaunchKernelGGL), so
// their elapsed time is the kernel's device time without queueing or marker overheads.
template <typename WT, typename XT, bool BUF>
hipError_t launch_rows_t(const void* x, int64_t B, int64_t d, const int32_t* offsets,
                         const int32_t* idx, int64_t nnz, const void* gu, const void* dc,
                         int64_t L, float* partials, int P, hipStream_t s, hipEvent_t ev0,
                         hipEvent_t ev1) {
    constexpr int V = Elem<WT>::V;
    const int64_t span = (int64_t)kThreads * V;
    const int ni = (int)((d + span - 1) / span);
    dim3 grid((unsigned)P, (unsigned)B);
    dim3 block(kThreads);
    const XT* xx = static_cast<const XT*>(x);
    const WT* g = static_cast<const WT*>(gu);
    const WT* dn = static_cast<const WT*>(dc);
#define SI_ROWS_CASE(N)                                                                        \
    case N:                                                                                    \
        hipExtLaunchKernelGGL((sffn_rows<WT, XT, N, BUF>), grid, block, 0, s, ev0, ev1, 0, xx, d, \
                              offsets, idx, nnz, g, dn, L, partials, P);                       \
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
    const int V = wdt == 1 ? 8 : 4;
    if (d <= 0 || d % V != 0) return 1;
    if (xdt == 1 && d % 8 != 0) return 1;
    if (d > (int64_t)4 * kThreads * V) return 1;
    return 0;
}

int decode_chunks(int64_t B, int64_t nnz, int num_cu) {
    if (B <= 0) return 1;
    const int64_t per_tok = (nnz + B - 1) / B;
    int64_t target = num_cu / B;
    if (target < 1) target = 1;
    int64_t P = per_tok < target ? per_tok : target;
    if (P < 1) P = 1;
    return (int)P;
}

hipError_t launch_decode(const void* x, int xdt, int64_t B, int64_t d, const int32_t* offsets,
                         const int32_t* idx, int64_t nnz, const void* gate_up_c,
                         const void* down_c, int64_t L, int wdt, float* partials, int P,
                         float* y, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
    if (B == 0) return hipSuccess;
    hipError_t e;
    // buffer loads take 32-bit byte offsets: both compacted tensors must stay below 2 GiB
    const int64_t es = wdt == 1 ? 2 : 4;
    const bool buf = L * 2 * d * es < ((int64_t)1 << 31);
#define SI_DEC(WT, XT)                                                                        \
    (buf ? launch_rows_t<WT, XT, true>(x, B, d, offsets, idx, nnz, gate_up_c, down_c, L,      \
                                       partials, P, s, ev0, ev1)                              \
         : launch_rows_t<WT, XT, false>(x, B, d, offsets, idx, nnz, gate_up_c, down_c, L,     \
                                        partials, P, s, ev0, ev1))
    if (wdt == 1 && xdt == 1)
        e = SI_DEC(bf16_t, bf16_t);
    else if (wdt == 1 && xdt == 0)
        e = SI_DEC(bf16_t, float);
    else if (wdt == 0 && xdt == 1)
        e = SI_DEC(float, bf16_t);
    else
        e = SI_DEC(float, float);
#undef SI_DEC
    if (e != hipSuccess) return e;
    return launch_reduce_partials(partials, P, B, d, y, s);
}

hipError_t launch_reduce_partials(const float* partials, int P, int64_t B, int64_t d, float* y,
                                  hipStream_t s) {
    if (B == 0) return hipSuccess;
    // one wave per float4 group, four waves per work-group
    dim3 grid((unsigned)((d + 15) / 16), (unsigned)B);
    hipLaunchKernelGGL(reduce_partials, grid, dim3(256), 0, s, partials, P, d, y);
    return hipGetLastError();
}

}  // namespace si
