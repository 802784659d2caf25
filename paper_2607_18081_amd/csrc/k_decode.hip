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
#include "common.h"
#include "launch.h"

namespace si {

namespace {

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * kWave;

template <int NI>
struct RowsPerBatch {
    static constexpr int value = NI == 1 ? 8 : NI == 2 ? 4 : 2;
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

template <typename WT, typename XT, int NI>
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

    __shared__ float red[2][NVAL][kWaves];
    int buf = 0;
    const int64_t two_d = 2 * d;

    for (int64_t rb = r0; rb < r1; rb += R) {
        const int nr = (int)((r1 - rb) < R ? (r1 - rb) : R);
        int32_t j[R];
        bool ok[R];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int32_t s = r < nr ? idx[rb + r] : -1;
            ok[r] = (s >= 0) && (s < L);
            j[r] = ok[r] ? s : 0;
        }
        V16 gv[R][NI], uv[R][NI], dv[R][NI];
#pragma unroll
        for (int r = 0; r < R; ++r) {
#pragma unroll
            for (int i = 0; i < NI; ++i) {
                if (ok[r] && cok[i]) {
                    const WT* gp = gate_up_c + (int64_t)j[r] * two_d + col[i];
                    gv[r][i] = ld16(gp);
                    uv[r][i] = ld16(gp + d);
                    dv[r][i] = ld16(down_c + (int64_t)j[r] * d + col[i]);
                } else {
                    gv[r][i] = V16{{0u, 0u, 0u, 0u}};
                    uv[r][i] = V16{{0u, 0u, 0u, 0u}};
                    dv[r][i] = V16{{0u, 0u, 0u, 0u}};
                }
            }
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
        const float tot = wave_transpose_sum<NVAL>(vals, lane);
        if ((lane % PER) == 0) red[buf][lane / PER][w] = tot;
        __syncthreads();
#pragma unroll
        for (int r = 0; r < R; ++r) {
            if (r < nr) {
                float g = 0.0f, u = 0.0f;
#pragma unroll
                for (int q = 0; q < kWaves; ++q) {
                    g += red[buf][r][q];
                    u += red[buf][R + r][q];
                }
                const float h = silu_f32(g) * u;
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

// y[b][c] = sum_{p = 0..P-1} partials[b][p][c], fixed order. Work-group: 32 columns (8 float4
// groups) x 32 lanes over p; lane (pg, cg) sums p = pg, pg + 32, ...; then a fixed LDS tree.
__global__ __launch_bounds__(256) void reduce_partials(const float* __restrict__ partials, int P,
                                                       int64_t d, float* __restrict__ y) {
    const int cg = threadIdx.x & 7;
    const int pg = threadIdx.x >> 3;
    const int b = blockIdx.y;
    const int64_t c = (int64_t)blockIdx.x * 32 + cg * 4;
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    if (c < d) {
        const float* base = partials + (int64_t)b * P * d + c;
        for (int p = pg; p < P; p += 32) {
            const float4 v = *reinterpret_cast<const float4*>(base + (int64_t)p * d);
            s.x += v.x;
            s.y += v.y;
            s.z += v.z;
            s.w += v.w;
        }
    }
    __shared__ float4 sh[32][8];
    sh[pg][cg] = s;
    __syncthreads();
#pragma unroll
    for (int st = 16; st >= 1; st >>= 1) {
        if (pg < st) {
            float4 a = sh[pg][cg];
            const float4 o = sh[pg + st][cg];
            a.x += o.x;
            a.y += o.y;
            a.z += o.z;
            a.w += o.w;
            sh[pg][cg] = a;
        }
        __syncthreads();
    }
    if (pg == 0 && c < d) *reinterpret_cast<float4*>(y + (int64_t)b * d + c) = sh[0][cg];
}

template <typename WT, typename XT>
hipError_t launch_rows_t(const void* x, int64_t B, int64_t d, const int32_t* offsets,
                         const int32_t* idx, int64_t nnz, const void* gu, const void* dc,
                         int64_t L, float* partials, int P, hipStream_t s) {
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
        hipLaunchKernelGGL((sffn_rows<WT, XT, N>), grid, block, 0, s, xx, d, offsets, idx, nnz, \
                           g, dn, L, partials, P);                                             \
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
                         float* y, hipStream_t s) {
    if (B == 0) return hipSuccess;
    hipError_t e;
    if (wdt == 1 && xdt == 1)
        e = launch_rows_t<bf16_t, bf16_t>(x, B, d, offsets, idx, nnz, gate_up_c, down_c, L,
                                          partials, P, s);
    else if (wdt == 1 && xdt == 0)
        e = launch_rows_t<bf16_t, float>(x, B, d, offsets, idx, nnz, gate_up_c, down_c, L,
                                         partials, P, s);
    else if (wdt == 0 && xdt == 1)
        e = launch_rows_t<float, bf16_t>(x, B, d, offsets, idx, nnz, gate_up_c, down_c, L,
                                         partials, P, s);
    else
        e = launch_rows_t<float, float>(x, B, d, offsets, idx, nnz, gate_up_c, down_c, L,
                                        partials, P, s);
    if (e != hipSuccess) return e;
    return launch_reduce_partials(partials, P, B, d, y, s);
}

hipError_t launch_reduce_partials(const float* partials, int P, int64_t B, int64_t d, float* y,
                                  hipStream_t s) {
    if (B == 0) return hipSuccess;
    dim3 grid((unsigned)((d + 31) / 32), (unsigned)B);
    hipLaunchKernelGGL(reduce_partials, grid, dim3(256), 0, s, partials, P, d, y);
    return hipGetLastError();
}

}  // namespace si
