// Union path of the selective SwiGLU FFN for a batch of B >= 2 tokens with bf16 weights and x.
//
// Each token b has its own active set A_b (Selective Computation section). Reading every
// token's rows separately would fetch a row once per token that uses it; instead the rows of
// the union U = A_1 u ... u A_B are read once and both projections become dense bf16 MFMA
// gather-GEMMs over U, with each token's h masked to its own set:
//
//   G, Uu = X[B][d] . gate_c[U]^T, X . up_c[U]^T         (GEMM1, fp32 accumulate)
//   H[b][n] = SiLU(G[b][n]) * Uu[b][n] * [U[n] in A_b]   (fused epilogue, fp32)
//   Y = H[B][|U|] . down_c[U]                             (GEMM2, fp32 accumulate)
//
// H enters GEMM2's bf16 MFMA as a pair hi = bf16(H), lo = bf16(H - hi), so the product keeps
// about 16 significant bits of H (SI_FLAG_FAST_H uses hi only).
//
// Kernels: per-token bitmaps of the active slots; one work-group ORs them into the union and
// lists its slots in ascending order; GEMM1 (v_mfma_f32_16x16x32_bf16, 16 tokens x 16 union
// rows per work-group, K split over 4 waves and summed in LDS in a fixed order); GEMM2 (16*MT
// tokens x 256 columns per work-group, down rows staged through LDS, K = union rows split in
// KS chunks whose float32 partials are added in a fixed order by the decode path's reducer).
#include "common.h"
#include "launch.h"

namespace si {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4_t;

namespace {

__device__ __forceinline__ bf16x8_t as_bf16x8(const V16& v) {
    const u32x4_t t = {v.w[0], v.w[1], v.w[2], v.w[3]};
    return __builtin_bit_cast(bf16x8_t, t);
}

__device__ __forceinline__ f32x4_t mfma16x16x32(const bf16x8_t& a, const bf16x8_t& b,
                                                const f32x4_t& c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

struct Plan {
    int64_t W;      // 32-bit words per token bitmap
    int64_t Lp;     // row stride of H (union index), multiple of 64
    int KS;         // GEMM2 split-K chunks
    int MT;         // GEMM2 m-subtiles (16 tokens each) per work-group
    size_t off_bits, off_list, off_count, off_h, off_part, total;
};

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

Plan make_plan(int64_t B, int64_t L, int64_t d, int num_cu) {
    Plan p;
    p.W = (L + 31) / 32;
    p.Lp = (L + 63) / 64 * 64;
    p.MT = B >= 128 ? 8 : (B >= 64 ? 4 : (B >= 32 ? 2 : 1));
    const int64_t ntn = (d + 255) / 256;
    const int64_t ntm = (B + 16 * p.MT - 1) / (16 * p.MT);
    int64_t ks = (2 * (int64_t)num_cu + ntn * ntm - 1) / (ntn * ntm);
    const int64_t kmax = (L + 31) / 32;
    if (ks > kmax) ks = kmax;
    if (ks > 64) ks = 64;
    if (ks < 1) ks = 1;
    p.KS = (int)ks;
    size_t o = 0;
    p.off_bits = o;
    o = align256(o + (size_t)B * p.W * 4);
    p.off_list = o;
    o = align256(o + (size_t)L * 4);
    p.off_count = o;
    o = align256(o + 16);
    p.off_h = o;
    o = align256(o + (size_t)B * p.Lp * 4);
    p.off_part = o;
    o = align256(o + (size_t)p.KS * B * d * 4);
    p.total = o;
    return p;
}

// Token b's active slots as a bitmap of L bits (LDS), written to bits[b][0..W).
__global__ __launch_bounds__(256) void token_bitmaps(const int32_t* __restrict__ offsets,
                                                     const int32_t* __restrict__ idx,
                                                     int64_t nnz, int64_t L, int64_t W,
                                                     uint32_t* __restrict__ bits) {
    extern __shared__ uint32_t bm[];
    const int64_t b = blockIdx.x;
    int64_t lo = offsets[b], hi = offsets[b + 1];
    lo = lo < 0 ? 0 : (lo > nnz ? nnz : lo);
    hi = hi < lo ? lo : (hi > nnz ? nnz : hi);
    for (int64_t q = threadIdx.x; q < W; q += 256) bm[q] = 0u;
    __syncthreads();
    for (int64_t r = lo + threadIdx.x; r < hi; r += 256) {
        const int32_t s = idx[r];
        if (s >= 0 && s < L) atomicOr(&bm[s >> 5], 1u << (s & 31));
    }
    __syncthreads();
    for (int64_t q = threadIdx.x; q < W; q += 256) bits[b * W + q] = bm[q];
}

// Union of the B bitmaps, listed as ascending slot ids; count[0] = |U|.
constexpr int kUThreads = 1024;
__global__ __launch_bounds__(kUThreads) void build_union(const uint32_t* __restrict__ bits,
                                                         int64_t B, int64_t W,
                                                         int32_t* __restrict__ ulist,
                                                         int32_t* __restrict__ count) {
    __shared__ int wave_cnt[kUThreads / kWave];
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    int64_t run = 0;
    for (int64_t base = 0; base < W; base += kUThreads) {
        const int64_t q = base + threadIdx.x;
        uint32_t u = 0u;
        if (q < W)
            for (int64_t b = 0; b < B; ++b) u |= bits[b * W + q];
        const int c = __popc(u);
        // exclusive prefix of c over the block: wave inclusive scan + wave totals
        int incl = c;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int t = __shfl_up(incl, o, kWave);
            if (lane >= o) incl += t;
        }
        if (lane == 63) wave_cnt[w] = incl;
        __syncthreads();
        int before = 0, all = 0;
        for (int qq = 0; qq < kUThreads / kWave; ++qq) {
            before += qq < w ? wave_cnt[qq] : 0;
            all += wave_cnt[qq];
        }
        __syncthreads();
        int64_t pos = run + before + incl - c;
        while (u) {
            const int bit = __ffs(u) - 1;
            ulist[pos++] = (int32_t)(q * 32 + bit);
            u &= u - 1u;
        }
        run += all;
    }
    if (threadIdx.x == 0) count[0] = (int32_t)run;
}

// GEMM1 + SiLU*up*mask epilogue. Work-group: 16 tokens (blockIdx.y) x 16 union rows
// (blockIdx.x); 4 waves take K blocks of 128 round-robin. Within a K block, lane (n, g)
// (n = lane % 16, g = lane / 16) reads 64 contiguous bytes of row n at offset g*32 and feeds
// them to 4 MFMAs; the token operand uses the same K permutation, so the sum is unchanged.
__global__ __launch_bounds__(256) void union_gemm1(const bf16_t* __restrict__ x, int64_t B,
                                                   int64_t d, const bf16_t* __restrict__ gu,
                                                   const int32_t* __restrict__ ulist,
                                                   const int32_t* __restrict__ count,
                                                   const uint32_t* __restrict__ bits, int64_t W,
                                                   float* __restrict__ H, int64_t Lp) {
    const int64_t nU = count[0];
    const int64_t n0 = (int64_t)blockIdx.x * 16;
    if (n0 >= nU) return;
    const int64_t m0 = (int64_t)blockIdx.y * 16;
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    const int nn = lane & 15;
    const int g = lane >> 4;
    const bool nok = n0 + nn < nU;
    const int64_t slot = nok ? ulist[n0 + nn] : 0;
    const bool mok = m0 + nn < B;
    const bf16_t* grow = gu + slot * 2 * d;
    const bf16_t* urow = grow + d;
    const bf16_t* xrow = x + (mok ? (m0 + nn) : 0) * d;

    f32x4_t accg = {0.f, 0.f, 0.f, 0.f};
    f32x4_t accu = {0.f, 0.f, 0.f, 0.f};
    const int64_t nkb = (d + 127) / 128;
    const V16 z = V16{{0u, 0u, 0u, 0u}};
    for (int64_t kb = w; kb < nkb; kb += 4) {
        const int64_t base = kb * 128 + g * 32;
        V16 gv[4], uv[4], xv[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int64_t pos = base + e * 8;
            const bool in = pos < d;
            gv[e] = (in && nok) ? ld16(grow + pos) : z;
            uv[e] = (in && nok) ? ld16(urow + pos) : z;
            xv[e] = (in && mok) ? ld16(xrow + pos) : z;
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const bf16x8_t a = as_bf16x8(xv[e]);
            accg = mfma16x16x32(a, as_bf16x8(gv[e]), accg);
            accu = mfma16x16x32(a, as_bf16x8(uv[e]), accu);
        }
    }
    __shared__ float red[4][2][4][64];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        red[w][0][i][lane] = accg[i];
        red[w][1][i][lane] = accu[i];
    }
    __syncthreads();
    if (w != 0) return;
    // accumulator layout: register i of lane l is (token 4*(l/16) + i, row l % 16)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        float gs = 0.f, us = 0.f;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            gs += red[q][0][i][lane];
            us += red[q][1][i][lane];
        }
        const int64_t tok = m0 + 4 * g + i;
        const int64_t n = n0 + nn;
        if (tok < B && n < nU) {
            const uint32_t s = (uint32_t)ulist[n];
            const bool act = (bits[tok * W + (s >> 5)] >> (s & 31)) & 1u;
            H[tok * Lp + n] = act ? silu_f32(gs) * us : 0.0f;
        }
    }
}

// GEMM2: partial[b][ks][c] = sum over union rows n in chunk ks of H[b][n] * down_c[U[n]][c].
// Work-group: 16*MT tokens x 256 columns; wave w owns columns w*64 .. w*64+63 (4 MFMA
// n-subtiles). Per K step of 32 union rows the 256 threads stage a [32][256] tile of down
// rows in LDS (16-byte loads); lane (n, g) then reads its B operand (8 rows of one column).
template <int MT>
__global__ __launch_bounds__(256) void union_gemm2(const float* __restrict__ H, int64_t Lp,
                                                   int64_t B, const bf16_t* __restrict__ dc,
                                                   int64_t d, const int32_t* __restrict__ ulist,
                                                   const int32_t* __restrict__ count,
                                                   float* __restrict__ part, int KS, int fast) {
    const int64_t nU = count[0];
    const int ks = blockIdx.z;
    int64_t chunk = (nU + KS - 1) / KS;
    chunk = (chunk + 31) / 32 * 32;
    const int64_t kbeg = (int64_t)ks * chunk;
    const int64_t kend = (kbeg + chunk < nU) ? kbeg + chunk : nU;
    const int64_t c0 = (int64_t)blockIdx.x * 256;
    const int64_t m0 = (int64_t)blockIdx.y * 16 * MT;
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    const int nn = lane & 15;
    const int g = lane >> 4;

    __shared__ __align__(16) uint16_t tile[32][256];
    f32x4_t acc[MT][4];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[mt][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    const int sr = threadIdx.x >> 3;        // staging: row 0..31
    const int sc = (threadIdx.x & 7) * 32;  // staging: first of 32 columns
    const V16 z = V16{{0u, 0u, 0u, 0u}};
    for (int64_t k0 = kbeg; k0 < kend; k0 += 32) {
        {
            const int64_t k = k0 + sr;
            const bool rok = k < kend;
            const int64_t slot = rok ? ulist[k] : 0;
            const bf16_t* src = dc + slot * d + c0 + sc;
            V16 v[4];
#pragma unroll
            for (int e = 0; e < 4; ++e)
                v[e] = (rok && c0 + sc + e * 8 < d) ? ld16(src + e * 8) : z;
            __syncthreads();
#pragma unroll
            for (int e = 0; e < 4; ++e) st16(&tile[sr][sc + e * 8], v[e]);
            __syncthreads();
        }
        bf16x8_t bop[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int col = w * 64 + j * 16 + nn;
            uint32_t pk[4];
#pragma unroll
            for (int q = 0; q < 4; ++q)
                pk[q] = (uint32_t)tile[g * 8 + 2 * q][col] |
                        ((uint32_t)tile[g * 8 + 2 * q + 1][col] << 16);
            bop[j] = as_bf16x8(V16{{pk[0], pk[1], pk[2], pk[3]}});
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const int64_t tok = m0 + mt * 16 + nn;
            float hv[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int64_t k = k0 + g * 8 + e;
                hv[e] = (tok < B && k < kend) ? H[tok * Lp + k] : 0.0f;
            }
            uint32_t hi[4], lo[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint32_t h0 = f32_to_bf16_rne(hv[2 * q]);
                const uint32_t h1 = f32_to_bf16_rne(hv[2 * q + 1]);
                hi[q] = h0 | (h1 << 16);
                const uint32_t l0 = f32_to_bf16_rne(hv[2 * q] - bf16_to_f32(h0));
                const uint32_t l1 = f32_to_bf16_rne(hv[2 * q + 1] - bf16_to_f32(h1));
                lo[q] = l0 | (l1 << 16);
            }
            const bf16x8_t ahi = as_bf16x8(V16{{hi[0], hi[1], hi[2], hi[3]}});
            const bf16x8_t alo = as_bf16x8(V16{{lo[0], lo[1], lo[2], lo[3]}});
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                acc[mt][j] = mfma16x16x32(ahi, bop[j], acc[mt][j]);
                if (!fast) acc[mt][j] = mfma16x16x32(alo, bop[j], acc[mt][j]);
            }
        }
    }
    // accumulator: register i of lane l is (token 4*(l/16) + i, column l % 16) of a subtile
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int64_t tok = m0 + mt * 16 + 4 * g + i;
                const int64_t col = c0 + w * 64 + j * 16 + nn;
                if (tok < B && col < d) part[(tok * KS + ks) * d + col] = acc[mt][j][i];
            }
}

}  // namespace

size_t union_workspace(int64_t B, int64_t L, int64_t d, int num_cu) {
    return make_plan(B, L, d, num_cu).total;
}

hipError_t launch_union(const void* x, int64_t B, int64_t d, const int32_t* offsets,
                        const int32_t* idx, int64_t nnz, const void* gate_up_c,
                        const void* down_c, int64_t L, float* y, void* ws, int flags,
                        int num_cu, hipStream_t s) {
    const Plan p = make_plan(B, L, d, num_cu);
    uint8_t* base = static_cast<uint8_t*>(ws);
    uint32_t* bits = reinterpret_cast<uint32_t*>(base + p.off_bits);
    int32_t* ulist = reinterpret_cast<int32_t*>(base + p.off_list);
    int32_t* count = reinterpret_cast<int32_t*>(base + p.off_count);
    float* H = reinterpret_cast<float*>(base + p.off_h);
    float* part = reinterpret_cast<float*>(base + p.off_part);
    const bf16_t* xx = static_cast<const bf16_t*>(x);
    const bf16_t* gu = static_cast<const bf16_t*>(gate_up_c);
    const bf16_t* dc = static_cast<const bf16_t*>(down_c);

    hipLaunchKernelGGL(token_bitmaps, dim3((unsigned)B), dim3(256), (size_t)p.W * 4, s, offsets,
                       idx, nnz, L, p.W, bits);
    hipLaunchKernelGGL(build_union, dim3(1), dim3(kUThreads), 0, s, bits, B, p.W, ulist, count);
    hipLaunchKernelGGL(union_gemm1, dim3((unsigned)((L + 15) / 16), (unsigned)((B + 15) / 16)),
                       dim3(256), 0, s, xx, B, d, gu, ulist, count, bits, p.W, H, p.Lp);
    const int fast = (flags & 4) ? 1 : 0;
    dim3 g2((unsigned)((d + 255) / 256), (unsigned)((B + 16 * p.MT - 1) / (16 * p.MT)),
            (unsigned)p.KS);
#define SI_G2(MTV)                                                                             \
    hipLaunchKernelGGL(union_gemm2<MTV>, g2, dim3(256), 0, s, H, p.Lp, B, dc, d, ulist, count, \
                       part, p.KS, fast)
    switch (p.MT) {
        case 8: SI_G2(8); break;
        case 4: SI_G2(4); break;
        case 2: SI_G2(2); break;
        default: SI_G2(1); break;
    }
#undef SI_G2
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_reduce_partials(part, p.KS, B, d, y, s);
}

}  // namespace si
