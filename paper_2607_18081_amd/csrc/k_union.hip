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
// Kernels:
//  - token bitmaps: one work-group per token marks its active slots in an L-bit bitmap;
//  - GEMM1 (v_mfma_f32_16x16x32_bf16): one work-group per 32-slot bitmap word and 16 x MT1
//    tokens. It ORs the word over the batch (the union's slots in this word), takes those rows
//    as two 16-row MFMA tiles (slots outside the union load nothing: their loads are out of
//    range), splits K over 8 waves that meet in LDS in a fixed order, and writes H by slot,
//    zero for slots outside the union. Within a K block of 128, the lanes of group g feed
//    elements 32 e + 8 g .. +7 to MFMA e; the token operand uses the same K permutation, so
//    the sum is unchanged. The weight rows are loaded in whole 128-byte lines and reach that
//    layout through the wave's own LDS area. The y = 0 work-groups also publish the union
//    word for GEMM2;
//  - GEMM2: a work-group takes 16 x MT tokens, 256 columns and one of KS chunks of bitmap
//    words, with K = slot: each non-empty word is one K step of 32 slots whose down rows (zero
//    rows outside the union, again without memory traffic) are staged in LDS, double buffered
//    with three tiles in flight, and read back transposed into the MFMA B-operand layout with
//    ds_read_b64_tr_b16 (non-temporal row loads when one token tile reads each row once).
//    The KS float32 partials are added in a fixed order by the shared partial reducer.
#include <hip/hip_ext.h>

#include "common.h"
#include "launch.h"
#include "mfma.h"
#include "selectinfer.h"

namespace si {

typedef __attribute__((ext_vector_type(4))) short s16x4_t;

namespace {

constexpr int kG2Waves = 4;                // GEMM2 waves per work-group, 64 columns each
constexpr int kG2Cols = 64 * kG2Waves;     // GEMM2 columns per work-group
constexpr int kG2Pitch = kG2Cols + 16;     // LDS row pitch (bf16): rows 32 bytes apart in bank
constexpr int kG2Tpr = kG2Cols / 32;       // staging threads per tile row (4 x 8 columns each)
constexpr int kGemm1Waves = 8;
constexpr int kWordRegs = 4;               // GEMM2 chunks span at most 64 kWordRegs words

struct Plan {
    int64_t W;      // 32-bit words per token bitmap (slot s is bit s % 32 of word s / 32)
    int64_t Lp;     // row stride of H, indexed by slot: 32 W rounded up to 64
    int KS;         // GEMM2 split-K chunks (of bitmap words)
    int MT;         // GEMM2 m-subtiles (16 tokens each) per work-group
    int MT1;        // GEMM1 m-subtiles per work-group
    size_t off_bits, off_words, off_h, off_part, total;
};

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

Plan make_plan(int64_t B, int64_t L, int64_t d, int num_cu) {
    Plan p;
    p.W = (L + 31) / 32;
    p.Lp = (p.W * 32 + 63) / 64 * 64;
    // token tiles of 16 MT (GEMM2) and 16 MT1 (GEMM1) tokens: the smallest that holds the
    // batch up to 64 tokens, since each tile streams the union rows again
    p.MT = B >= 128 ? 8 : (B > 32 ? 4 : (B > 16 ? 2 : 1));
    p.MT1 = B > 32 ? 4 : (B > 16 ? 2 : 1);
    const int64_t ntn = (d + kG2Cols - 1) / kG2Cols;
    const int64_t ntm = (B + 16 * p.MT - 1) / (16 * p.MT);
    int64_t ks = ((int64_t)num_cu + ntn * ntm - 1) / (ntn * ntm);
    if (ks > p.W) ks = p.W;
    if (ks > 64) ks = 64;
    // no chunk longer than GEMM2 holds in registers (W <= 16384 keeps this at most 64)
    const int64_t ks_min = (p.W + 64 * kWordRegs - 1) / (64 * kWordRegs);
    if (ks < ks_min) ks = ks_min;
    if (ks < 1) ks = 1;
    p.KS = (int)ks;
    size_t o = 0;
    p.off_bits = o;
    o = align256(o + (size_t)B * p.W * 4);
    p.off_words = o;
    o = align256(o + (size_t)p.W * 4);
    p.off_h = o;
    o = align256(o + (size_t)B * p.Lp * 4);
    p.off_part = o;
    o = align256(o + (size_t)p.KS * B * part_chunks(d) * kChunk * 4);
    p.total = o;
    return p;
}

__device__ __forceinline__ void clamp_range(const int32_t* offsets, int64_t b, int64_t nnz,
                                            int64_t& lo, int64_t& hi) {
    lo = offsets[b];
    hi = offsets[b + 1];
    lo = lo < 0 ? 0 : (lo > nnz ? nnz : lo);
    hi = hi < lo ? lo : (hi > nnz ? nnz : hi);
}

// Position of the r-th (0-based) set bit of u; requires r < popcount(u).
__device__ __forceinline__ int nth_set_bit(uint32_t u, int r) {
    int pos = 0;
#pragma unroll
    for (int half = 16; half >= 1; half >>= 1) {
        const uint32_t low = (1u << half) - 1u;
        const int c = __popc(u & low);
        if (r >= c) {
            r -= c;
            u >>= half;
            pos += half;
        } else {
            u &= low;
        }
    }
    return pos;
}

// Token b's active slots as a bitmap (LDS), written to bits[b][0..W). The ids are read 4096
// at a time, four range-checked loads per thread issued together, so a token's list costs one
// memory round trip per 4096 ids rather than one per 256.
constexpr int kBmThreads = 1024;
__global__ __launch_bounds__(kBmThreads) void token_bitmaps(const int32_t* __restrict__ offsets,
                                                            const int32_t* __restrict__ idx,
                                                            int64_t nnz, int64_t L, int64_t W,
                                                            uint32_t* __restrict__ bits) {
    extern __shared__ uint32_t bm[];
    constexpr int U = 4;
    const int64_t b = blockIdx.x;
    for (int64_t q = threadIdx.x; q < W; q += kBmThreads) bm[q] = 0u;
    int64_t lo, hi;
    clamp_range(offsets, b, nnz, lo, hi);
    __syncthreads();
    for (int64_t r0 = lo; r0 < hi; r0 += (int64_t)kBmThreads * U) {
        const int64_t nr = hi - r0 < (int64_t)kBmThreads * U ? hi - r0 : (int64_t)kBmThreads * U;
        const __amdgpu_buffer_rsrc_t ri = make_rsrc(idx + r0, nr * 4);
        int32_t sv[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
            sv[u] = __builtin_amdgcn_raw_buffer_load_b32(ri, (u * kBmThreads + (int)threadIdx.x) * 4,
                                                         0, 0);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int32_t sl = sv[u];
            if (u * kBmThreads + (int)threadIdx.x < nr && sl >= 0 && sl < L)
                atomicOr(&bm[sl >> 5], 1u << (sl & 31));
        }
    }
    __syncthreads();
    for (int64_t q = threadIdx.x; q < W; q += kBmThreads) bits[b * W + q] = bm[q];
}

// GEMM1 + SiLU*up*mask epilogue (see the file comment). Grid: (W, ceil(B/(16*MT1))).
// NT: one token tile, so each weight row is read once: its loads carry the non-temporal
// policy (with two tiles the second would miss the rows the first brought in)
template <typename ET, int MT1, bool NT>
__global__ __launch_bounds__(64 * kGemm1Waves) void union_gemm1(
    const uint16_t* __restrict__ x, int64_t B, int64_t d, const uint16_t* __restrict__ gu,
    int64_t L, const uint32_t* __restrict__ bits, int64_t W, uint32_t* __restrict__ words,
    float* __restrict__ H, int64_t Lp) {
    constexpr int MTOK = 16 * MT1;
    const int64_t wd = blockIdx.x;                 // slots 32 wd .. 32 wd + 31
    const int64_t m0 = (int64_t)blockIdx.y * MTOK;
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    const int nn = lane & 15;
    const int g = lane >> 4;

    // this word of the union (OR over the batch) and of each token of the tile
    // (both first reads in one memory round trip: range-checked loads, no branches)
    __shared__ uint32_t wor[kGemm1Waves];
    __shared__ uint32_t tokw[MTOK];
    const __amdgpu_buffer_rsrc_t rbits = make_rsrc(bits, B * W * 4);
    constexpr int kT1 = 64 * kGemm1Waves;
    const int64_t tk = m0 + threadIdx.x;
    const uint32_t tw = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(
        rbits, (threadIdx.x < MTOK && tk < B) ? (int)((tk * W + wd) * 4) : kOOB, 0, 0);
    uint32_t uw = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(
        rbits, threadIdx.x < B ? (int)((threadIdx.x * W + wd) * 4) : kOOB, 0, 0);
    for (int64_t b = threadIdx.x + kT1; b < B; b += kT1) uw |= bits[b * W + wd];
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) uw |= (uint32_t)__shfl_xor((int)uw, m, kWave);
    if (lane == 0) wor[w] = uw;
    if (threadIdx.x < MTOK) tokw[threadIdx.x] = tw;
    __syncthreads();
    uint32_t u = 0u;
#pragma unroll
    for (int q = 0; q < kGemm1Waves; ++q) u |= wor[q];
    if (blockIdx.y == 0 && threadIdx.x == 0) words[wd] = u;
    const int n = __popc(u);

    // H of the slots outside the union is zero
    for (int q = threadIdx.x; q < MTOK * 32; q += 64 * kGemm1Waves) {
        const int64_t tok = m0 + q / 32;
        const int j = q % 32;
        if (tok < B && !((u >> j) & 1u)) H[tok * Lp + wd * 32 + j] = 0.0f;
    }
    if (n == 0) return;

    // row nn of MFMA tile st is the (16 st + nn)-th union slot of this word
    const __amdgpu_buffer_rsrc_t rg = make_rsrc(gu, L * 2 * d * 2);
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(x, B * d * 2);
    int64_t slot[2];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
        const int r = 16 * st + nn;
        slot[st] = r < n ? wd * 32 + nth_set_bit(u, r) : -1;
    }
    // loads take whole 128-byte lines: load q of tile st gives lane l row 4 q + l / 16 of the
    // tile, 16-byte chunk l % 16 of the K block (8 lanes per line, 8 lines per instruction)
    int goff[2][4];
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int r = 16 * st + 4 * q + (lane >> 4);
            goff[st][q] = r < n ? (int)((wd * 32 + nth_set_bit(u, r)) * 4 * d) : kOOB;  // gate row
        }
    int xoff[MT1];
#pragma unroll
    for (int mt = 0; mt < MT1; ++mt) {
        const int64_t tok = m0 + mt * 16 + nn;
        xoff[mt] = tok < B ? (int)(tok * 2 * d) : kOOB;
    }
    f32x4_t accg[MT1][2], accu[MT1][2];
#pragma unroll
    for (int mt = 0; mt < MT1; ++mt)
#pragma unroll
        for (int st = 0; st < 2; ++st) {
            accg[mt][st] = f32x4_t{0.f, 0.f, 0.f, 0.f};
            accu[mt][st] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        }
    const int ntile = n > 16 ? 2 : 1;
    const int64_t nkb = (d + 127) / 128;
    constexpr int kStgPitch = 256;                      // bytes per staged row (unpadded)
    constexpr int kStgWave = 4 * 16 * kStgPitch;        // gate and up rows of both tiles
    __shared__ __align__(16) uint8_t stg[kGemm1Waves * kStgWave];
    // The wave's K blocks are kb = w, w + 8, ...: the loads of the next block are in flight
    // while the MFMAs of the current one run (two register sets, the loop unrolled by two).
    // Blocks past the end load nothing (out-of-range offsets) and add zeros. The MFMAs of the
    // second tile run even when it is empty: a load used only under a branch would be moved
    // into it, behind the MFMAs of the first tile.
    struct Blk {
        V16 g[2][4], u[2][4], x[MT1][4];
    };
    auto load = [&](int64_t kb, Blk& bk) {
        const int64_t wpos = kb * 128 + 8 * nn;  // this lane's element of the row (chunk nn)
#pragma unroll
        for (int st = 0; st < 2; ++st)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const bool in = wpos < d && goff[st][q] != kOOB;
                const int og = in ? goff[st][q] + (int)(wpos * 2) : kOOB;
                const int ou = in ? goff[st][q] + (int)((d + wpos) * 2) : kOOB;
                bk.g[st][q] = NT ? bload16nt(rg, og) : bload16(rg, og);
                bk.u[st][q] = NT ? bload16nt(rg, ou) : bload16(rg, ou);
            }
#pragma unroll
        for (int mt = 0; mt < MT1; ++mt)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int64_t pos = kb * 128 + e * 32 + g * 8;
                bk.x[mt][e] = bload16(rx, (pos < d && xoff[mt] != kOOB) ? xoff[mt] + (int)(pos * 2)
                                                                        : kOOB);
            }
    };
    // The lines pass through this wave's own LDS area (no barrier: a wave's LDS accesses
    // complete in order) and come back in the MFMA layout, lane (nn, g) holding row nn, chunk
    // 4 e + g for MFMA e. 16-byte chunk c of row r is stored at position c ^ (r % 16), so the
    // 16 rows one read touches, and the 16 chunks one row's store writes, fall in distinct
    // banks (the hardware's bank-conflict counter reads zero; with rows padded to 272 bytes
    // it read 1.7 cycles per access).
    uint8_t* my_stg = stg + w * kStgWave;
    auto mma = [&](const Blk& bk) {
#pragma unroll
        for (int st = 0; st < 2; ++st)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int row = 4 * q + (lane >> 4);
                const int off = row * kStgPitch + 16 * (nn ^ (row & 15));
                st16(my_stg + (2 * st) * 16 * kStgPitch + off, bk.g[st][q]);
                st16(my_stg + (2 * st + 1) * 16 * kStgPitch + off, bk.u[st][q]);
            }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            typename Mfma<ET>::vec8 wg_[2], wu_[2];
#pragma unroll
            for (int st = 0; st < 2; ++st) {
                const int off = nn * kStgPitch + 16 * ((4 * e + g) ^ nn);
                wg_[st] = Mfma<ET>::vec(ld16(my_stg + (2 * st) * 16 * kStgPitch + off));
                wu_[st] = Mfma<ET>::vec(ld16(my_stg + (2 * st + 1) * 16 * kStgPitch + off));
            }
#pragma unroll
            for (int mt = 0; mt < MT1; ++mt) {
                const typename Mfma<ET>::vec8 a = Mfma<ET>::vec(bk.x[mt][e]);
#pragma unroll
                for (int st = 0; st < 2; ++st) {
                    accg[mt][st] = Mfma<ET>::mma(a, wg_[st], accg[mt][st]);
                    accu[mt][st] = Mfma<ET>::mma(a, wu_[st], accu[mt][st]);
                }
            }
        }
    };
    // (the scheduling barriers keep each block's loads ahead of the other block's MFMAs).
    // With two or four token tiles two register sets do not fit: one block at a time.
    if constexpr (MT1 == 1) {
        Blk b0, b1;
        load(w, b0);
        for (int64_t kb = w; kb < nkb; kb += 2 * kGemm1Waves) {
            load(kb + kGemm1Waves, b1);
            __builtin_amdgcn_sched_barrier(0);
            mma(b0);
            __builtin_amdgcn_sched_barrier(0);
            load(kb + 2 * kGemm1Waves, b0);
            __builtin_amdgcn_sched_barrier(0);
            mma(b1);
            __builtin_amdgcn_sched_barrier(0);
        }
    } else {
        for (int64_t kb = w; kb < nkb; kb += kGemm1Waves) {
            Blk b0;
            load(kb, b0);
            __builtin_amdgcn_sched_barrier(0);
            mma(b0);
        }
    }
    // the 8 waves' partial tiles meet in LDS; wave 0 adds them in a fixed order
    __shared__ float red[kGemm1Waves][2][4][64];
#pragma unroll
    for (int mt = 0; mt < MT1; ++mt)
#pragma unroll
        for (int st = 0; st < 2; ++st) {
            if (st >= ntile) continue;                    // uniform
            __syncthreads();
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                red[w][0][i][lane] = accg[mt][st][i];
                red[w][1][i][lane] = accu[mt][st][i];
            }
            __syncthreads();
            if (w == 0) {
                // accumulator layout: register i of lane l is (token 4*(l/16) + i, row l % 16)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    float gs = 0.f, us = 0.f;
#pragma unroll
                    for (int q = 0; q < kGemm1Waves; ++q) {
                        gs += red[q][0][i][lane];
                        us += red[q][1][i][lane];
                    }
                    const int tl = mt * 16 + 4 * g + i;       // token within the tile
                    const int64_t tok = m0 + tl;
                    if (tok < B && slot[st] >= 0) {
                        const bool act = (tokw[tl] >> (slot[st] - wd * 32)) & 1u;
                        H[tok * Lp + slot[st]] = act ? silu_f32(gs) * us : 0.0f;
                    }
                }
            }
        }
}

// GEMM2 (see the file comment). Grid: (ceil(d / kG2Cols), ceil(B/(16*MT)), KS); kG2Waves waves,
// wave w taking columns 64 w .. 64 w + 63 of the tile.
// FAST: H enters the MFMA as its bf16 (or half) rounding alone, without the low part.
// NT: one token tile, so each down row is read once: non-temporal loads.
template <typename ET, int MT, bool FAST, bool NT>
__global__ __launch_bounds__(64 * kG2Waves) void union_gemm2(const float* __restrict__ H, int64_t Lp,
                                                   int64_t B, const uint16_t* __restrict__ dc,
                                                   int64_t d, int64_t L,
                                                   const uint32_t* __restrict__ words, int64_t W,
                                                   float* __restrict__ part, int KS) {
    const int ks = blockIdx.z;
    const int64_t cw = (W + KS - 1) / KS;          // bitmap words per chunk
    const int64_t w0 = (int64_t)ks * cw < W ? (int64_t)ks * cw : W;  // chunk ks may be empty
    const int64_t w1 = (w0 + cw < W) ? w0 + cw : W;
    const int64_t c0 = (int64_t)blockIdx.x * kG2Cols;
    const int64_t m0 = (int64_t)blockIdx.y * 16 * MT;
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    const int nn = lane & 15;
    const int g = lane >> 4;

    __shared__ __align__(16) uint16_t tile[2][32][kG2Pitch];
    f32x4_t acc[MT][4];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[mt][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    const __amdgpu_buffer_rsrc_t rd = make_rsrc(dc, L * d * 2);
    const int sr = threadIdx.x / kG2Tpr;     // staging: tile row (slot 32 wd + sr)
    // staging: the kG2Tpr lanes of a tile row take 16 contiguous bytes each of kG2Cols / 4
    // columns per load (columns kG2Cols / 4 * e + 8 (t % kG2Tpr) .. + 7 in load e), so a load
    // reads whole 128-byte lines
    const int sc = (threadIdx.x % kG2Tpr) * 8;
    // words of down rows in flight in registers ahead of the LDS tile being consumed: deeper
    // for few tokens, where the kernel only streams rows and register room is plentiful
    constexpr int kDepth = MT == 1 ? 8 : (MT == 2 ? 6 : 3);
    // The lane's chunk of a word's down rows and its H values (the A operand of its MT token
    // tiles) travel kDepth words ahead: consuming a word then waits for no memory access.
    V16 nxt[kDepth][4];
    float nh[kDepth][MT][8];
    const __amdgpu_buffer_rsrc_t rh = make_rsrc(H, B * Lp * 4);
    // The chunk's union words (at most 64 kWordRegs) are read once, spread over the lanes:
    // word w0 + 64 i + l sits in register i of lane l (0 past the chunk), and each step takes
    // its word from there with a lane read, so the row fetches never wait for a word load.
    uint32_t wl[kWordRegs];
    {
        const __amdgpu_buffer_rsrc_t rw = make_rsrc(words + w0, (w1 - w0) * 4);
#pragma unroll
        for (int i = 0; i < kWordRegs; ++i)
            wl[i] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(rw, (i * 64 + lane) * 4, 0, 0);
    }
    auto word_at = [&](int64_t wd) -> uint32_t {
        const int r = (int)(wd - w0);            // uniform; 0 <= r
        uint32_t u = 0u;
#pragma unroll
        for (int i = 0; i < kWordRegs; ++i)
            u = (r >> 6) == i ? (uint32_t)__builtin_amdgcn_readlane((int)wl[i], r & 63) : u;
        return u;
    };
    auto fetch = [&](int64_t wd, V16 (&v)[4], float (&hv)[MT][8]) {
        const uint32_t u = word_at(wd);
        const bool rok = (u >> sr) & 1u;
        const int64_t slot = wd * 32 + sr;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int64_t col = c0 + e * (kG2Cols / 4) + sc;
            const int off = (rok && col < d) ? (int)((slot * d + col) * 2) : kOOB;
            v[e] = NT ? bload16nt(rd, off) : bload16(rd, off);
        }
        // H of token tok at slots 32 wd + 8 g .. +7 (contiguous, 32-byte aligned)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const int64_t tok = m0 + mt * 16 + nn;
            const int off = (tok < B && u != 0u) ? (int)((tok * Lp + wd * 32 + g * 8) * 4) : kOOB;
            const V16 lo = bload16(rh, off);
            const V16 hi = bload16(rh, off == kOOB ? kOOB : off + 16);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                hv[mt][e] = __uint_as_float(lo.w[e]);
                hv[mt][4 + e] = __uint_as_float(hi.w[e]);
            }
        }
    };
    // the A operands of the MT token tiles from a word's H values: the hi and lo roundings
    typedef typename Mfma<ET>::vec8 AV;
    auto a_ops = [&](const float (&hvs)[MT][8], AV (&ahi)[MT], AV (&alo)[MT]) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const float* hv = hvs[mt];
            uint32_t hi[4], lo[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint32_t h0 = Mfma<ET>::rne(hv[2 * q]);
                const uint32_t h1 = Mfma<ET>::rne(hv[2 * q + 1]);
                hi[q] = h0 | (h1 << 16);
                if (!FAST) {
                    const uint32_t l0 = Mfma<ET>::rne(hv[2 * q] - Mfma<ET>::widen(h0));
                    const uint32_t l1 = Mfma<ET>::rne(hv[2 * q + 1] - Mfma<ET>::widen(h1));
                    lo[q] = l0 | (l1 << 16);
                }
            }
            ahi[mt] = Mfma<ET>::vec(V16{{hi[0], hi[1], hi[2], hi[3]}});
            if (!FAST) alo[mt] = Mfma<ET>::vec(V16{{lo[0], lo[1], lo[2], lo[3]}});
        }
    };
    // consume the LDS tile `bsel` holding slots 32 wd .. 32 wd + 31, with the word's A operands
    auto consume = [&](int bsel, const AV (&ahi)[MT], const AV (&alo)[MT]) {
        // B operand: lane (nn, g) needs rows 8g..8g+7 of column nn of each 16-column subtile;
        // ds_read_b64_tr_b16 hands lane i of a 16-lane group element i%4 of the 8-byte pieces
        // addressed by lanes i/4 + 4j, so lane nn addresses row 8g + nn/4 (+4), columns
        // 4*(nn%4) .. +3 of the subtile.
        typename Mfma<ET>::vec8 bop[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int col = w * 64 + j * 16 + 4 * (nn & 3);
            const int row = 8 * g + (nn >> 2);
            const s16x4_t lo4 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (__attribute__((address_space(3))) s16x4_t*)&tile[bsel][row][col]);
            const s16x4_t hi4 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (__attribute__((address_space(3))) s16x4_t*)&tile[bsel][row + 4][col]);
            const uint32_t p0 = (uint16_t)lo4[0] | ((uint32_t)(uint16_t)lo4[1] << 16);
            const uint32_t p1 = (uint16_t)lo4[2] | ((uint32_t)(uint16_t)lo4[3] << 16);
            const uint32_t p2 = (uint16_t)hi4[0] | ((uint32_t)(uint16_t)hi4[1] << 16);
            const uint32_t p3 = (uint16_t)hi4[2] | ((uint32_t)(uint16_t)hi4[3] << 16);
            bop[j] = Mfma<ET>::vec(V16{{p0, p1, p2, p3}});
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                acc[mt][j] = Mfma<ET>::mma(ahi[mt], bop[j], acc[mt][j]);
                if (!FAST) acc[mt][j] = Mfma<ET>::mma(alo[mt], bop[j], acc[mt][j]);
            }
    };
#pragma unroll
    for (int q = 0; q < kDepth; ++q) fetch(w0 + q, nxt[q], nh[q]);
    // The chunk runs to a multiple of kDepth words; the words past its end are empty (their
    // loads are out of range). The unrolled body then has no exit, and every register of the
    // pipeline keeps its place, so no wait for a load in flight is forced before its turn.
    const int64_t wend = w0 + (w1 - w0 + kDepth - 1) / kDepth * kDepth;
    int buf = 0;
    for (int64_t wg = w0; wg < wend; wg += kDepth) {
#pragma unroll
        for (int q = 0; q < kDepth; ++q) {
            const int64_t wd = wg + q;
#pragma unroll
            for (int e = 0; e < 4; ++e) st16(&tile[buf][sr][e * (kG2Cols / 4) + sc], nxt[q][e]);
            const uint32_t word = word_at(wd);
            AV ahi[MT], alo[MT];
            a_ops(nh[q], ahi, alo);
            // the A operands are made here, before nh[q] is refilled: computed where they are
            // used, after the refill, they would keep the old and new H values alive together,
            // and the pipeline's registers would rotate through copies that wait for loads
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                asm volatile("" : "+v"(ahi[mt]));
                if (!FAST) asm volatile("" : "+v"(alo[mt]));
            }
            __syncthreads();
            fetch(wd + kDepth, nxt[q], nh[q]);        // refill: kDepth words ahead
            if (word != 0u) consume(buf, ahi, alo);   // uniform: empty words add nothing
            buf ^= 1;
        }
    }
    // accumulator: register i of lane l is (token 4*(l/16) + i, column l % 16) of a subtile;
    // the 16 lanes of a row write 64 contiguous bytes of the chunked partial layout
    const int64_t nch = part_chunks(d);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int64_t tok = m0 + mt * 16 + 4 * g + i;
                const int64_t col = c0 + w * 64 + j * 16 + nn;
                if (tok < B && col < d) part[part_off(tok, ks, col, KS, nch)] = acc[mt][j][i];
            }
}

}  // namespace

hipError_t launch_token_bitmaps(const int32_t* offsets, const int32_t* idx, int64_t nnz,
                                int64_t B, int64_t L, int64_t W, uint32_t* bits, hipStream_t s) {
    hipLaunchKernelGGL(token_bitmaps, dim3((unsigned)B), dim3(kBmThreads), (size_t)W * 4, s,
                       offsets, idx, nnz, L, W, bits);
    return hipGetLastError();
}

// batches from which the LDS-tiled GEMMs (k_tiled.hip) take over: below, the weights are
// streamed once and the row-word kernels here are bandwidth bound; above, reuse across the
// batch makes the products compute bound
constexpr int64_t kTiledMinB = 128;

static bool use_tiled(int64_t B, int64_t L, int64_t d) {
    return B >= kTiledMinB && tiled_supported(B, L, d);
}

bool union_supported(int64_t B, int64_t L, int64_t d) {
    // buffer loads take 32-bit byte offsets
    return L * 2 * d * 2 < ((int64_t)1 << 31) && B * d * 2 < ((int64_t)1 << 31) &&
           L <= 524288 && B * ((L + 31) / 32) * 4 < ((int64_t)1 << 31);
}

size_t union_workspace(int64_t B, int64_t L, int64_t d, int num_cu, int flags) {
    if (use_tiled(B, L, d)) return tiled_workspace(B, L, d, num_cu, flags);
    return make_plan(B, L, d, num_cu).total;
}

namespace {

template <typename ET>
hipError_t launch_union_t(const void* x, int64_t B, int64_t d, const int32_t* offsets,
                          const int32_t* idx, int64_t nnz, const void* gate_up_c,
                          const void* down_c, int64_t L, float* y, void* ws, int flags,
                          int num_cu, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
    const Plan p = make_plan(B, L, d, num_cu);
    if ((p.W + p.KS - 1) / p.KS > 64 * kWordRegs) return hipErrorInvalidValue;
    uint8_t* base = static_cast<uint8_t*>(ws);
    uint32_t* bits = reinterpret_cast<uint32_t*>(base + p.off_bits);
    uint32_t* words = reinterpret_cast<uint32_t*>(base + p.off_words);
    float* H = reinterpret_cast<float*>(base + p.off_h);
    float* part = reinterpret_cast<float*>(base + p.off_part);
    const uint16_t* xx = static_cast<const uint16_t*>(x);
    const uint16_t* gu = static_cast<const uint16_t*>(gate_up_c);
    const uint16_t* dc = static_cast<const uint16_t*>(down_c);

    hipError_t e = launch_token_bitmaps(offsets, idx, nnz, B, L, p.W, bits, s);
    if (e != hipSuccess) return e;
    const dim3 g1((unsigned)p.W, (unsigned)((B + 16 * p.MT1 - 1) / (16 * p.MT1)));
#define SI_G1(M, N)                                                                            \
    hipExtLaunchKernelGGL((union_gemm1<ET, M, N>), g1, dim3(64 * kGemm1Waves), 0, s, ev0,       \
                          nullptr, 0, xx, B, d, gu, L, bits, p.W, words, H, p.Lp)
    if (g1.y == 1) {
        switch (p.MT1) {
            case 4: SI_G1(4, true); break;
            case 2: SI_G1(2, true); break;
            default: SI_G1(1, true); break;
        }
    } else {  // more than 64 tokens: tiles of 64
        SI_G1(4, false);
    }
#undef SI_G1
    const bool fast = (flags & SI_FLAG_FAST_H) != 0;
    dim3 g2((unsigned)((d + kG2Cols - 1) / kG2Cols),
            (unsigned)((B + 16 * p.MT - 1) / (16 * p.MT)), (unsigned)p.KS);
#define SI_G2F(MTV, F, N)                                                                       \
    hipExtLaunchKernelGGL((union_gemm2<ET, MTV, F, N>), g2, dim3(64 * kG2Waves), 0, s, nullptr,  \
                          ev1, 0,                                                             \
                          H, p.Lp, B, dc, d, L, words, p.W, part, p.KS)
#define SI_G2(MTV)                                                                              \
    if (g2.y == 1) {                                                                            \
        if (fast) SI_G2F(MTV, true, true); else SI_G2F(MTV, false, true);                       \
    } else {                                                                                    \
        if (fast) SI_G2F(MTV, true, false); else SI_G2F(MTV, false, false);                     \
    }
    switch (p.MT) {
        case 8: SI_G2(8); break;
        case 4: SI_G2(4); break;
        case 2: SI_G2(2); break;
        default: SI_G2(1); break;
    }
#undef SI_G2
#undef SI_G2F
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_reduce_partials(part, p.KS, B, d, y, s);
}

}  // namespace

hipError_t launch_union(const void* x, int64_t B, int64_t d, const int32_t* offsets,
                        const int32_t* idx, int64_t nnz, const void* gate_up_c,
                        const void* down_c, int64_t L, int et, float* y, void* ws, int flags,
                        int num_cu, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
    if (use_tiled(B, L, d))
        return launch_union_tiled(x, B, d, offsets, idx, nnz, gate_up_c, down_c, L, et, y, ws,
                                  flags, num_cu, s, ev0, ev1);
    if (et == 2)
        return launch_union_t<f16_t>(x, B, d, offsets, idx, nnz, gate_up_c, down_c, L, y, ws,
                                     flags, num_cu, s, ev0, ev1);
    return launch_union_t<bf16_t>(x, B, d, offsets, idx, nnz, gate_up_c, down_c, L, y, ws, flags,
                                  num_cu, s, ev0, ev1);
}

}  // namespace si
