// Union path for large batches (prefill-like): LDS-tiled bf16 MFMA gather-GEMMs over an
// explicit list of the union's slots.
//
// The computation is the one of the union path (Selective Computation section; see
// k_union.hip): with U = A_1 u ... u A_B,
//   H[b][u] = SiLU(x_b . gate_c[U_u]) * (x_b . up_c[U_u]) * [U_u in A_b],   Y = H . down_c[U].
// For many tokens the weights are reused across the batch, so both products are compute
// bound and are tiled for MFMA throughput instead of streamed:
//  - or_blocks / union_scan: the OR of the token bitmaps per block of 64 tokens, then one
//    work-group ORs the blocks and turns the union into the ascending list of its slots;
//  - gemm1_tiled: a work-group computes TM tokens x 80 union slots, K = d in steps of 64,
//    with TM / 32 waves of 32 tokens each. TM = 256 (two waves per SIMD) when that grid fits
//    in one round of work-groups on the CUs; otherwise TM = 128, whose work-groups (46 KB of
//    LDS) run two or three to a CU, so the grid's last round is not a partial one.
//    The 160 weight rows of its tile are ordered per group of 16 slots as 16 gate rows then
//    16 up rows, so gate and up of one (token, slot) land in the same lane and register of two
//    neighbouring MFMA tiles and the SiLU*up*mask epilogue needs no data exchange. Both
//    operands are K-contiguous rows (token rows of x, neuron rows of gate_up_c) staged in LDS
//    with a 160-byte pitch, at which neither the ds_read_b128 of 16 rows nor the staging
//    stores meet bank conflicts.
//    H is written as bf16(h), and with SI_FLAG_EXACT_H also lo = bf16(h - hi) as a second
//    plane.
//  - gemm2_tiled: Y partials for 256 tokens x 128-256 columns over one of KS chunks of the
//    union, K = union position in steps of 64. H rows are K-contiguous; the down rows are
//    staged as row segments and read back transposed into the MFMA B layout with
//    ds_read_b64_tr_b16. Each XCD takes whole (token tile, K chunk) pairs, so the H slice of
//    a pair is fetched into one XCD's L2 only. The products are compute bound, so H enters
//    the MFMA as one 16-bit value (about 8 significant bits of h for bf16) unless
//    SI_FLAG_EXACT_H asks for the hi + lo pair (about 16 bits, twice the MFMA work). The KS
//    partials are added in a fixed order by the shared partial reducer.
// Tiles are loaded with range-checked buffer loads (zeros outside), staged through registers
// while the previous tile is multiplied out of LDS. Where the registers allow (GEMM1 with
// 256-token tiles, GEMM2 with one 16-bit h and up to 160 columns) two or three tiles are in
// flight in rotating register sets, and a step's loads are spread over its MFMAs.
#include <hip/hip_ext.h>

#include <atomic>

#include "common.h"
#include "launch.h"
#include "mfma.h"
#include "selectinfer.h"

namespace si {

namespace {

typedef __attribute__((ext_vector_type(4))) short s16x4_t;

constexpr int kBK = 64;          // K step (elements)
// LDS pitch (bf16) of K-contiguous tiles: 160 bytes. Measured with the hardware's bank-conflict
// counter on the fragment reads (16 rows at one 16-byte column, ds_read_b128) and the staging
// writes: none at 160 bytes (or at 128 with an XOR swizzle), 3.6 cycles per read at 144.
constexpr int kKP = kBK + 16;
constexpr int kT1S = 80;         // GEMM1 union slots per work-group (5 groups of 16)
constexpr int kT1N = 2 * kT1S;   // GEMM1 weight rows per work-group
constexpr int kT2M = 256;        // GEMM2 tokens per work-group (4 waves x 64)
constexpr int kT2T = 512;        // GEMM2 threads per work-group (8 waves, two per SIMD)

// part[c][w] = OR of bits[b][w] over the 64 tokens b of block c. Work-group (wx, c): 64 words
// x 64 tokens; each wave ORs 16 tokens of the 64 words, then the 4 waves meet in LDS.
__global__ __launch_bounds__(256) void or_blocks(const uint32_t* __restrict__ bits, int64_t B,
                                                 int64_t W, uint32_t* __restrict__ part) {
    const int lane = threadIdx.x & 63;
    const int wv = threadIdx.x >> 6;
    const int64_t w = (int64_t)blockIdx.x * 64 + lane;
    const int64_t b0 = (int64_t)blockIdx.y * 64 + 16 * wv;
    // range-checked buffer loads, issued together (a load behind each token's condition made
    // the compiler wait for it before the next)
    const __amdgpu_buffer_rsrc_t rb = make_rsrc(bits, B * W * 4);
    uint32_t v[16];
#pragma unroll
    for (int i = 0; i < 16; ++i)
        v[i] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(
            rb, (w < W && b0 + i < B) ? (int)(((b0 + i) * W + w) * 4) : kOOB, 0, 0);
    uint32_t u = 0u;
#pragma unroll
    for (int i = 0; i < 16; ++i) u |= v[i];
    __shared__ uint32_t red[4][64];
    red[wv][lane] = u;
    __syncthreads();
    if (wv == 0 && w < W) part[(int64_t)blockIdx.y * W + w] = red[0][lane] | red[1][lane] |
                                                               red[2][lane] | red[3][lane];
}

// One work-group: the union of the nb block bitmaps part[0..nb)[W], its set bits in ascending
// order -> ulist, their number -> *ucount. The union words are formed once into LDS (thread t
// takes words t, t + 1024, ...; the block rows of a word are read eight at a time with
// range-checked loads issued together, so a word costs one memory round trip per eight
// blocks). Thread t then owns a contiguous run of words; an exclusive scan of the runs' counts
// (wave scans, then the 16 wave totals) gives each run its first position. Dynamic LDS: W
// words (W <= 16368).
__global__ __launch_bounds__(1024) void union_scan(const uint32_t* __restrict__ part, int64_t nb,
                                                   int64_t W, int32_t* __restrict__ ulist,
                                                   int* __restrict__ ucount) {
    extern __shared__ uint32_t uw[];
    __shared__ int wtot[16];
    const int t = threadIdx.x;
    const int lane = t & 63;
    const int wv = t >> 6;
    const __amdgpu_buffer_rsrc_t rp = make_rsrc(part, nb * W * 4);
    for (int64_t w = t; w < W; w += 1024) {
        uint32_t u = 0u;
        for (int64_t c0 = 0; c0 < nb; c0 += 8) {
            uint32_t v[8];
#pragma unroll
            for (int c = 0; c < 8; ++c)
                v[c] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(
                    rp, c0 + c < nb ? (int)(((c0 + c) * W + w) * 4) : kOOB, 0, 0);
#pragma unroll
            for (int c = 0; c < 8; ++c) u |= v[c];
        }
        uw[w] = u;
    }
    __syncthreads();
    const int64_t per = (W + 1023) / 1024;
    const int64_t w0 = (int64_t)t * per;
    const int64_t w1 = (w0 + per < W) ? w0 + per : W;
    int c = 0;
    for (int64_t w = w0; w < w1; ++w) c += __popc(uw[w]);
    const int incl = wave_incl_scan(c);
    if (lane == kWave - 1) wtot[wv] = incl;
    __syncthreads();
    int before = 0, all = 0;
#pragma unroll
    for (int q = 0; q < 16; ++q) {
        before += q < wv ? wtot[q] : 0;
        all += wtot[q];
    }
    int pos = before + incl - c;
    for (int64_t w = w0; w < w1; ++w) {
        uint32_t u = uw[w];
        while (u) {
            const int j = __ffs(u) - 1;
            ulist[pos++] = (int32_t)(w * 32 + j);
            u &= u - 1u;
        }
    }
    if (t == 0) *ucount = all;
}

// ---- GEMM1 ---------------------------------------------------------------------------------
// Grid: 8 * ntm * ceil(nst / 8) work-groups of 256 threads. Work-groups 8 apart (same XCD)
// share a slot tile, so its weight rows are fetched from HBM once per XCD.
// MODE selects what the epilogue produces (the product itself is the same):
//   kUnion:  h masked by the token bitmaps, over the union list, as bf16 hi/lo planes;
//   kAct:    the activation of every slot (the union list is the identity, no mask), float32
//            out[tok * Up + slot];
//   kScore:  Eq. 1 for this work-group's tokens: sum over its 256 tokens of |a| per slot,
//            added in a fixed order, float32 out[tm * Up + slot] (one partial row per token
//            tile; the host-side reducer adds the rows in order).
enum { kUnion = 0, kAct = 1, kScore = 2 };

template <typename ET, int MODE, int TM>
__global__ __launch_bounds__(2 * TM) void gemm1_tiled(
    const uint16_t* __restrict__ x, int64_t B, int64_t d, const uint16_t* __restrict__ gu, int64_t L,
    const int32_t* __restrict__ ulist, const int* __restrict__ ucount,
    const uint32_t* __restrict__ bits, int64_t W, uint16_t* __restrict__ Hhi,
    uint16_t* __restrict__ Hlo, int64_t Up, int ntm, float* __restrict__ out) {
    const int id = blockIdx.x;
    const int st = (id / (8 * ntm)) * 8 + (id % 8);
    const int tm = (id / 8) % ntm;
    const int nU = MODE == kUnion ? *ucount : (int)L;
    const int64_t u0 = (int64_t)st * kT1S;
    if (u0 >= nU) return;  // uniform
    constexpr int kT1M = TM, kT1W = TM / 32, kT1T = 2 * TM;
    const int64_t m0 = (int64_t)tm * kT1M;
    const int t = threadIdx.x;
    const int lane = t & 63;
    const int w = t >> 6;
    const int nn = lane & 15;
    const int g = lane >> 4;

    __shared__ __align__(16) uint16_t sA[kT1M][kKP];
    __shared__ __align__(16) uint16_t sB[kT1N][kKP];

    // staging: thread t moves 16-byte chunk t % 8 of rows t / 8 + kRP j (weight rows below
    // 160 only)
    constexpr int kRP = kT1T / 8;  // rows per staging pass
    constexpr int kAJ = kT1M / kRP, kBJ = (kT1N + kRP - 1) / kRP;
    const int ch = t & 7;
    const int r0 = t >> 3;
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(x, B * d * 2);
    const __amdgpu_buffer_rsrc_t rg = make_rsrc(gu, L * 2 * d * 2);
    int aoff[kAJ], boff[kBJ];  // byte offset of the row start, or kOOB
#pragma unroll
    for (int j = 0; j < kAJ; ++j) {
        const int64_t tok = m0 + r0 + kRP * j;
        aoff[j] = tok < B ? (int)(tok * d * 2) : kOOB;
    }
    // Union slot ids (the union list in kUnion mode, the union position itself otherwise) are
    // read with range-checked buffer loads, issued together: behind a per-lane condition each
    // load made the compiler wait for it before the next (one memory round trip apiece).
    const __amdgpu_buffer_rsrc_t rul = make_rsrc(ulist, MODE == kUnion ? (int64_t)nU * 4 : 0);
    auto union_slot = [&](int64_t u, bool ok) -> int32_t {
        if constexpr (MODE == kUnion)
            return ok ? (int32_t)__builtin_amdgcn_raw_buffer_load_b32(rul, (int)(u * 4), 0, 0)
                      : -1;
        else
            return ok ? (int32_t)u : -1;
    };
    int32_t bslot[kBJ];
#pragma unroll
    for (int j = 0; j < kBJ; ++j) {
        const int r = r0 + kRP * j;             // weight row of the tile
        const int64_t u = u0 + 16 * (r / 32) + (r % 16);
        bslot[j] = union_slot(u, r < kT1N && u < nU);
    }
#pragma unroll
    for (int j = 0; j < kBJ; ++j) {
        const int plane = ((r0 + kRP * j) % 32) / 16;  // 0 gate, 1 up
        const int32_t slot = bslot[j];
        boff[j] = (slot >= 0 && slot < L) ? (int)(((int64_t)slot * 2 + plane) * d * 2) : kOOB;
    }
    V16 pa0[kAJ], pb0[kBJ], pa1[kAJ], pb1[kBJ], pa2[kAJ], pb2[kBJ];
    auto fetch = [&](int64_t k0, V16(&pa)[kAJ], V16(&pb)[kBJ]) {
        const int64_t k = k0 + 8 * ch;
        const bool kin = k < d;  // d % 8 == 0: a chunk is all in or all out
#pragma unroll
        for (int j = 0; j < kAJ; ++j)
            pa[j] = bload16(rx, (kin && aoff[j] != kOOB) ? aoff[j] + (int)(k * 2) : kOOB);
#pragma unroll
        for (int j = 0; j < kBJ; ++j)
            pb[j] = bload16(rg, (kin && boff[j] != kOOB) ? boff[j] + (int)(k * 2) : kOOB);
    };

    f32x4_t acc[2][10];
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int nj = 0; nj < 10; ++nj) acc[mi][nj] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    // One K step: the staged tile (pa, pb) goes to LDS, the loads of a later tile are issued
    // into the same registers, then the tile is multiplied out of LDS.
    auto step = [&](int64_t k0, V16(&pa)[kAJ], V16(&pb)[kBJ]) {
        __syncthreads();  // the previous tile has been read
#pragma unroll
        for (int j = 0; j < kAJ; ++j) st16(&sA[r0 + kRP * j][8 * ch], pa[j]);
#pragma unroll
        for (int j = 0; j < kBJ; ++j)
            if (r0 + kRP * j < kT1N) st16(&sB[r0 + kRP * j][8 * ch], pb[j]);
        __syncthreads();
        if constexpr (TM == 256) {
            fetch(k0 + 3 * kBK, pa, pb);  // three steps ahead (past the end: reads nothing)
        } else {
            fetch(k0 + kBK, pa, pb);  // one step ahead (past the end: reads nothing)
            // keep the prefetch ahead of the MFMAs (the scheduler would otherwise sink the
            // loads to the end of the step and expose their whole latency at the next LDS store)
            __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            typename Mfma<ET>::vec8 a[2];
#pragma unroll
            for (int mi = 0; mi < 2; ++mi)
                a[mi] = Mfma<ET>::vec(ld16(&sA[32 * w + 16 * mi + nn][32 * ks + 8 * g]));
            // B fragments one ahead: the next one's LDS read is in flight during this one's
            // MFMAs
            typename Mfma<ET>::vec8 bq[2];
            bq[0] = Mfma<ET>::vec(ld16(&sB[nn][32 * ks + 8 * g]));
#pragma unroll
            for (int nj = 0; nj < 10; ++nj) {
                if (nj + 1 < 10)
                    bq[(nj + 1) & 1] = Mfma<ET>::vec(ld16(&sB[16 * (nj + 1) + nn][32 * ks + 8 * g]));
                const typename Mfma<ET>::vec8 b = bq[nj & 1];
#pragma unroll
                for (int mi = 0; mi < 2; ++mi) acc[mi][nj] = Mfma<ET>::mma(a[mi], b, acc[mi][nj]);
            }
        }
        if constexpr (TM == 256) {
            // the loads spread over the step's MFMAs, one after every five
#pragma unroll
            for (int i = 0; i < kAJ + kBJ; ++i) {
                __builtin_amdgcn_sched_group_barrier(0x008, 5, 0);  // MFMA
                __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // vector memory read
            }
        }
    };
    if constexpr (TM == 256) {
        // Three tiles in flight, in rotating register sets: the loads of a tile have three
        // steps to land, and go out spread over the MFMAs rather than in one burst (13B
        // prefill GEMM1 128 -> 124 us with two sets, 111 us with three). The 128-token form,
        // which runs two or three work-groups to a CU, keeps one set: a second set's registers
        // would cost it a work-group per CU.
        const int nks = (int)((d + kBK - 1) / kBK);
        fetch(0, pa0, pb0);
        fetch(kBK, pa1, pb1);
        fetch(2 * kBK, pa2, pb2);
        int ks0 = 0;
        for (; ks0 + 3 <= nks; ks0 += 3) {
            step((int64_t)ks0 * kBK, pa0, pb0);
            step((int64_t)(ks0 + 1) * kBK, pa1, pb1);
            step((int64_t)(ks0 + 2) * kBK, pa2, pb2);
        }
        if (ks0 < nks) step((int64_t)ks0 * kBK, pa0, pb0);
        if (ks0 + 1 < nks) step((int64_t)(ks0 + 1) * kBK, pa1, pb1);
    } else {
        fetch(0, pa0, pb0);
        for (int64_t k0 = 0; k0 < d; k0 += kBK) step(k0, pa0, pb0);
    }

    // epilogue: register i of lane l of tile (mi, nj) is token 32 w + 16 mi + 4 g + i and
    // weight row 16 nj + nn; tiles 2q and 2q + 1 are gate and up of slots u0 + 16 q + nn
    if (MODE == kScore) {
        // |a| summed over this lane's 8 tokens, then over the 4 lane groups (32 tokens of the
        // wave), then over the 8 waves in LDS, each in a fixed order
        __shared__ float ssum[kT1W][kT1S];
#pragma unroll
        for (int q = 0; q < 5; ++q) {
            float v = 0.0f;
#pragma unroll
            for (int mi = 0; mi < 2; ++mi)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int64_t tok = m0 + 32 * w + 16 * mi + 4 * g + i;
                    if (tok < B) v += fabsf(silu_f32(acc[mi][2 * q][i]) * acc[mi][2 * q + 1][i]);
                }
            v += __shfl_xor(v, 16, kWave);
            v += __shfl_xor(v, 32, kWave);
            if (g == 0) ssum[w][16 * q + nn] = v;
        }
        __syncthreads();
        if (t < kT1S && u0 + t < nU) {
            float a = ssum[0][t];
#pragma unroll
            for (int q = 1; q < kT1W; ++q) a += ssum[q][t];
            out[(int64_t)tm * Up + u0 + t] = a;
        }
        return;
    }
    // The lane's 5 slots, then (kUnion) the bitmap word of each of its 8 tokens at each slot:
    // all loads issued together, range-checked (an invalid pair reads nothing, as zero), then
    // used. Loaded under the per-element condition they cost one memory round trip each, 40
    // per work-group at the end of the kernel.
    int32_t eslot[5];
#pragma unroll
    for (int q = 0; q < 5; ++q) {
        const int64_t u = u0 + 16 * q + nn;
        eslot[q] = union_slot(u, u < nU);
    }
    uint32_t tword[5][2][4];
    if constexpr (MODE == kUnion) {
        const __amdgpu_buffer_rsrc_t rbm = make_rsrc(bits, B * W * 4);
#pragma unroll
        for (int q = 0; q < 5; ++q)
#pragma unroll
            for (int mi = 0; mi < 2; ++mi)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int64_t tok = m0 + 32 * w + 16 * mi + 4 * g + i;
                    const int32_t sl = eslot[q];
                    const bool ok = tok < B && sl >= 0 && sl < L;
                    tword[q][mi][i] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(
                        rbm, ok ? (int)((tok * W + sl / 32) * 4) : kOOB, 0, 0);
                }
    }
#pragma unroll
    for (int q = 0; q < 5; ++q) {
        const int64_t u = u0 + 16 * q + nn;
        const int32_t slot = eslot[q];
#pragma unroll
        for (int mi = 0; mi < 2; ++mi)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int64_t tok = m0 + 32 * w + 16 * mi + 4 * g + i;
                if (tok < B && slot >= 0) {
                    if (MODE == kAct) {
                        out[tok * Up + u] = silu_f32(acc[mi][2 * q][i]) * acc[mi][2 * q + 1][i];
                    } else {
                        const bool act = (tword[q][mi][i] >> (slot % 32)) & 1u;
                        const float h =
                            act ? silu_f32(acc[mi][2 * q][i]) * acc[mi][2 * q + 1][i] : 0.0f;
                        const uint32_t hb = Mfma<ET>::rne(h);
                        Hhi[tok * Up + u] = (uint16_t)hb;
                        if (Hlo)  // the lo plane exists only for SI_FLAG_EXACT_H
                            Hlo[tok * Up + u] = (uint16_t)Mfma<ET>::rne(h - Mfma<ET>::widen(hb));
                    }
                }
            }
    }
}

// ---- GEMM2 ---------------------------------------------------------------------------------
// Work-group: 256 tokens x 32 NJ columns over one of KS chunks of the union, 512 threads:
// wave w computes tokens 64 (w / 2) .. and columns 16 NJ (w % 2) .. of the tile. Partials in
// the chunked layout. A (token tile, K chunk) pair is a combo: combo c is token tile c % ntm
// of K chunk c / ntm.
// XCD (xcd = 1): the hardware deals work-groups to the 8 XCDs in turn, so in the grid
// (8, ntn, combos / 8) work-group (x, y, z) runs on XCD x and takes column tile y of combo
// x + 8 z: each XCD takes whole combos, and the H slice of a combo (256 tokens x its chunk) is
// read by the work-groups of one XCD only and stays in that XCD's L2. Otherwise the grid is
// (ntn, combos), column tile fastest.
// The two divisions by run-time sizes use host-computed reciprocals (n / q = mulhi(n, m),
// m = ceil(2^32 / q), exact for n q < 2^32): the compiler lowers an integer division through
// the vector unit, and the K range derived from one sizes a buffer descriptor, which would
// then be a vector value and put every load through it in a loop over the lanes.
// FAST: H enters the MFMA as one 16-bit value (no lo plane, and half the H tile in LDS).
struct G2Grid {
    int KS, ntm, xcd;
    uint32_t ks_m, ntm_m;  // ceil(2^32 / KS), ceil(2^32 / ntm)
};

template <typename ET, int NJ, bool FAST>
__global__ __launch_bounds__(kT2T) void gemm2_tiled(
    const uint16_t* __restrict__ Hhi, const uint16_t* __restrict__ Hlo, int64_t Up, int64_t B,
    const uint16_t* __restrict__ dc, int64_t d, int64_t L, const int32_t* __restrict__ ulist,
    const int* __restrict__ ucount, float* __restrict__ part, G2Grid gg) {
    constexpr int kCols = 32 * NJ;                        // columns per work-group
    // LDS pitch (bf16) of the down tile: padded by 16 except for 160 columns, where the pad
    // put the staging writes into bank conflicts (1.5 cycles per store, none unpadded); the
    // transposing reads cost the same at either pitch
    constexpr int kPitch = kCols + (NJ == 5 ? 0 : 16);
    constexpr int kCpr = kCols / 8;                       // 16-byte chunks per row segment
    constexpr int kDJ = (kBK * kCpr + kT2T - 1) / kT2T;   // staging passes of the down rows
    constexpr int kPlanes = FAST ? 1 : 2;
    // tiles in flight (rotating register sets) as the registers allow: with one 16-bit h,
    // three at 128 columns and two at 160; the hi + lo form and 192 columns keep one set
    constexpr int kSets = !FAST ? 1 : (NJ <= 4 ? 3 : (NJ == 5 ? 2 : 1));
    const int KS = gg.KS;
    const uint32_t combo = gg.xcd ? blockIdx.x + 8 * blockIdx.z : blockIdx.y;
    const uint32_t ct = gg.xcd ? blockIdx.y : blockIdx.x;
    // (a divisor of 1 has no 32-bit reciprocal: taken apart)
    const uint32_t ks = gg.ntm == 1 ? combo : __umulhi(combo, gg.ntm_m);
    const uint32_t tmi = combo - ks * (uint32_t)gg.ntm;
    const int nU = *ucount;
    const uint32_t nk = (uint32_t)(nU + KS - 1);
    const int kper = (int)((KS == 1 ? nk : __umulhi(nk, gg.ks_m)) + kBK - 1) / kBK * kBK;
    const int kb = (int)ks * kper;
    const int ke = kb + kper < nU ? kb + kper : nU;
    const int64_t n0 = (int64_t)ct * kCols;
    const int64_t m0 = (int64_t)tmi * kT2M;
    const int t = threadIdx.x;
    const int lane = t & 63;
    const int w = t >> 6;
    const int wm = w >> 1;  // 0..3
    const int wn = w & 1;
    const int nn = lane & 15;
    const int g = lane >> 4;

    __shared__ __align__(16) uint16_t sH[kPlanes][kT2M][kKP];
    __shared__ __align__(16) uint16_t sD[kBK][kPitch];

    // staging of H: chunk t % 8 of rows t / 8 + 64 j; of the down rows: 16-byte chunk
    // q % kCpr of union position q / kCpr, q = t + 512 j (q past the tile: nothing)
    const int ch = t & 7;
    const int r0 = t >> 3;
    const __amdgpu_buffer_rsrc_t rh = make_rsrc(Hhi, B * Up * 2);
    const __amdgpu_buffer_rsrc_t rl = make_rsrc(Hlo, B * Up * 2);
    const __amdgpu_buffer_rsrc_t rd = make_rsrc(dc, L * d * 2);
    constexpr int kHJ = kT2M / 64;
    int hoff[kHJ];
#pragma unroll
    for (int j = 0; j < kHJ; ++j) {
        const int64_t tok = m0 + r0 + 64 * j;
        hoff[j] = tok < B ? (int)(tok * Up * 2) : kOOB;
    }
    int drow[kDJ], dcol[kDJ];  // staged position and element column; dcol < 0: no chunk
#pragma unroll
    for (int j = 0; j < kDJ; ++j) {
        const int q = t + kT2T * j;
        drow[j] = q / kCpr;
        const int64_t c = n0 + 8 * (q % kCpr);
        dcol[j] = (q < kBK * kCpr && c < d) ? (int)c : -1;  // d % 8 == 0
    }
    V16 ph0[kHJ], pl0[kHJ], pd0[kDJ], ph1[kHJ], pl1[kHJ], pd1[kDJ], ph2[kHJ], pl2[kHJ],
        pd2[kDJ];
    // slot ids of the down rows of the next fetch, loaded one K step ahead of their use so
    // the row loads do not wait on them. The loads are unconditional (a union position past
    // the chunk has an out-of-range offset and reads nothing): validity is applied where the
    // ids are used, so no branch or select makes the compiler wait for them early.
    const __amdgpu_buffer_rsrc_t ru = make_rsrc(ulist, ke * 4);
    int32_t sl[kDJ];
    auto load_slots = [&](int64_t k0) {
#pragma unroll
        for (int j = 0; j < kDJ; ++j) {
            const int64_t u = k0 + drow[j];
            sl[j] = (int32_t)__builtin_amdgcn_raw_buffer_load_b32(
                ru, (u < ke && dcol[j] >= 0) ? (int)(u * 4) : kOOB, 0, 0);
        }
    };
    auto fetch = [&](int64_t k0, V16(&ph)[kHJ], V16(&pl)[kHJ], V16(&pd)[kDJ]) {
        const int64_t k = k0 + 8 * ch;  // 8 union positions of one chunk
        const int64_t nv = ke - k;      // valid positions in the chunk, if below 8
#pragma unroll
        for (int j = 0; j < kHJ; ++j) {
            const int off = (nv > 0 && hoff[j] != kOOB) ? hoff[j] + (int)(k * 2) : kOOB;
            ph[j] = bload16(rh, off);
            if constexpr (!FAST) pl[j] = bload16(rl, off);
        }
#pragma unroll
        for (int j = 0; j < kDJ; ++j) {
            const bool ok = k0 + drow[j] < ke && dcol[j] >= 0 && sl[j] >= 0 && sl[j] < L;
            pd[j] = bload16(rd, ok ? (int)(((int64_t)sl[j] * d + dcol[j]) * 2) : kOOB);
        }
        load_slots(k0 + kBK);
    };

    f32x4_t acc[4][NJ];
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
        for (int nj = 0; nj < NJ; ++nj) acc[mi][nj] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    // One K step: the staged tile goes to LDS, the loads of a later tile are issued into the
    // same registers, then the tile is multiplied out of LDS.
    auto step = [&](int64_t k0, V16(&ph)[kHJ], V16(&pl)[kHJ], V16(&pd)[kDJ]) {
        // H past the chunk's K range is not part of this sum: zero it (branch-free). Applied
        // here, where the tile is stored, and not where it is loaded: there it made the
        // compiler wait for the loads before the step's MFMAs.
        uint32_t keep[4];
        {
            const int64_t nv = ke - (k0 + 8 * ch);
#pragma unroll
            for (int e = 0; e < 4; ++e)
                keep[e] = (2 * e + 1 < nv) ? 0xffffffffu : (2 * e < nv ? 0x0000ffffu : 0u);
        }
        __syncthreads();
#pragma unroll
        for (int j = 0; j < kHJ; ++j) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                ph[j].w[e] &= keep[e];
                if constexpr (!FAST) pl[j].w[e] &= keep[e];
            }
            st16(&sH[0][r0 + 64 * j][8 * ch], ph[j]);
            if constexpr (!FAST) st16(&sH[kPlanes - 1][r0 + 64 * j][8 * ch], pl[j]);
        }
#pragma unroll
        for (int j = 0; j < kDJ; ++j)
            if (dcol[j] >= 0) st16(&sD[drow[j]][dcol[j] - n0], pd[j]);
        __syncthreads();
        if constexpr (kSets > 1) {
            fetch(k0 + kSets * kBK, ph, pl, pd);  // kSets steps ahead (past the chunk: nothing)
        } else {
            fetch(k0 + kBK, ph, pl, pd);  // one step ahead (past the chunk: reads nothing)
            __builtin_amdgcn_sched_barrier(0);  // the prefetch stays ahead of the MFMAs
        }
#pragma unroll
        for (int ks2 = 0; ks2 < 2; ++ks2) {
            // B operand: lane (nn, g) needs union positions 8 g .. 8 g + 7 of column nn of a
            // 16-column subtile; ds_read_b64_tr_b16 hands lane i of a 16-lane group element
            // i % 4 of the 8-byte pieces addressed by lanes i / 4 + 4 j, so lane nn addresses
            // position 8 g + nn / 4 (and + 4), columns 4 (nn % 4) .. + 3 of the subtile.
            typename Mfma<ET>::vec8 bop[NJ];
#pragma unroll
            for (int nj = 0; nj < NJ; ++nj) {
                const int col = 16 * NJ * wn + 16 * nj + 4 * (nn & 3);
                const int row = 32 * ks2 + 8 * g + (nn >> 2);
                const s16x4_t lo4 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (__attribute__((address_space(3))) s16x4_t*)&sD[row][col]);
                const s16x4_t hi4 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (__attribute__((address_space(3))) s16x4_t*)&sD[row + 4][col]);
                const uint32_t p0 = (uint16_t)lo4[0] | ((uint32_t)(uint16_t)lo4[1] << 16);
                const uint32_t p1 = (uint16_t)lo4[2] | ((uint32_t)(uint16_t)lo4[3] << 16);
                const uint32_t p2 = (uint16_t)hi4[0] | ((uint32_t)(uint16_t)hi4[1] << 16);
                const uint32_t p3 = (uint16_t)hi4[2] | ((uint32_t)(uint16_t)hi4[3] << 16);
                bop[nj] = Mfma<ET>::vec(V16{{p0, p1, p2, p3}});
            }
            // A fragments (hi, lo) one row-tile ahead of their MFMAs
            typename Mfma<ET>::vec8 ah[2], al[2];
            ah[0] = Mfma<ET>::vec(ld16(&sH[0][64 * wm + nn][32 * ks2 + 8 * g]));
            if constexpr (!FAST)
                al[0] = Mfma<ET>::vec(ld16(&sH[kPlanes - 1][64 * wm + nn][32 * ks2 + 8 * g]));
#pragma unroll
            for (int mi = 0; mi < 4; ++mi) {
                if (mi + 1 < 4) {
                    const int row = 64 * wm + 16 * (mi + 1) + nn;
                    ah[(mi + 1) & 1] = Mfma<ET>::vec(ld16(&sH[0][row][32 * ks2 + 8 * g]));
                    if constexpr (!FAST)
                        al[(mi + 1) & 1] =
                            Mfma<ET>::vec(ld16(&sH[kPlanes - 1][row][32 * ks2 + 8 * g]));
                }
#pragma unroll
                for (int nj = 0; nj < NJ; ++nj)
                    acc[mi][nj] = Mfma<ET>::mma(ah[mi & 1], bop[nj], acc[mi][nj]);
                if constexpr (!FAST) {
#pragma unroll
                    for (int nj = 0; nj < NJ; ++nj)
                        acc[mi][nj] = Mfma<ET>::mma(al[mi & 1], bop[nj], acc[mi][nj]);
                }
            }
        }
        if constexpr (kSets > 1) {
            // the loads spread over the step's MFMAs
#pragma unroll
            for (int i = 0; i < kHJ + 2 * kDJ; ++i) {
                __builtin_amdgcn_sched_group_barrier(0x008, (8 * NJ) / (kHJ + 2 * kDJ), 0);
                __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
            }
        }
    };
    if (kb < ke) {
        load_slots(kb);
        fetch(kb, ph0, pl0, pd0);
        if constexpr (kSets > 1) fetch(kb + kBK, ph1, pl1, pd1);
        if constexpr (kSets > 2) fetch(kb + 2 * kBK, ph2, pl2, pd2);
    }
    if constexpr (kSets > 1) {
        // kSets tiles in flight, in rotating register sets (as in GEMM1); the steps are
        // counted, and those left over run after the loop
        const int ns = ke > kb ? (ke - kb + kBK - 1) / kBK : 0;
        int s2 = 0;
        for (; s2 + kSets <= ns; s2 += kSets) {
            step(kb + (int64_t)s2 * kBK, ph0, pl0, pd0);
            step(kb + (int64_t)(s2 + 1) * kBK, ph1, pl1, pd1);
            if constexpr (kSets > 2) step(kb + (int64_t)(s2 + 2) * kBK, ph2, pl2, pd2);
        }
        if (s2 < ns) step(kb + (int64_t)s2 * kBK, ph0, pl0, pd0);
        if (kSets > 2 && s2 + 1 < ns) step(kb + (int64_t)(s2 + 1) * kBK, ph1, pl1, pd1);
    } else {
        for (int64_t k0 = kb; k0 < ke; k0 += kBK) step(k0, ph0, pl0, pd0);
    }

    // register i of lane l of tile (mi, nj): token 64 wm + 16 mi + 4 g + i, column
    // 16 NJ wn + 16 nj + nn; the 16 lanes of a row write 64 contiguous bytes
    const int64_t nch = part_chunks(d);
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
        for (int nj = 0; nj < NJ; ++nj)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int64_t tok = m0 + 64 * wm + 16 * mi + 4 * g + i;
                const int64_t col = n0 + 16 * NJ * wn + 16 * nj + nn;
                if (tok < B && col < d) part[part_off(tok, ks, col, KS, nch)] = acc[mi][nj][i];
            }
}

struct TPlan {
    int64_t W, Lp, Up;
    int tm1, ntm1, nst, ntm2, ntn2, KS;  // tm1: GEMM1 token tile (gemm1_tm)
    int nj2;     // GEMM2 column tile: 32 nj2 columns
    int xcd2;    // GEMM2 grid: combos dealt to XCDs (see gemm2_tiled)
    int64_t nb;  // blocks of 64 tokens
    size_t off_bits, off_words, off_ulist, off_count, off_hhi, off_hlo, off_part, total;
};

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

// exact: H as a hi + lo pair (SI_FLAG_EXACT_H), else one 16-bit value (no lo plane)
TPlan make_tplan(int64_t B, int64_t L, int64_t d, int num_cu, bool exact) {
    TPlan p;
    p.W = (L + 31) / 32;
    p.Lp = p.W * 32;
    p.Up = (L + kBK - 1) / kBK * kBK;
    p.tm1 = gemm1_tm(B, L, num_cu);
    p.ntm1 = (int)((B + p.tm1 - 1) / p.tm1);
    p.nst = (int)((L + kT1S - 1) / kT1S);
    p.ntm2 = (int)((B + kT2M - 1) / kT2M);
    // GEMM2 column tile: the narrowest of 128, 160 and 192 columns that splits d into at most
    // 32 tiles (one per CU of an XCD), else 192
    p.nj2 = 4;
    while (p.nj2 < 6 && (d + 32 * p.nj2 - 1) / (32 * p.nj2) > 32) ++p.nj2;
    p.ntn2 = (int)((d + 32 * p.nj2 - 1) / (32 * p.nj2));
    // split K so that the combos (token tile x K chunk) fill the CUs' column tiles in whole
    // rounds: num_cu / ntn2 combos in all
    int64_t ks = num_cu / ((int64_t)p.ntm2 * p.ntn2);
    if (ks < 1) ks = 1;
    const int64_t kmax = (L + kBK - 1) / kBK;
    if (ks > kmax) ks = kmax;
    if (ks > 64) ks = 64;
    p.KS = (int)ks;
    p.xcd2 = (p.ntm2 * p.KS) % 8 == 0 ? 1 : 0;
    size_t o = 0;
    p.off_bits = o;
    o = align256(o + (size_t)B * p.W * 4);
    p.nb = (B + 63) / 64;
    p.off_words = o;
    o = align256(o + (size_t)p.nb * p.W * 4);
    p.off_ulist = o;
    o = align256(o + (size_t)p.Lp * 4);
    p.off_count = o;
    o = align256(o + 4);
    p.off_hhi = o;
    o = align256(o + (size_t)B * p.Up * 2);
    p.off_hlo = o;
    if (exact) o = align256(o + (size_t)B * p.Up * 2);
    p.off_part = o;
    o = align256(o + (size_t)p.KS * B * part_chunks(d) * kChunk * 4);
    p.total = o;
    return p;
}

}  // namespace

hipError_t launch_bits_to_list(const uint32_t* bits, int64_t W, int32_t* list, int* count,
                               hipStream_t s) {
    hipLaunchKernelGGL(union_scan, dim3(1), dim3(1024), (unsigned)(W * 4), s, bits, (int64_t)1, W,
                       list, count);
    return hipGetLastError();
}

// GEMM1 token tile: 256 when the 256-token grid fits in one round on the CUs, else 128
int gemm1_tm(int64_t T, int64_t L, int num_cu) {
    const int64_t nst8 = ((L + kT1S - 1) / kT1S + 7) / 8 * 8;
    return nst8 * ((T + 255) / 256) <= num_cu ? 256 : 128;
}

// compute units of the current device, looked up once per device
int current_cu_count() {
    static std::atomic<int> cache[64] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    int n = cache[dev].load(std::memory_order_relaxed);
    if (n == 0) {
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            n <= 0)
            n = 256;
        cache[dev].store(n, std::memory_order_relaxed);
    }
    return n;
}

int activation_tiles(int64_t T, int64_t L) {
    const int tm = gemm1_tm(T, L, current_cu_count());
    return (int)((T + tm - 1) / tm);
}
int activation_tiles_max(int64_t T) { return (int)((T + 127) / 128); }

bool tiled_supported(int64_t B, int64_t L, int64_t d) {
    const int64_t Up = (L + kBK - 1) / kBK * kBK;
    const int64_t lim = (int64_t)1 << 31;
    // 32-bit buffer offsets; the token bitmaps are built in LDS (at most 64 KB), and the union
    // scan keeps the union words and its 16 wave totals there (W * 4 + 64 <= 64 KB)
    return L * 2 * d * 2 < lim && B * d * 2 < lim && B * Up * 2 < lim && L <= 523776;
}

// The tiled path is compute bound: by default H enters GEMM2 as one 16-bit value (about 8
// significant bits for bf16; GEMM2 then does half the MFMA work); SI_FLAG_EXACT_H asks for the
// hi + lo pair, SI_FLAG_FAST_H for the single value explicitly.
bool tiled_exact_h(int flags) { return (flags & SI_FLAG_EXACT_H) && !(flags & SI_FLAG_FAST_H); }

size_t tiled_workspace(int64_t B, int64_t L, int64_t d, int num_cu, int flags) {
    return make_tplan(B, L, d, num_cu, tiled_exact_h(flags)).total;
}

template <typename ET>
hipError_t launch_union_tiled_t(const void* x, int64_t B, int64_t d, const int32_t* offsets,
                                const int32_t* idx, int64_t nnz, const void* gate_up_c,
                                const void* down_c, int64_t L, float* y, void* ws, int flags,
                                int num_cu, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
    const bool fast = !tiled_exact_h(flags);
    const TPlan p = make_tplan(B, L, d, num_cu, !fast);
    uint8_t* base = static_cast<uint8_t*>(ws);
    uint32_t* bits = reinterpret_cast<uint32_t*>(base + p.off_bits);
    uint32_t* words = reinterpret_cast<uint32_t*>(base + p.off_words);
    int32_t* ulist = reinterpret_cast<int32_t*>(base + p.off_ulist);
    int* ucount = reinterpret_cast<int*>(base + p.off_count);
    uint16_t* hhi = reinterpret_cast<uint16_t*>(base + p.off_hhi);
    uint16_t* hlo = fast ? nullptr : reinterpret_cast<uint16_t*>(base + p.off_hlo);
    float* part = reinterpret_cast<float*>(base + p.off_part);
    const uint16_t* xx = static_cast<const uint16_t*>(x);
    const uint16_t* gu = static_cast<const uint16_t*>(gate_up_c);
    const uint16_t* dc = static_cast<const uint16_t*>(down_c);

    hipError_t e = launch_token_bitmaps(offsets, idx, nnz, B, L, p.W, bits, s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(or_blocks, dim3((unsigned)((p.W + 63) / 64), (unsigned)p.nb), dim3(256), 0,
                       s, bits, B, p.W, words);
    hipLaunchKernelGGL(union_scan, dim3(1), dim3(1024), (unsigned)(p.W * 4), s, words, p.nb, p.W,
                       ulist, ucount);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int nst8 = (p.nst + 7) / 8 * 8;
    if (p.tm1 == 256)
        hipExtLaunchKernelGGL((gemm1_tiled<ET, kUnion, 256>), dim3((unsigned)(nst8 * p.ntm1)),
                              dim3(512), 0, s, ev0, nullptr, 0, xx, B, d, gu, L, ulist, ucount,
                              bits, p.W, hhi, hlo, p.Up, p.ntm1, nullptr);
    else
        hipExtLaunchKernelGGL((gemm1_tiled<ET, kUnion, 128>), dim3((unsigned)(nst8 * p.ntm1)),
                              dim3(256), 0, s, ev0, nullptr, 0, xx, B, d, gu, L, ulist, ucount,
                              bits, p.W, hhi, hlo, p.Up, p.ntm1, nullptr);
    const unsigned ncombo = (unsigned)(p.ntm2 * p.KS);
    const dim3 g2 = p.xcd2 ? dim3(8, (unsigned)p.ntn2, ncombo / 8) : dim3((unsigned)p.ntn2, ncombo);
    G2Grid gg;
    gg.KS = p.KS;
    gg.ntm = p.ntm2;
    gg.xcd = p.xcd2;
    // reciprocals ceil(2^32 / q); q = 1 (2^32) is not used by the kernel
    gg.ks_m = (uint32_t)((((uint64_t)1 << 32) + (uint64_t)p.KS - 1) / (uint64_t)p.KS);
    gg.ntm_m = (uint32_t)((((uint64_t)1 << 32) + (uint64_t)p.ntm2 - 1) / (uint64_t)p.ntm2);
#define SI_G2T(NJ, F)                                                                           \
    hipExtLaunchKernelGGL((gemm2_tiled<ET, NJ, F>), g2, dim3(kT2T), 0, s, nullptr, ev1, 0, hhi,  \
                          hlo, p.Up, B, dc, d, L, ulist, ucount, part, gg)
#define SI_G2NJ(NJ)                                                                             \
    if (fast) SI_G2T(NJ, true); else SI_G2T(NJ, false);
    switch (p.nj2) {
        case 4: SI_G2NJ(4) break;
        case 5: SI_G2NJ(5) break;
        default: SI_G2NJ(6) break;
    }
#undef SI_G2NJ
#undef SI_G2T
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_reduce_partials(part, p.KS, B, d, y, s);
}

template <typename ET>
hipError_t launch_activations_mfma_t(const void* x, int64_t T, int64_t d, const void* gate_up_c,
                                     int64_t L, float* out, int64_t ldo, int score, hipStream_t s,
                                     hipEvent_t ev0, hipEvent_t ev1) {
    if (T == 0 || L == 0) return hipSuccess;
    const int tm = gemm1_tm(T, L, current_cu_count());
    const int ntm = (int)((T + tm - 1) / tm);
    const int nst = (int)((L + kT1S - 1) / kT1S);
    const int nst8 = (nst + 7) / 8 * 8;
    const uint16_t* xx = static_cast<const uint16_t*>(x);
    const uint16_t* gu = static_cast<const uint16_t*>(gate_up_c);
#define SI_ACT_LAUNCH(MODE, TMV)                                                               \
    hipExtLaunchKernelGGL((gemm1_tiled<ET, MODE, TMV>), dim3((unsigned)(nst8 * ntm)),          \
                          dim3(2 * TMV), 0, s, ev0, ev1, 0, xx, T, d, gu, L, nullptr, nullptr,  \
                          nullptr, (int64_t)0, nullptr, nullptr, ldo, ntm, out)
    if (score) {
        if (tm == 256)
            SI_ACT_LAUNCH(kScore, 256);
        else
            SI_ACT_LAUNCH(kScore, 128);
    } else {
        if (tm == 256)
            SI_ACT_LAUNCH(kAct, 256);
        else
            SI_ACT_LAUNCH(kAct, 128);
    }
#undef SI_ACT_LAUNCH
    return hipGetLastError();
}

hipError_t launch_union_tiled(const void* x, int64_t B, int64_t d, const int32_t* offsets,
                              const int32_t* idx, int64_t nnz, const void* gate_up_c,
                              const void* down_c, int64_t L, int et, float* y, void* ws,
                              int flags, int num_cu, hipStream_t s, hipEvent_t ev0,
                              hipEvent_t ev1) {
    if (et == 2)
        return launch_union_tiled_t<f16_t>(x, B, d, offsets, idx, nnz, gate_up_c, down_c, L, y,
                                           ws, flags, num_cu, s, ev0, ev1);
    return launch_union_tiled_t<bf16_t>(x, B, d, offsets, idx, nnz, gate_up_c, down_c, L, y, ws,
                                        flags, num_cu, s, ev0, ev1);
}

hipError_t launch_activations_mfma(const void* x, int64_t T, int64_t d, const void* gate_up_c,
                                   int64_t L, int et, float* out, int64_t ldo, int score,
                                   hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
    if (et == 2)
        return launch_activations_mfma_t<f16_t>(x, T, d, gate_up_c, L, out, ldo, score, s, ev0,
                                                ev1);
    return launch_activations_mfma_t<bf16_t>(x, T, d, gate_up_c, L, out, ldo, score, s, ev0, ev1);
}

}  // namespace si
