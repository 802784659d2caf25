// Host-side launchers of the selective-FFN kernels (one per kernel file).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace si {

// ---- k_decode.hip: per-token path ------------------------------------------------------
// Input of a stacked layer given as the previous layer's pair: x = RMSNorm(x_prev + y_prev),
// unit gain, computed in the prologue of the per-token kernel and stored to x_out (float32 or
// bf16, the type of x).
struct ResNormIn {
    const void* x_prev;
    const float* y_prev;
    float eps;
    void* x_out;
};
// Number of row chunks (work-groups) per token for the per-token path.
int decode_chunks(int64_t B, int64_t nnz, int num_cu);
// 0 if the shape is supported, else nonzero.
int decode_supported(int xdt, int wdt, int64_t d);
// Workspace bytes of the per-token path: B * P float32 partials of d columns (chunked layout).
size_t decode_workspace(int64_t B, int64_t nnz, int64_t d, int num_cu);
// y[b][c] = sum over p of the partials of token b, column c (column-chunked layout of
// common.h), p in fixed order.
hipError_t launch_reduce_partials(const float* partials, int P, int64_t B, int64_t d, float* y,
                                  hipStream_t s);
hipError_t launch_decode(const void* x, int xdt, int64_t B, int64_t d, const int32_t* offsets,
                         const int32_t* idx, int64_t nnz, const void* gate_up_c,
                         const void* down_c, int64_t L, int wdt, float* partials, int P,
                         float* y, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1,
                         const ResNormIn* rn = nullptr);

// ---- k_union.hip: union (MFMA) path -----------------------------------------------------
// sizes the union kernels handle (their buffer loads take 32-bit byte offsets)
bool union_supported(int64_t B, int64_t L, int64_t d);
size_t union_workspace(int64_t B, int64_t L, int64_t d, int num_cu, int flags);
// et: the 16-bit element type of x and the weights (1 = bf16, 2 = IEEE half)
hipError_t launch_union(const void* x, int64_t B, int64_t d, const int32_t* offsets,
                        const int32_t* idx, int64_t nnz, const void* gate_up_c,
                        const void* down_c, int64_t L, int et, float* y, void* ws, int flags,
                        int num_cu, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1);

// one bitmap of L bits per token (W = ceil(L / 32) words): bit s of token b is set iff slot s
// is in the token's active list
hipError_t launch_token_bitmaps(const int32_t* offsets, const int32_t* idx, int64_t nnz,
                                int64_t B, int64_t L, int64_t W, uint32_t* bits, hipStream_t s);

// ---- k_tiled.hip: union path for large batches (LDS-tiled MFMA GEMMs) ----------------------
bool tiled_supported(int64_t B, int64_t L, int64_t d);
size_t tiled_workspace(int64_t B, int64_t L, int64_t d, int num_cu, int flags);
hipError_t launch_union_tiled(const void* x, int64_t B, int64_t d, const int32_t* offsets,
                              const int32_t* idx, int64_t nnz, const void* gate_up_c,
                              const void* down_c, int64_t L, int et, float* y, void* ws,
                              int flags, int num_cu, hipStream_t s, hipEvent_t ev0,
                              hipEvent_t ev1);

// all-slots modes of the tiled GEMM1 (bf16): activations out[t * ldo + j] (score = 0) or one
// Eq. 1 partial row per 256-token tile, out[tile * ldo + j] (score = 1)
hipError_t launch_activations_mfma(const void* x, int64_t T, int64_t d, const void* gate_up_c,
                                   int64_t L, int et, float* out, int64_t ldo, int score,
                                   hipStream_t s, hipEvent_t ev0 = nullptr,
                                   hipEvent_t ev1 = nullptr);
// token tiles of the MFMA activation kernel for T tokens over L slots (one Eq. 1 partial row
// each), and an upper bound over L for sizing a workspace
int activation_tiles(int64_t T, int64_t L);
int activation_tiles_max(int64_t T);
// GEMM1 token tile (256 or 128) for T tokens over L slots on num_cu compute units
int gemm1_tm(int64_t T, int64_t L, int num_cu);
// ascending list of the set bits of bits[0..W) and their number
hipError_t launch_bits_to_list(const uint32_t* bits, int64_t W, int32_t* list, int* count,
                               hipStream_t s);

// ---- k_topk.hip ---------------------------------------------------------------------------
hipError_t launch_topk(const float* scores, int64_t B, int64_t L, int64_t k, int mode,
                       int32_t* out, hipStream_t s);
hipError_t launch_topk_strided(const float* scores, int64_t B, int64_t L, int64_t ld, int64_t k,
                               int mode, int32_t* out, hipStream_t s);
// the same choice as a bitmap per row: bits[b * W + w] bit j set iff slot 32 w + j is taken;
// W = ceil(L / 32) exactly and L <= 32768, else hipErrorInvalidValue; k = 0 clears the rows
hipError_t launch_topk_bitmap(const float* scores, int64_t B, int64_t L, int64_t ld, int64_t k,
                              int mode, uint32_t* bits, int64_t W, hipStream_t s);
// one row of L <= 32768 keys: the ids join_ids[0..n_join) (those in [0, L)) joined with the k
// largest keys among the other slots, in ascending order, at most cap of them -> list, their
// number -> *count. mode 2 takes the keys as unsigned integers.
hipError_t launch_topk_join(const float* scores, int64_t L, int64_t k, int mode,
                            const int32_t* join_ids, int64_t n_join, int32_t* list, int64_t cap,
                            int* count, hipStream_t s);

// ---- k_select.hip: dynamic-set construction and profiler scores ----------------------------
// ev0/ev1 (optional) are attached to the MFMA activation kernel's dispatch when it is used
hipError_t launch_activations(const void* x, int xdt, int64_t T, int64_t d, const void* gate_up_c,
                              int64_t L, int wdt, float* out, int64_t ldo, hipStream_t s,
                              hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr);
size_t score_workspace(int64_t T, int64_t N, int64_t d, int xdt, int wdt);
hipError_t launch_scores(const void* x, int xdt, int64_t T, int64_t d, const void* gate_up,
                         int64_t N, int wdt, double* scores, void* ws, hipStream_t s,
                         hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr);
// up to this many slots the tokens' top-alpha picks travel as bitmaps (the register top-k)
constexpr int64_t kTokenBitsMaxL = 32768;
struct DynPlan {
    int64_t lda, W;
    bool token_bits;
    size_t off_act, off_lists, off_counts, off_keys, off_dyn, off_bits, off_count, total;
};
DynPlan dyn_plan(int64_t T, int64_t L, int64_t alpha, int64_t n_total);
hipError_t launch_dynamic_set(const void* x, int xdt, int64_t T, int64_t d, const void* gate_up_c,
                              int64_t L, int wdt, const int32_t* static_slots, int64_t n_static,
                              int64_t alpha, int64_t n_total, int key, int32_t* out,
                              int32_t* counts_out,
                              void* ws, hipStream_t s, hipEvent_t ev0 = nullptr,
                              hipEvent_t ev1 = nullptr);
hipError_t launch_merge_file(const double* sc, int64_t N, double tokens, int first, double* out,
                             hipStream_t s);
hipError_t launch_rank(const double* sc, int64_t N, int32_t* order, hipStream_t s);

// ---- k_compact.hip ------------------------------------------------------------------------
hipError_t launch_compact_maps(const int32_t* loaded, int64_t L, int64_t N,
                               int32_t* slot_to_orig, int32_t* orig_to_slot, int* err,
                               hipStream_t s);
hipError_t launch_compact_gather(const void* w_gate, const void* w_up, const void* w_down,
                                 int64_t N, int64_t d, int esize, const int32_t* slot_to_orig,
                                 int64_t L, void* gate_up_c, void* down_c, hipStream_t s);
// dst[s][i] = src[i][s]: a [d][L] matrix of esize-byte elements into [L][d]
hipError_t launch_transpose_cols(const void* src, int64_t d, int64_t L, int esize, void* dst,
                                 hipStream_t s);

// ---- k_ceiling.hip: memory-system references (measurement only) ---------------------------
// sink: blocks (or P) * 512 words; ev0/ev1 (optional) stamped by the kernel's dispatch
hipError_t launch_ceiling_stream(const void* buf, int64_t bytes, int blocks, uint32_t* sink,
                                 hipStream_t s, hipEvent_t ev0, hipEvent_t ev1);
hipError_t launch_ceiling_gather(const void* gate_up_c, const void* down_c, int64_t L,
                                 int64_t row_bytes, const int32_t* idx, int64_t k, int P,
                                 uint32_t* sink, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1);

// ---- k_misc.hip ---------------------------------------------------------------------------
hipError_t launch_remap(const int32_t* orig_to_slot, int64_t N, const int32_t* ids, int64_t n,
                        int32_t* slots, int* err, hipStream_t s);
// sorted: also require each token's slots in strictly ascending order (else error 1)
hipError_t launch_check_csr(const int32_t* offsets, const int32_t* idx, int64_t B,
                            int64_t nnz, int64_t L, bool sorted, int* err, hipStream_t s);
hipError_t launch_residual_rmsnorm(const void* x, int xdt, const float* y, int64_t B, int64_t d,
                                   float eps, void* x_out, hipStream_t s);

}  // namespace si
