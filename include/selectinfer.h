/*
 * selectinfer.h — C ABI of the selective-computation gated FFN on MI355X (gfx950).
 *
 * The method (SelectInfer: selective neuron loading and computation): an FFN layer keeps only
 * a "loaded" subset of its neurons (Selective Loading section), and each token computes only
 * an "active" subset of the loaded neurons (Selective Computation section). Neuron n of a
 * SwiGLU FFN is row n of gate_proj and up_proj and column n of down_proj (LLM Profiler
 * section), so the selective FFN output is
 *
 *     y = sum_{j in active} SiLU(W_gate[j] . x) * (W_up[j] . x) * W_down[:, j].
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Every pointer argument is a DEVICE pointer unless stated otherwise. The caller allocates
 *   and owns all buffers; the library keeps no pointer after a call returns.
 * - Calls are enqueued on `hip_stream` (a hipStream_t, NULL = the null stream) and return
 *   before the work finishes, except where a call is documented as synchronous. Buffers must
 *   stay alive until the enqueued work completes.
 * - Errors that can be seen from the host (NULL pointers, bad sizes, unsupported dtypes,
 *   misaligned pointers, too small a workspace) return a nonzero status and enqueue nothing.
 * - Kernels never read or write out of bounds whatever the CONTENT of index arrays: an out of
 *   range slot id is skipped (contributes nothing), offsets are clamped to [0, nnz].
 *   Index content is validated on the device only under SI_FLAG_CHECK (synchronous).
 * - Matrices are row-major. bf16 values are IEEE bfloat16 bit patterns (2 bytes).
 * - Index spaces: "original ids" are neuron numbers in [0, N); "slots" are positions in a
 *   compacted layer, in [0, L). Slot s holds the loaded neuron with the s-th smallest id.
 * - Results are deterministic: no floating-point atomics are used, every reduction has a
 *   fixed order, and repeated calls with the same inputs give the same bits.
 */
#ifndef SELECTINFER_H
#define SELECTINFER_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* element types: float32, bfloat16, IEEE half (the paper's float16 storage, Memory Footprint
   section) */
typedef enum { SI_F32 = 0, SI_BF16 = 1, SI_F16 = 2 } si_dtype;

typedef enum {
    SI_OK = 0,
    SI_ERR_INVALID = 1,     /* bad argument: NULL pointer, negative size, k > L, misalignment */
    SI_ERR_RANGE = 2,       /* an id, slot or offset outside its range (device check)        */
    SI_ERR_DUPLICATE = 3,   /* an id listed twice where a set is required (device check)     */
    SI_ERR_NOT_LOADED = 4,  /* an original id whose neuron is not in the compacted layer     */
    SI_ERR_UNSUPPORTED = 5, /* dtype or size the kernels do not handle                       */
    SI_ERR_HIP = 6,         /* a HIP runtime call failed                                     */
    SI_ERR_WORKSPACE = 7    /* workspace NULL or smaller than the *_workspace query says     */
} si_status;

/* Ranking keys (the `mode` of si_select_topk and si_dynamic_set) and call flags. The values
   are distinct bits, so a mode and flags can share one int. */
enum {
    SI_TOPK_ABS = 1,        /* rank by |score| (the profiler ranks absolute activations)        */
    SI_TOPK_RAW = 2,        /* rank by the score itself ("descending order" read literally)     */
    SI_FLAG_CHECK = 4,      /* validate index content on the device, synchronise, report       */
    SI_FLAG_SORTED = 8,     /* si_selective_ffn: every token's slot list is strictly ascending
                               (a si_select_topk output); si_select_topk: rows are wanted
                               ascending, which they always are                                 */
    SI_FLAG_PER_TOKEN = 16, /* B > 1: use the per-token path even when the union path applies   */
    SI_FLAG_FAST_H = 32,    /* union path: feed SiLU(g)*u to the second MFMA GEMM as one 16-bit
                               value instead of a hi + lo pair (faster, ~1e-3 rel. err); the
                               default from 128 tokens on (the compute-bound tiled GEMMs)       */
    SI_FLAG_UNION = 64,     /* 2 <= B < 5: use the union path where the dtypes allow it         */
    SI_FLAG_EXACT_H = 128   /* union path from 128 tokens on: feed SiLU(g)*u as the hi + lo
                               pair (about 16 significant bits, twice the second GEMM's MFMA
                               work); below 128 tokens the pair is the default. FAST_H wins   */
};

/* Library version (major * 10000 + minor * 100 + patch). */
int si_version(void);

/* Static string naming a status code. Never NULL. */
const char* si_status_string(int status);

/*
 * Selective loading (Selective Loading section): keep only the loaded neurons of one FFN
 * layer, laid out neuron-major for row gathers.
 *
 *   w_gate, w_up  [N][d]  gate_proj / up_proj weights (PyTorch [out, in] storage), dtype wdt
 *   w_down        [d][N]  down_proj weights, dtype wdt
 *   loaded        [L]     int32 original ids, any order, unique, each in [0, N)
 *   gate_up_c     [L][2][d] out: slot s holds (W_gate[n], W_up[n]) for its neuron n
 *   down_c        [L][d]  out: slot s holds column n of W_down, contiguous
 *   slot_to_orig  [L]     out: ascending original ids
 *   orig_to_slot  [N]     out: slot of each neuron, -1 when not loaded
 *
 * A pure copy: outputs are bit-identical to the inputs' values. Compacted size is 3*d*L*s
 * bytes and the memory left out is 3*d*(N-L)*s bytes (s = element size), per Eq. 2.
 * SYNCHRONOUS: waits for the stream, so that it can report SI_ERR_RANGE (an id outside
 * [0, N)) and SI_ERR_DUPLICATE. On such an error the outputs are unspecified.
 * Requires 1 <= L <= N, d >= 1. Calls that overlap on one device are serialised internally.
 */
int si_compact_ffn(const void* w_gate, const void* w_up, const void* w_down,
                   int64_t N, int64_t d, si_dtype wdt,
                   const int32_t* loaded, int64_t L,
                   void* gate_up_c, void* down_c,
                   int32_t* slot_to_orig, int32_t* orig_to_slot,
                   void* hip_stream);

/*
 * Original ids -> slots (Selective Computation section: only loaded neurons are computed).
 *
 *   orig_to_slot [N] int32 map from si_compact_ffn;  ids [n] int32;  slots [n] int32 out.
 *
 * slots[i] = orig_to_slot[ids[i]], or -1 when ids[i] is outside [0, N) or not loaded.
 * With SI_FLAG_CHECK the call synchronises and returns SI_ERR_RANGE or SI_ERR_NOT_LOADED if
 * any entry maps to -1 (the output is still written). n = 0 is allowed.
 */
int si_remap_ids(const int32_t* orig_to_slot, int64_t N,
                 const int32_t* ids, int64_t n, int32_t* slots,
                 int flags, void* hip_stream);

/*
 * Per-token top-k over loaded neurons (dynamic-neuron selection, Selective Computation
 * section: rank a token's activations over the loaded neurons, descending, keep the top).
 *
 *   scores  [B][L] float32;  out_idx [B][k] int32 out, each row ascending;
 *   mode    SI_TOPK_ABS or SI_TOPK_RAW, optionally with SI_FLAG_SORTED (no effect: rows are
 *           always ascending);
 *   ws      workspace of si_select_topk_workspace(B, L, k) bytes (NULL when that is 0).
 *
 * Row b selects the k slots with the largest key: key = |score| (SI_TOPK_ABS) or score
 * (SI_TOPK_RAW). Equal keys go to the lower index; -0 and +0 are equal; NaN ranks below every
 * number. The selected set is therefore unique. Requires 0 <= k <= L (k > L is
 * SI_ERR_INVALID), L <= 2^24, exactly one ranking key in mode. B = 0 or k = 0 enqueue nothing.
 * The selection runs in one work-group per row with its state in registers and LDS, so the
 * workspace query returns 0 for every size; ws and ws_bytes are checked against it.
 */
size_t si_select_topk_workspace(int64_t B, int64_t L, int64_t k);
int si_select_topk(const float* scores, int64_t B, int64_t L, int64_t k, int mode,
                   int32_t* out_idx, void* ws, size_t ws_bytes, void* hip_stream);

/*
 * Workspace bytes si_selective_ffn needs for these sizes and flags (0 means none needed but a
 * NULL workspace is still accepted only when 0 is returned). The value depends on B, nnz, L,
 * d, the dtypes and flags only.
 */
size_t si_selective_ffn_workspace(int64_t B, int64_t nnz, int64_t L, int64_t d,
                                  si_dtype xdt, si_dtype wdt, int flags);

/*
 * Selective computation (Selective Computation section) of one compacted SwiGLU FFN layer
 * for B tokens:
 *
 *   y[b] = sum_{j in A_b} SiLU(gate_c[j] . x[b]) * (up_c[j] . x[b]) * down_c[j]
 *
 *   x         [B][d]   token activations, dtype xdt: SI_F32, or the weights' type (f32
 *                      weights also take SI_BF16 x)
 *   offsets   [B+1]    int32: token b's active slots are idx[offsets[b] .. offsets[b+1])
 *   idx       [nnz]    int32 slot ids in [0, L), any order, no duplicates within a token
 *   gate_up_c [L][2][d], down_c [L][d]  compacted layer from si_compact_ffn, dtype wdt
 *   y         [B][d]   float32 out
 *   ws                 workspace of at least si_selective_ffn_workspace(...) bytes
 *
 * Accumulation is float32. An empty active set gives y[b] = 0 exactly. Paths:
 *   - per-token (B < 5, fp32 weights or x, or SI_FLAG_PER_TOKEN): a gather-GEMV streams only
 *     the active rows with 16-byte loads and a fused SiLU*up epilogue, then accumulates the
 *     down rows into float32 partial sums that a second kernel adds in a fixed order;
 *   - union (B >= 5, or B >= 2 with SI_FLAG_UNION; x and weights both bf16 or both half): the
 *     union of the B active sets is built on the device and both projections run as MFMA
 *     gather-GEMMs over the union rows, with each token's h masked to its own set; below 128
 *     tokens the union rows are streamed once (bandwidth bound) and h enters the second GEMM
 *     as a 16-bit hi + lo pair (about 16 significant bits for bf16; for half 22 bits, but no
 *     finer than 2^-25 absolute once |h| < 2^-3 and the low half is subnormal); from 128
 *     tokens on the products are LDS-tiled (compute bound) and h enters as one 16-bit value
 *     (about 8 significant bits for bf16, a relative error near 1e-3; SI_FLAG_EXACT_H: the
 *     pair).
 * Requirements: d % 8 == 0 for 16-bit data, d % 4 == 0 for f32; d <= 16384 (16-bit weights)
 * or 8192 (f32 weights), else SI_ERR_UNSUPPORTED; 16-byte aligned x, gate_up_c, down_c, y and
 * ws; B >= 0; nnz >= 0; L >= 1.
 * SI_FLAG_CHECK validates offsets (non-decreasing, within [0, nnz]), slot range and duplicates
 * on the device, synchronises and returns SI_ERR_RANGE / SI_ERR_DUPLICATE before computing;
 * with SI_FLAG_SORTED it also returns SI_ERR_INVALID for a list that is not ascending. Without
 * SI_FLAG_CHECK, SI_FLAG_SORTED is a promise of the caller that the result does not depend on:
 * the sum is the same for any order of a token's list.
 */
int si_selective_ffn(const void* x, si_dtype xdt, int64_t B, int64_t d,
                     const int32_t* offsets, const int32_t* idx, int64_t nnz,
                     const void* gate_up_c, const void* down_c, int64_t L, si_dtype wdt,
                     float* y, void* ws, size_t ws_bytes, int flags, void* hip_stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph capture, serving loops
 * or harnesses that forbid allocation): si_selective_ffn without the workspace arguments. Its
 * kernels take their workspace from a static device array of SI_NOALLOC_SCRATCH_BYTES that the
 * library holds on every device it runs on until the process ends; the call itself allocates
 * nothing. Arguments, results, paths and errors are those of si_selective_ffn, plus
 * SI_ERR_UNSUPPORTED when si_selective_ffn_workspace(...) for the same arguments exceeds
 * SI_NOALLOC_SCRATCH_BYTES. All calls on one device share that array, so calls that overlap in
 * time on one device (on different streams, or from several host threads) race and give
 * undefined results; calls in one stream are ordered and safe. The array keeps the last call's
 * contents: every kernel writes the workspace it reads, so nothing depends on them.
 */
#define SI_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int si_selective_ffn_noalloc(const void* x, si_dtype xdt, int64_t B, int64_t d,
                             const int32_t* offsets, const int32_t* idx, int64_t nnz,
                             const void* gate_up_c, const void* down_c, int64_t L, si_dtype wdt,
                             float* y, int flags, void* hip_stream);

/*
 * Instrumentation: time the main kernel of si_selective_ffn with caller-owned HIP events.
 *
 *   start, stop: hipEvent_t handles (created with timing enabled), or both NULL to stop.
 *
 * The setting belongs to the calling host thread. While set, every si_selective_ffn call from
 * that thread launches its weight-streaming kernels with these events attached to their
 * dispatch (hipExtLaunchKernelGGL): `start` takes the start time of the first of them and
 * `stop` the end time of the last (per-token path: the gather-GEMV kernel; union path: GEMM1
 * through GEMM2), so hipEventElapsedTime(start, stop) is their device time, without queueing
 * or marker overheads. si_dynamic_set and si_profile_scores attach them in the same way to
 * their MFMA activation kernel (bf16 data). Meant for eager timing runs, not for graph capture. Returns
 * SI_ERR_INVALID if exactly one of the two is NULL.
 */
int si_set_timing_events(void* start, void* stop);

/*
 * Memory-system references (measurement only; not part of the method): the read rates the
 * per-token path is compared with. Both load and discard, storing one folded word per thread
 * to `sink` so that the loads cannot be removed; neither computes any part of the FFN.
 *
 * si_ceiling_stream: a contiguous read of buf[0 .. bytes) with 16-byte non-temporal loads,
 *   split into `blocks` work-groups of 512 threads (one contiguous part each).
 *   16 <= bytes < 2^31, 1 <= blocks <= 65535, buf 16-byte aligned; sink [blocks * 512] uint32.
 * si_ceiling_gather: the per-token path's row pattern for one token with k active slots
 *   idx[0 .. k) over a compacted layer: P work-groups of 512 threads take the slots as that
 *   path deals them, and for each batch of 16 rows load every gate and up row, then every down
 *   row (16 bytes per thread per row, non-temporal). Slots outside [0, L) load nothing.
 *   Requires d * s % 16 == 0 (s = element size of wdt), L * 2 * d * s < 2^31, k * P < 2^32,
 *   1 <= P <= 65535; sink [P * 512] uint32.
 * Asynchronous, stream-ordered. Timing events set with si_set_timing_events are attached to
 * their dispatch as to the main kernel of si_selective_ffn.
 */
int si_ceiling_stream(const void* buf, int64_t bytes, int blocks, uint32_t* sink,
                      void* hip_stream);
int si_ceiling_gather(const void* gate_up_c, const void* down_c, int64_t L, int64_t d,
                      si_dtype wdt, const int32_t* idx, int64_t k, int P, uint32_t* sink,
                      void* hip_stream);

/*
 * Layer step of a stacked FFN: x_out[b] = RMSNorm(x[b] + y[b]) with unit gain,
 * r / sqrt(mean(r^2) + eps), computed in float32 and stored in xdt (bf16: round to nearest
 * even). x [B][d] (xdt: SI_F32 or SI_BF16), y [B][d] float32, x_out [B][d] (xdt); x_out may
 * alias x.
 */
int si_residual_rmsnorm(const void* x, si_dtype xdt, const float* y, int64_t B, int64_t d,
                        float eps, void* x_out, void* hip_stream);

/*
 * One layer of a stacked FFN whose input is the previous layer's pair (the per-layer step of
 * an FFN stack fed sequentially; the paper's Selective Computation section for the FFN):
 *
 *   x_out[b] = RMSNorm(x_prev[b] + y_prev[b])   (as si_residual_rmsnorm, unit gain, eps)
 *   y[b]     = the selective FFN of x_out[b]    (as si_selective_ffn, same arguments)
 *
 *   x_prev [B][d] xdt (SI_F32 or SI_BF16), y_prev [B][d] float32: the previous layer's input
 *                 and output
 *   x_out  [B][d] xdt out: this layer's input, kept for the next layer's residual
 *
 * On the per-token path the normalisation runs in the prologue of the gather-GEMV kernel:
 * every work-group of a token computes it for its own columns (the sum of squares is reduced
 * in a fixed order, the same in each work-group) and the token's first work-group stores
 * x_out, so a layer takes one kernel launch less than si_residual_rmsnorm followed by
 * si_selective_ffn. On the union path the two run one after the other. The result equals that
 * pair of calls up to the summation order of the mean square (x_out may differ by one bf16
 * unit where r / rms falls next to a rounding boundary).
 * x_out must not overlap x_prev, y_prev or y; y may alias y_prev. Other requirements, errors
 * and the workspace are those of si_selective_ffn; x_prev, y_prev and x_out 16-byte aligned,
 * eps >= 0.
 */
int si_selective_ffn_resnorm(const void* x_prev, const float* y_prev, float eps, void* x_out,
                             si_dtype xdt, int64_t B, int64_t d,
                             const int32_t* offsets, const int32_t* idx, int64_t nnz,
                             const void* gate_up_c, const void* down_c, int64_t L,
                             si_dtype wdt, float* y, void* ws, size_t ws_bytes, int flags,
                             void* hip_stream);

/*
 * Dynamic-set construction (Selective Computation section) for one prompt of T tokens over a
 * compacted layer:
 *   1. a_t[j] = SiLU(gate_c[j] . x[t]) * (up_c[j] . x[t]) for every loaded slot j (float32);
 *   2. per token, the alpha slots with the largest key, |a_t[j]| (mode SI_TOPK_ABS) or a_t[j]
 *      (SI_TOPK_RAW); equal keys to the lower slot, -0 = +0, NaN last, as in si_select_topk;
 *   3. counts[j] = number of the T per-token lists that hold j;
 *   4. the n_total - n_static slots outside the static set with the largest count (equal
 *      counts to the lower slot), joined with the static slots.
 *
 *   x            [T][d]     prompt activations, dtype xdt
 *   gate_up_c    [L][2][d]  compacted layer, dtype wdt
 *   static_slots [n_static] int32 slots always computed (the base neurons), unique, in [0, L)
 *   out_slots    [n_total]  int32 out: the per-prompt active set, ascending
 *   counts       [L]        int32 out, optional (NULL: kept in the workspace)
 *   ws                      workspace of at least si_dynamic_set_workspace(...) bytes
 *
 * Requires 0 <= alpha <= L, 0 <= n_static <= n_total <= L <= 2^24, T >= 0, d >= 1, 16-byte
 * aligned x and gate_up_c. Static slots out of range are ignored; repeated static slots leave
 * the result shorter than n_total (unspecified tail). Asynchronous, stream-ordered.
 */
size_t si_dynamic_set_workspace(int64_t T, int64_t L, int64_t alpha, int64_t n_total);
int si_dynamic_set(const void* x, si_dtype xdt, int64_t T, int64_t d,
                   const void* gate_up_c, int64_t L, si_dtype wdt,
                   const int32_t* static_slots, int64_t n_static,
                   int64_t alpha, int64_t n_total, int mode,
                   int32_t* out_slots, int32_t* counts,
                   void* ws, size_t ws_bytes, void* hip_stream);

/*
 * Profiler scores (LLM Profiler section, Eq. 1): scores[n] += sum over the T tokens of
 * |a_n(t)|, a_n(t) = SiLU(gate[n] . x[t]) * (up[n] . x[t]), for the N neurons of a full FFN
 * layer held in the compacted layout (si_compact_ffn with every neuron loaded).
 *
 *   x [T][d] (xdt);  gate_up [N][2][d] (wdt);  scores [N] float64, accumulated in place, so
 *   batches of tokens add up (the caller keeps the token count);  ws of at least
 *   si_profile_scores_workspace(...) bytes.
 *
 * Activations are float32; a call's |a| sums are float32 over at most 256 tokens, then added
 * to scores in float64, all in a fixed order (bitwise reproducible). A profile of tens of
 * millions of tokens then keeps the ranking precision of its float64 sums. Requires d >= 1,
 * N >= 1, 16-byte aligned x and gate_up. Asynchronous, stream-ordered.
 */
size_t si_profile_scores_workspace(int64_t T, int64_t N, int64_t d, si_dtype xdt, si_dtype wdt);
int si_profile_scores(const void* x, si_dtype xdt, int64_t T, int64_t d,
                      const void* gate_up, int64_t N, si_dtype wdt,
                      double* scores, void* ws, size_t ws_bytes, void* hip_stream);

/*
 * Merging score files (LLM Profiler section): out[n] = sum over files f of
 * scores[f][n] / tokens[f], files added in order, in float64.
 *
 *   scores [F][N] float64 (device);  tokens [F] int64 token counts, HOST memory, each >= 1
 *   (divided as exact float64 values up to 2^53);  out [N] float64 (device; may not alias
 *   scores).  Requires F >= 1, N >= 1.
 */
int si_merge_scores(const double* scores, const int64_t* tokens, int64_t F, int64_t N,
                    double* out, void* hip_stream);

/*
 * Ranking (LLM Profiler section): order[r] = the neuron with the r-th largest score; equal
 * scores keep the lower index first, -0 = +0, NaN ranks last.
 *
 *   scores [N] float64;  order [N] int32 out.  Requires 1 <= N <= 2^24.
 */
int si_rank_neurons(const double* scores, int64_t N, int32_t* order, void* hip_stream);

/*
 * Loaded-set construction (Selective Loading section): the base neurons are the first n_base
 * entries of the task-specific ranking; secondary neurons follow the model-level ranking, most
 * relevant first, skipping neurons already chosen, until n_loaded neurons in all.
 *
 *   task_rank, model_rank [N] int32, HOST memory: each lists every neuron exactly once, most
 *                             relevant first (si_rank_neurons of merged score files)
 *   loaded     [n_loaded]     int32 out, HOST memory, in the order filled (base first)
 *
 * Host only: no device work. Requires 0 <= n_base <= n_loaded <= N. SI_ERR_INVALID when a
 * ranking is not a permutation of [0, N).
 */
int si_build_loaded_set(const int32_t* task_rank, const int32_t* model_rank, int64_t N,
                        int64_t n_base, int64_t n_loaded, int32_t* loaded);

/*
 * Layer range of selective loading and computation (Evaluation, Table 1: first layer 5, last
 * layer -2, i.e. the last two layers skipped; Memory Footprint section: r_layer is the
 * fraction of layers selected): mask[i] = 1 for the layers first <= i < n_layers + last, 0 for
 * the others, whose FFN stays whole (every neuron loaded and computed).
 *
 *   mask  [n_layers] uint8 out, HOST memory (may be NULL when n_layers = 0)
 *   count (optional)  HOST int64 out: the number of selected layers
 *
 * Host only. SI_ERR_INVALID for n_layers < 0, first < 0, last > 0, or a NULL mask with
 * n_layers > 0. A range that is empty (first >= n_layers + last) selects no layer.
 */
int si_selective_layers(int64_t n_layers, int64_t first, int64_t last, uint8_t* mask,
                        int64_t* count);

/*
 * Selective loading from host memory (Selective Loading section): the same outputs as
 * si_compact_ffn, but the full layer stays in host memory (any host buffer, e.g. a weight file
 * mapped into memory) and only the loaded neurons' slices are read and moved to the device:
 * 3 * d * L * s bytes (Eq. 2's compacted size) instead of 3 * d * N * s.
 *
 *   w_gate, w_up [N][d], w_down [d][N]  HOST memory, dtype wdt (PyTorch [out, in] storage)
 *   loaded       [L]     int32 original ids, HOST memory, any order, unique, in [0, N)
 *   gate_up_c    [L][2][d], down_c [L][d], slot_to_orig [L], orig_to_slot [N]  DEVICE out, as
 *                        for si_compact_ffn (slots in ascending original id)
 *
 * Host threads cut each row of W_down to its loaded columns and gather the gate/up rows into
 * two pinned staging buffers in turn while their copies to the device run on the stream; the
 * cut rows pass through gate_up_c (overwritten afterwards) and a device transpose writes
 * down_c. SYNCHRONOUS: returns after the copies have finished. SI_ERR_RANGE /
 * SI_ERR_DUPLICATE for bad ids (nothing is moved); SI_ERR_UNSUPPORTED when 2 * d * s or
 * L * s exceeds 64 MiB (one staging buffer). Calls are serialised within the process.
 */
int si_load_selected(const void* w_gate, const void* w_up, const void* w_down, int64_t N,
                     int64_t d, si_dtype wdt, const int32_t* loaded, int64_t L,
                     void* gate_up_c, void* down_c, int32_t* slot_to_orig, int32_t* orig_to_slot,
                     void* hip_stream);

#ifdef __cplusplus
}
#endif

#endif /* SELECTINFER_H */
