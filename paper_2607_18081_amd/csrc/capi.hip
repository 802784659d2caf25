// C ABI of the selective-FFN library: argument checks, dispatch to the kernels, status codes.
#include <mutex>

#include "common.h"
#include "launch.h"
#include "selectinfer.h"

namespace {

constexpr int kMaxDevices = 64;

// Per-device status word written by device-side checks. Only synchronous calls use it, under
// g_check_mu, so overlapping checked calls on one device cannot mix their results.
__device__ int si_status_word[2];

std::mutex g_check_mu;
int* g_status_ptr[kMaxDevices] = {};
int g_num_cu[kMaxDevices] = {};

// Workspace of si_selective_ffn_noalloc: a static array that each device holds for the life of
// the process. In host code `scratch` names a host-side stand-in, not device memory: its device
// address comes from hipGetSymbolAddress, once per device, and only that address is used.
__device__ __align__(256) unsigned char scratch[SI_NOALLOC_SCRATCH_BYTES];
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int current_device() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return -1;
    return dev;
}

// caller holds g_check_mu
int* status_word(int dev) {
    if (!g_status_ptr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(si_status_word)) != hipSuccess) return nullptr;
        g_status_ptr[dev] = static_cast<int*>(p);
    }
    return g_status_ptr[dev];
}

// the device address of this device's copy of `scratch` (the device must be current)
void* scratch_ptr(int dev) {
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
        g_scratch_ptr[dev] = p;
    }
    return g_scratch_ptr[dev];
}

int num_cu(int dev) {
    static std::mutex mu;
    std::lock_guard<std::mutex> lk(mu);
    if (!g_num_cu[dev]) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            n <= 0)
            n = 256;
        g_num_cu[dev] = n;
    }
    return g_num_cu[dev];
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int from_hip(hipError_t e) { return e == hipSuccess ? SI_OK : SI_ERR_HIP; }

// Clears the status word, runs `enqueue`, waits, and returns the device's verdict.
template <typename F>
int checked(hipStream_t s, int dev, F enqueue) {
    std::lock_guard<std::mutex> lk(g_check_mu);
    int* w = status_word(dev);
    if (!w) return SI_ERR_HIP;
    if (hipMemsetAsync(w, 0, 2 * sizeof(int), s) != hipSuccess) return SI_ERR_HIP;
    if (enqueue(w) != hipSuccess) return SI_ERR_HIP;
    int host[2] = {0, 0};
    if (hipMemcpyAsync(host, w, sizeof(host), hipMemcpyDeviceToHost, s) != hipSuccess)
        return SI_ERR_HIP;
    if (hipStreamSynchronize(s) != hipSuccess) return SI_ERR_HIP;
    return host[0];
}

// per host thread: events bracketing the main kernel of si_selective_ffn
thread_local hipEvent_t t_ev_start = nullptr;
thread_local hipEvent_t t_ev_stop = nullptr;

bool valid_dtype(int t) { return t == SI_F32 || t == SI_BF16 || t == SI_F16; }

// x and weight types used together: x is float32 or of the weights' type (and f32 weights
// also take bf16 or half x)
bool valid_pair(int xdt, int wdt) {
    return valid_dtype(xdt) && valid_dtype(wdt) && (xdt == SI_F32 || wdt == SI_F32 || xdt == wdt);
}

// The kernels' ranking key from a public mode (exactly one of SI_TOPK_ABS, SI_TOPK_RAW):
// 0 = |score|, 1 = score; -1 for anything else
int topk_key(int mode) {
    if (mode == SI_TOPK_ABS) return 0;
    if (mode == SI_TOPK_RAW) return 1;
    return -1;
}

// Smallest batch that takes the union path by default. Reading the union once costs |U| rows
// instead of nnz >= |U|, but the union path runs four kernels with a fixed cost of about
// 11 000 row reads (measured on the 7B shape: a step is about 28.5 us + 3.6 ns per union row,
// against 8 us + 2.5 ns per active row on the per-token path). With the workloads' overlap
// the two meet between B = 4 (36.5 us per-token, 43.0 us union) and B = 6 (55.0 / 45.8 us).
constexpr int64_t kUnionMinB = 5;

bool use_union(int64_t B, int64_t L, int64_t d, si_dtype xdt, si_dtype wdt, int flags) {
    return B >= 2 && (B >= kUnionMinB || (flags & SI_FLAG_UNION)) && xdt == wdt &&
           (wdt == SI_BF16 || wdt == SI_F16) && !(flags & SI_FLAG_PER_TOKEN) &&
           si::union_supported(B, L, d);
}

// [a, a + na) and [b, b + nb) share a byte
bool overlap(const void* a, int64_t na, const void* b, int64_t nb) {
    const uintptr_t pa = reinterpret_cast<uintptr_t>(a), pb = reinterpret_cast<uintptr_t>(b);
    return pa < pb + (uintptr_t)nb && pb < pa + (uintptr_t)na;
}

// si_selective_ffn, and with rn the same call whose x is first computed from the previous
// layer's pair (si_selective_ffn_resnorm; x then points at rn->x_out)
int selective_ffn(const void* x, si_dtype xdt, int64_t B, int64_t d, const int32_t* offsets,
                  const int32_t* idx, int64_t nnz, const void* gate_up_c, const void* down_c,
                  int64_t L, si_dtype wdt, float* y, void* ws, size_t ws_bytes, int flags,
                  void* hip_stream, const si::ResNormIn* rn) {
    if (B < 0 || d < 1 || L < 1 || nnz < 0) return SI_ERR_INVALID;
    if (!valid_pair(xdt, wdt)) return SI_ERR_UNSUPPORTED;
    if (B > 65535 || nnz > INT32_MAX || L > INT32_MAX) return SI_ERR_UNSUPPORTED;
    if (si::decode_supported(xdt, wdt, d)) return SI_ERR_UNSUPPORTED;
    if (B == 0) return SI_OK;
    if (!x || !offsets || !gate_up_c || !down_c || !y) return SI_ERR_INVALID;
    if (nnz > 0 && !idx) return SI_ERR_INVALID;
    if (!aligned16(x) || !aligned16(gate_up_c) || !aligned16(down_c) || !aligned16(y))
        return SI_ERR_INVALID;
    const size_t need = si_selective_ffn_workspace(B, nnz, L, d, xdt, wdt, flags);
    if (need > 0 && (!ws || ws_bytes < need || !aligned16(ws))) return SI_ERR_WORKSPACE;
    const int dev = current_device();
    if (dev < 0) return SI_ERR_HIP;
    hipStream_t s = static_cast<hipStream_t>(hip_stream);
    if (flags & SI_FLAG_CHECK) {
        if (L > 524288) return SI_ERR_UNSUPPORTED;
        const bool sorted = (flags & SI_FLAG_SORTED) != 0;
        const int st = checked(s, dev, [&](int* err) {
            return si::launch_check_csr(offsets, idx, B, nnz, L, sorted, err, s);
        });
        if (st != SI_OK) return st;
    }
    const int ncu = num_cu(dev);
    if (use_union(B, L, d, xdt, wdt, flags)) {
        // the union kernels take x as is: the normalisation runs as its own kernel first
        if (rn) {
            const hipError_t e = si::launch_residual_rmsnorm(rn->x_prev, xdt, rn->y_prev, B, d,
                                                             rn->eps, rn->x_out, s);
            if (e != hipSuccess) return SI_ERR_HIP;
        }
        return from_hip(si::launch_union(x, B, d, offsets, idx, nnz, gate_up_c, down_c, L, wdt, y,
                                         ws, flags, ncu, s, t_ev_start, t_ev_stop));
    }
    const int P = si::decode_chunks(B, nnz, ncu);
    return from_hip(si::launch_decode(x, xdt, B, d, offsets, idx, nnz, gate_up_c, down_c, L, wdt,
                                      static_cast<float*>(ws), P, y, s, t_ev_start, t_ev_stop,
                                      rn));
}

}  // namespace

extern "C" {

int si_version(void) { return 200; }

const char* si_status_string(int status) {
    switch (status) {
        case SI_OK: return "ok";
        case SI_ERR_INVALID: return "invalid argument";
        case SI_ERR_RANGE: return "id, slot or offset out of range";
        case SI_ERR_DUPLICATE: return "duplicate id";
        case SI_ERR_NOT_LOADED: return "neuron not loaded";
        case SI_ERR_UNSUPPORTED: return "unsupported dtype or size";
        case SI_ERR_HIP: return "HIP runtime error";
        case SI_ERR_WORKSPACE: return "workspace missing or too small";
        default: return "unknown status";
    }
}

int si_compact_ffn(const void* w_gate, const void* w_up, const void* w_down, int64_t N,
                   int64_t d, si_dtype wdt, const int32_t* loaded, int64_t L, void* gate_up_c,
                   void* down_c, int32_t* slot_to_orig, int32_t* orig_to_slot,
                   void* hip_stream) {
    if (!w_gate || !w_up || !w_down || !loaded || !gate_up_c || !down_c || !slot_to_orig ||
        !orig_to_slot)
        return SI_ERR_INVALID;
    if (!valid_dtype(wdt)) return SI_ERR_UNSUPPORTED;
    if (N < 1 || d < 1 || L < 1 || L > N || N > INT32_MAX) return SI_ERR_INVALID;
    const int es = wdt == SI_F32 ? 4 : 2;
    if ((d * es) % 16 != 0) return SI_ERR_UNSUPPORTED;
    if (!aligned16(w_gate) || !aligned16(w_up) || !aligned16(gate_up_c)) return SI_ERR_INVALID;
    const int dev = current_device();
    if (dev < 0) return SI_ERR_HIP;
    hipStream_t s = static_cast<hipStream_t>(hip_stream);
    int st = checked(s, dev, [&](int* err) {
        return si::launch_compact_maps(loaded, L, N, slot_to_orig, orig_to_slot, err, s);
    });
    if (st != SI_OK) return st;
    hipError_t e = si::launch_compact_gather(w_gate, w_up, w_down, N, d, es, slot_to_orig, L,
                                             gate_up_c, down_c, s);
    if (e != hipSuccess) return SI_ERR_HIP;
    return from_hip(hipStreamSynchronize(s));
}

int si_remap_ids(const int32_t* orig_to_slot, int64_t N, const int32_t* ids, int64_t n,
                 int32_t* slots, int flags, void* hip_stream) {
    if (n < 0 || N < 1) return SI_ERR_INVALID;
    if (n == 0) return SI_OK;
    if (!orig_to_slot || !ids || !slots) return SI_ERR_INVALID;
    hipStream_t s = static_cast<hipStream_t>(hip_stream);
    if (flags & SI_FLAG_CHECK) {
        const int dev = current_device();
        if (dev < 0) return SI_ERR_HIP;
        return checked(s, dev, [&](int* err) {
            return si::launch_remap(orig_to_slot, N, ids, n, slots, err, s);
        });
    }
    return from_hip(si::launch_remap(orig_to_slot, N, ids, n, slots, nullptr, s));
}

size_t si_select_topk_workspace(int64_t, int64_t, int64_t) { return 0; }

int si_select_topk(const float* scores, int64_t B, int64_t L, int64_t k, int mode,
                   int32_t* out_idx, void* ws, size_t ws_bytes, void* hip_stream) {
    if (B < 0 || L < 1 || k < 0 || k > L || L > (1 << 24)) return SI_ERR_INVALID;
    const int key = topk_key(mode & ~SI_FLAG_SORTED);
    if (key < 0) return SI_ERR_INVALID;
    if (ws_bytes < si_select_topk_workspace(B, L, k) || (ws_bytes > 0 && !ws))
        return SI_ERR_WORKSPACE;
    if (B == 0 || k == 0) return SI_OK;
    if (!scores || !out_idx) return SI_ERR_INVALID;
    return from_hip(si::launch_topk(scores, B, L, k, key, out_idx,
                                    static_cast<hipStream_t>(hip_stream)));
}

size_t si_selective_ffn_workspace(int64_t B, int64_t nnz, int64_t L, int64_t d, si_dtype xdt,
                                  si_dtype wdt, int flags) {
    if (B <= 0 || d <= 0 || L <= 0 || nnz < 0) return 0;
    const int dev = current_device();
    const int ncu = dev < 0 ? 256 : num_cu(dev);
    if (use_union(B, L, d, xdt, wdt, flags)) return si::union_workspace(B, L, d, ncu, flags);
    return si::decode_workspace(B, nnz, d, ncu);
}

int si_selective_ffn(const void* x, si_dtype xdt, int64_t B, int64_t d, const int32_t* offsets,
                     const int32_t* idx, int64_t nnz, const void* gate_up_c, const void* down_c,
                     int64_t L, si_dtype wdt, float* y, void* ws, size_t ws_bytes, int flags,
                     void* hip_stream) {
    return selective_ffn(x, xdt, B, d, offsets, idx, nnz, gate_up_c, down_c, L, wdt, y, ws,
                         ws_bytes, flags, hip_stream, nullptr);
}

int si_selective_ffn_noalloc(const void* x, si_dtype xdt, int64_t B, int64_t d,
                             const int32_t* offsets, const int32_t* idx, int64_t nnz,
                             const void* gate_up_c, const void* down_c, int64_t L, si_dtype wdt,
                             float* y, int flags, void* hip_stream) {
    if (B < 0 || d < 1 || L < 1 || nnz < 0) return SI_ERR_INVALID;
    if (B == 0) return SI_OK;
    if (si_selective_ffn_workspace(B, nnz, L, d, xdt, wdt, flags) > SI_NOALLOC_SCRATCH_BYTES)
        return SI_ERR_UNSUPPORTED;
    const int dev = current_device();
    if (dev < 0) return SI_ERR_HIP;
    void* ws = scratch_ptr(dev);
    if (!ws) return SI_ERR_HIP;
    return selective_ffn(x, xdt, B, d, offsets, idx, nnz, gate_up_c, down_c, L, wdt, y, ws,
                         SI_NOALLOC_SCRATCH_BYTES, flags, hip_stream, nullptr);
}

int si_selective_ffn_resnorm(const void* x_prev, const float* y_prev, float eps, void* x_out,
                             si_dtype xdt, int64_t B, int64_t d, const int32_t* offsets,
                             const int32_t* idx, int64_t nnz, const void* gate_up_c,
                             const void* down_c, int64_t L, si_dtype wdt, float* y, void* ws,
                             size_t ws_bytes, int flags, void* hip_stream) {
    if (xdt != SI_F32 && xdt != SI_BF16) return SI_ERR_UNSUPPORTED;
    if (!(eps >= 0.0f)) return SI_ERR_INVALID;
    if (B > 0) {
        if (!x_prev || !y_prev || !x_out) return SI_ERR_INVALID;
        if (!aligned16(x_prev) || !aligned16(y_prev) || !aligned16(x_out)) return SI_ERR_INVALID;
        // x_out is written while x_prev and y_prev are read, and before y is
        const int64_t xb = B * d * (xdt == SI_F32 ? 4 : 2);
        if (overlap(x_out, xb, x_prev, xb) || overlap(x_out, xb, y_prev, B * d * 4) ||
            (y && overlap(x_out, xb, y, B * d * 4)))
            return SI_ERR_INVALID;
    }
    const si::ResNormIn rn{x_prev, y_prev, eps, x_out};
    return selective_ffn(x_out, xdt, B, d, offsets, idx, nnz, gate_up_c, down_c, L, wdt, y, ws,
                         ws_bytes, flags, hip_stream, &rn);
}

int si_ceiling_stream(const void* buf, int64_t bytes, int blocks, uint32_t* sink,
                      void* hip_stream) {
    if (!buf || !sink || bytes < 16 || bytes >= ((int64_t)1 << 31) || blocks < 1 ||
        blocks > 65535)
        return SI_ERR_INVALID;
    if (!aligned16(buf)) return SI_ERR_INVALID;
    return from_hip(si::launch_ceiling_stream(buf, bytes, blocks, sink,
                                              static_cast<hipStream_t>(hip_stream), t_ev_start,
                                              t_ev_stop));
}

int si_ceiling_gather(const void* gate_up_c, const void* down_c, int64_t L, int64_t d,
                      si_dtype wdt, const int32_t* idx, int64_t k, int P, uint32_t* sink,
                      void* hip_stream) {
    if (!valid_dtype(wdt)) return SI_ERR_UNSUPPORTED;
    const int64_t rb = d * (wdt == SI_F32 ? 4 : 2);
    if (!gate_up_c || !down_c || !sink || L < 1 || d < 1 || k < 0 || P < 1 || P > 65535)
        return SI_ERR_INVALID;
    if (k > 0 && !idx) return SI_ERR_INVALID;
    if (rb % 16 != 0 || L * 2 * rb >= ((int64_t)1 << 31) || k * P >= ((int64_t)1 << 32))
        return SI_ERR_UNSUPPORTED;
    if (!aligned16(gate_up_c) || !aligned16(down_c)) return SI_ERR_INVALID;
    return from_hip(si::launch_ceiling_gather(gate_up_c, down_c, L, rb, idx, k, P, sink,
                                              static_cast<hipStream_t>(hip_stream), t_ev_start,
                                              t_ev_stop));
}

int si_set_timing_events(void* start, void* stop) {
    if ((start == nullptr) != (stop == nullptr)) return SI_ERR_INVALID;
    t_ev_start = static_cast<hipEvent_t>(start);
    t_ev_stop = static_cast<hipEvent_t>(stop);
    return SI_OK;
}

int si_residual_rmsnorm(const void* x, si_dtype xdt, const float* y, int64_t B, int64_t d,
                        float eps, void* x_out, void* hip_stream) {
    if (B < 0 || d < 1 || !(eps >= 0.0f)) return SI_ERR_INVALID;
    if (xdt != SI_F32 && xdt != SI_BF16) return SI_ERR_UNSUPPORTED;
    if (B == 0) return SI_OK;
    if (!x || !y || !x_out) return SI_ERR_INVALID;
    return from_hip(si::launch_residual_rmsnorm(x, xdt, y, B, d, eps, x_out,
                                                static_cast<hipStream_t>(hip_stream)));
}

size_t si_dynamic_set_workspace(int64_t T, int64_t L, int64_t alpha, int64_t n_total) {
    if (T < 0 || L < 1 || alpha < 0 || n_total < 0) return 0;
    return si::dyn_plan(T, L, alpha, n_total).total;
}

int si_dynamic_set(const void* x, si_dtype xdt, int64_t T, int64_t d, const void* gate_up_c,
                   int64_t L, si_dtype wdt, const int32_t* static_slots, int64_t n_static,
                   int64_t alpha, int64_t n_total, int mode, int32_t* out_slots, int32_t* counts,
                   void* ws, size_t ws_bytes, void* hip_stream) {
    if (T < 0 || d < 1 || L < 1 || L > (1 << 24)) return SI_ERR_INVALID;
    const int key = topk_key(mode);
    if (key < 0) return SI_ERR_INVALID;
    if (alpha < 0 || alpha > L || n_static < 0 || n_static > n_total || n_total > L)
        return SI_ERR_INVALID;
    if (!valid_pair(xdt, wdt)) return SI_ERR_UNSUPPORTED;
    if ((T > 0 && !x) || !gate_up_c || (n_static > 0 && !static_slots)) return SI_ERR_INVALID;
    if (n_total > 0 && !out_slots) return SI_ERR_INVALID;
    if (!aligned16(x) || !aligned16(gate_up_c)) return SI_ERR_INVALID;
    const size_t need = si_dynamic_set_workspace(T, L, alpha, n_total);
    if (!ws || ws_bytes < need || !aligned16(ws)) return SI_ERR_WORKSPACE;
    if (current_device() < 0) return SI_ERR_HIP;
    return from_hip(si::launch_dynamic_set(x, xdt, T, d, gate_up_c, L, wdt, static_slots,
                                           n_static, alpha, n_total, key, out_slots, counts, ws,
                                           static_cast<hipStream_t>(hip_stream), t_ev_start,
                                           t_ev_stop));
}

size_t si_profile_scores_workspace(int64_t T, int64_t N, int64_t d, si_dtype xdt, si_dtype wdt) {
    if (T < 0 || N < 1 || d < 1) return 0;
    return si::score_workspace(T, N, d, xdt, wdt);
}

int si_profile_scores(const void* x, si_dtype xdt, int64_t T, int64_t d, const void* gate_up,
                      int64_t N, si_dtype wdt, double* scores, void* ws, size_t ws_bytes,
                      void* hip_stream) {
    if (T < 0 || d < 1 || N < 1 || N > INT32_MAX) return SI_ERR_INVALID;
    if (!valid_pair(xdt, wdt)) return SI_ERR_UNSUPPORTED;
    if (T == 0) return SI_OK;
    if (!x || !gate_up || !scores) return SI_ERR_INVALID;
    if (!aligned16(x) || !aligned16(gate_up)) return SI_ERR_INVALID;
    const size_t need = si_profile_scores_workspace(T, N, d, xdt, wdt);
    if (!ws || ws_bytes < need || !aligned16(ws)) return SI_ERR_WORKSPACE;
    if (current_device() < 0) return SI_ERR_HIP;
    return from_hip(si::launch_scores(x, xdt, T, d, gate_up, N, wdt, scores, ws,
                                      static_cast<hipStream_t>(hip_stream), t_ev_start,
                                      t_ev_stop));
}

int si_merge_scores(const double* scores, const int64_t* tokens, int64_t F, int64_t N,
                    double* out, void* hip_stream) {
    if (F < 1 || N < 1 || !scores || !tokens || !out) return SI_ERR_INVALID;
    for (int64_t f = 0; f < F; ++f)
        if (tokens[f] < 1 || tokens[f] > ((int64_t)1 << 53)) return SI_ERR_INVALID;
    if (overlap(out, N * 8, scores, F * N * 8)) return SI_ERR_INVALID;
    hipStream_t s = static_cast<hipStream_t>(hip_stream);
    for (int64_t f = 0; f < F; ++f) {
        const hipError_t e =
            si::launch_merge_file(scores + f * N, N, (double)tokens[f], f == 0 ? 1 : 0, out, s);
        if (e != hipSuccess) return from_hip(e);
    }
    return SI_OK;
}

int si_rank_neurons(const double* scores, int64_t N, int32_t* order, void* hip_stream) {
    if (N < 1 || N > (1 << 24) || !scores || !order) return SI_ERR_INVALID;
    return from_hip(si::launch_rank(scores, N, order, static_cast<hipStream_t>(hip_stream)));
}

}  // extern "C"
