// Selective loading from host memory (Selective Loading section): build the loaded set of a
// layer from the profiler's rankings, and move only the loaded neurons' slices of a full FFN
// layer held in host memory (a weight file mapped into memory, or any host buffer) into the
// compacted, neuron-major device layout. The full layer never sits on the device; the bytes
// moved are the compacted size of Eq. 2, 3 * d * L * s.
//
// Host side: a pool of threads gathers the loaded rows of W_gate and W_up and each row of
// W_down cut down to its loaded columns ([d][L], a streaming pass) into two pinned staging
// buffers in turn; each buffer's host-to-device copy runs on the caller's stream while the
// other is being filled. The cut W_down rows pass through the first half of gate_up_c, and a
// device transpose writes down_c from there before that half's gate/up rows overwrite it.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <condition_variable>
#include <functional>
#include <cstring>
#include <mutex>
#include <thread>
#include <vector>

#include "launch.h"
#include "selectinfer.h"

namespace {

constexpr size_t kStage = (size_t)64 << 20;  // bytes per pinned staging buffer
// bytes filled per copy: small enough that the first fill and the last copy, which do not
// overlap anything, stay short; large enough for full-rate copies
constexpr size_t kChunk = (size_t)16 << 20;

struct Staging {
    void* buf[2] = {nullptr, nullptr};
    hipEvent_t done[2] = {nullptr, nullptr};
    bool pending[2] = {false, false};
};

std::mutex g_mu;  // one staging pair per process, one loading call at a time
Staging g_st;

int workers() {
    const unsigned n = std::thread::hardware_concurrency();
    return n == 0 ? 4 : (int)std::min(n, 16u);
}

// Worker threads that live as long as the process: a loading call fills many staging chunks,
// and starting threads for each would cost about as much as filling a small one.
class Pool {
public:
    explicit Pool(int n) : n_(n) {
        for (int i = 0; i < n_; ++i) th_.emplace_back([this, i] { loop(i); });
    }
    ~Pool() {
        {
            std::lock_guard<std::mutex> l(m_);
            stop_ = true;
        }
        cv_.notify_all();
        for (auto& t : th_) t.join();
    }
    int size() const { return n_; }
    // job(i) on every worker i; returns when all have finished
    void run(const std::function<void(int)>& job) {
        std::unique_lock<std::mutex> l(m_);
        job_ = &job;
        left_ = n_;
        ++gen_;
        cv_.notify_all();
        done_.wait(l, [this] { return left_ == 0; });
        job_ = nullptr;
    }

private:
    void loop(int i) {
        int seen = 0;
        for (;;) {
            const std::function<void(int)>* job;
            {
                std::unique_lock<std::mutex> l(m_);
                cv_.wait(l, [&] { return stop_ || gen_ != seen; });
                if (stop_) return;
                seen = gen_;
                job = job_;
            }
            (*job)(i);
            std::lock_guard<std::mutex> l(m_);
            if (--left_ == 0) done_.notify_one();
        }
    }
    int n_;
    std::vector<std::thread> th_;
    std::mutex m_;
    std::condition_variable cv_, done_;
    const std::function<void(int)>* job_ = nullptr;
    int gen_ = 0, left_ = 0;
    bool stop_ = false;
};

Pool& pool() {
    static Pool p(workers());
    return p;
}

// f(lo, hi) on contiguous pieces of [0, n), one per worker
template <class F>
void parallel_for(int64_t n, F f) {
    const int w = pool().size();
    pool().run([&](int i) {
        const int64_t lo = n * i / w, hi = n * (i + 1) / w;
        if (lo < hi) f(lo, hi);
    });
}

hipError_t ensure_staging() {
    for (int b = 0; b < 2; ++b) {
        if (!g_st.buf[b]) {
            hipError_t e = hipHostMalloc(&g_st.buf[b], kStage, hipHostMallocDefault);
            if (e != hipSuccess) return e;
        }
        if (!g_st.done[b]) {
            hipError_t e = hipEventCreateWithFlags(&g_st.done[b], hipEventDisableTiming);
            if (e != hipSuccess) return e;
        }
    }
    return hipSuccess;
}

// wait until staging buffer b's previous copy has finished
hipError_t claim(int b) {
    if (!g_st.pending[b]) return hipSuccess;
    g_st.pending[b] = false;
    return hipEventSynchronize(g_st.done[b]);
}

hipError_t ship(int b, void* dst, size_t bytes, hipStream_t s) {
    hipError_t e = hipMemcpyAsync(dst, g_st.buf[b], bytes, hipMemcpyHostToDevice, s);
    if (e != hipSuccess) return e;
    e = hipEventRecord(g_st.done[b], s);
    g_st.pending[b] = (e == hipSuccess);
    return e;
}

// dst[i - i0][s] = w_down[i][S[s]] for rows i in [i0, i1): each row cut to its loaded columns
template <typename T>
void cut_rows(const T* wd, int64_t N, const int32_t* S, int64_t L, int64_t i0, int64_t i1,
              T* dst) {
    parallel_for(i1 - i0, [&](int64_t a, int64_t z) {
        for (int64_t r = a; r < z; ++r) {
            const T* src = wd + (i0 + r) * N;
            T* o = dst + r * L;
            for (int64_t s = 0; s < L; ++s) o[s] = src[S[s]];
        }
    });
}

}  // namespace

extern "C" {

int si_build_loaded_set(const int32_t* task_rank, const int32_t* model_rank, int64_t N,
                        int64_t n_base, int64_t n_loaded, int32_t* loaded) {
    if (N < 1 || !task_rank || !model_rank || !loaded) return SI_ERR_INVALID;
    if (n_base < 0 || n_loaded < n_base || n_loaded > N) return SI_ERR_INVALID;
    std::vector<uint8_t> seen((size_t)N, 0);
    for (const int32_t* r : {task_rank, model_rank}) {  // each ranking lists every neuron once
        std::fill(seen.begin(), seen.end(), 0);
        for (int64_t i = 0; i < N; ++i) {
            const int32_t v = r[i];
            if (v < 0 || v >= N || seen[v]) return SI_ERR_INVALID;
            seen[v] = 1;
        }
    }
    std::fill(seen.begin(), seen.end(), 0);
    int64_t m = 0;
    for (int64_t i = 0; i < n_base; ++i) {
        loaded[m++] = task_rank[i];
        seen[task_rank[i]] = 1;
    }
    for (int64_t i = 0; i < N && m < n_loaded; ++i) {
        const int32_t v = model_rank[i];
        if (!seen[v]) {
            loaded[m++] = v;
            seen[v] = 1;
        }
    }
    return SI_OK;
}

int si_selective_layers(int64_t n_layers, int64_t first, int64_t last, uint8_t* mask,
                        int64_t* count) {
    if (n_layers < 0 || first < 0 || last > 0 || (n_layers > 0 && !mask)) return SI_ERR_INVALID;
    int64_t c = 0;
    for (int64_t i = 0; i < n_layers; ++i) {
        mask[i] = (i >= first && i < n_layers + last) ? 1 : 0;
        c += mask[i];
    }
    if (count) *count = c;
    return SI_OK;
}

int si_load_selected(const void* w_gate, const void* w_up, const void* w_down, int64_t N,
                     int64_t d, si_dtype wdt, const int32_t* loaded, int64_t L, void* gate_up_c,
                     void* down_c, int32_t* slot_to_orig, int32_t* orig_to_slot,
                     void* hip_stream) {
    if (N < 1 || d < 1 || L < 1 || L > N || N > INT32_MAX) return SI_ERR_INVALID;
    if (wdt != SI_F32 && wdt != SI_BF16 && wdt != SI_F16) return SI_ERR_UNSUPPORTED;
    if (!w_gate || !w_up || !w_down || !loaded || !gate_up_c || !down_c || !slot_to_orig ||
        !orig_to_slot)
        return SI_ERR_INVALID;
    const int64_t es = wdt == SI_F32 ? 4 : 2;
    const size_t row = (size_t)(d * es);
    const size_t lrow = (size_t)(L * es);  // bytes of a W_down row cut to the loaded columns
    if (2 * row > kStage || lrow > kStage) return SI_ERR_UNSUPPORTED;
    // slots in ascending original id; reject ids out of range or repeated
    std::vector<int32_t> S(loaded, loaded + L);
    std::sort(S.begin(), S.end());
    if (S.front() < 0 || S.back() >= N) return SI_ERR_RANGE;
    for (int64_t i = 1; i < L; ++i)
        if (S[i] == S[i - 1]) return SI_ERR_DUPLICATE;
    std::vector<int32_t> o2s((size_t)N, -1);
    for (int64_t s = 0; s < L; ++s) o2s[S[s]] = (int32_t)s;

    std::lock_guard<std::mutex> lock(g_mu);
    hipStream_t st = static_cast<hipStream_t>(hip_stream);
    hipError_t e = ensure_staging();
    int b = 0;
    auto fail = [&](hipError_t err) {
        (void)hipStreamSynchronize(st);
        g_st.pending[0] = g_st.pending[1] = false;
        return err == hipSuccess ? SI_OK : SI_ERR_HIP;
    };
    if (e != hipSuccess) return fail(e);

    // the two maps
    e = hipMemcpyAsync(slot_to_orig, S.data(), (size_t)L * 4, hipMemcpyHostToDevice, st);
    if (e == hipSuccess)
        e = hipMemcpyAsync(orig_to_slot, o2s.data(), (size_t)N * 4, hipMemcpyHostToDevice, st);
    if (e != hipSuccess) return fail(e);

    // gate_up_c[s] = (W_gate[S[s]], W_up[S[s]]) for slots [s_lo, s_hi)
    const char* wg = static_cast<const char*>(w_gate);
    const char* wu = static_cast<const char*>(w_up);
    const int64_t cs_gu = (int64_t)(std::max(kChunk, 2 * row) / (2 * row));
    auto gate_up = [&](int64_t s_lo, int64_t s_hi) -> hipError_t {
        for (int64_t s0 = s_lo; s0 < s_hi; s0 += cs_gu) {
            const int64_t s1 = std::min(s_hi, s0 + cs_gu);
            hipError_t err = claim(b);
            if (err != hipSuccess) return err;
            char* dst = static_cast<char*>(g_st.buf[b]);
            parallel_for(s1 - s0, [&](int64_t a, int64_t z) {
                for (int64_t s = a; s < z; ++s) {
                    const int64_t n = S[s0 + s];
                    std::memcpy(dst + s * 2 * row, wg + n * row, row);
                    std::memcpy(dst + s * 2 * row + row, wu + n * row, row);
                }
            });
            err = ship(b, static_cast<char*>(gate_up_c) + s0 * 2 * row, (s1 - s0) * 2 * row, st);
            if (err != hipSuccess) return err;
            b ^= 1;
        }
        return hipSuccess;
    };
    // The cut W_down rows ([d][L], d * L * es bytes) pass through the first half of gate_up_c;
    // the slots from s_mid on lie past it. Those gate/up rows go first: a plain row copy is the
    // quickest fill, so the first copy to the device starts sooner.
    const int64_t s_mid = (L + 1) / 2;
    if ((e = gate_up(s_mid, L)) != hipSuccess) return fail(e);
    // down_c[s] = column S[s] of W_down: rows cut to the loaded columns, shipped into the
    // first half of gate_up_c, transposed on the device
    char* cut = static_cast<char*>(gate_up_c);
    const int64_t rows_per = (int64_t)(std::max(kChunk, lrow) / lrow);
    for (int64_t i0 = 0; i0 < d; i0 += rows_per) {
        const int64_t i1 = std::min(d, i0 + rows_per);
        if ((e = claim(b)) != hipSuccess) return fail(e);
        if (es == 2)
            cut_rows(static_cast<const uint16_t*>(w_down), N, S.data(), L, i0, i1,
                     static_cast<uint16_t*>(g_st.buf[b]));
        else
            cut_rows(static_cast<const uint32_t*>(w_down), N, S.data(), L, i0, i1,
                     static_cast<uint32_t*>(g_st.buf[b]));
        if ((e = ship(b, cut + i0 * lrow, (i1 - i0) * lrow, st)) != hipSuccess) return fail(e);
        b ^= 1;
    }
    if ((e = si::launch_transpose_cols(cut, d, L, (int)es, down_c, st)) != hipSuccess)
        return fail(e);
    // then the gate/up rows of the first half, over the cut rows (after the transpose, in
    // stream order)
    if ((e = gate_up(0, s_mid)) != hipSuccess) return fail(e);
    // the maps' host vectors and the staging buffers must outlive the copies
    e = hipStreamSynchronize(st);
    g_st.pending[0] = g_st.pending[1] = false;
    return e == hipSuccess ? SI_OK : SI_ERR_HIP;
}

}  // extern "C"
