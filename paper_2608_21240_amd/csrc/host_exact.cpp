// Exact CPU residual for exact-miss slots (Sec. 4.3: the M_cpu part of Eq. 12).
// Expert weights are in the cfg dtype, or MXFP4 blobs (cfg.wfmt), decoded on the fly.
//
// resid[t] = sum_{k in EXACT(t)} g[t][k] * W2_e (silu(W1_e x_t) * (W3_e x_t)),
// computed from host-resident expert weights.  Work is grouped by expert so each
// weight row is read from DRAM once for all tokens that need it:
//   phase 1: tasks of 32 rows of W1/W3 of one expert -> h[slot][i] (fp32)
//   phase 2: tasks of 64 rows of W2 of one expert    -> y[slot][j] (fp32)
//   phase 3: per token, the gate-weighted sum in ascending k.
// Every output element is produced by one task with a fixed summation order, so
// the result is identical for any thread count.  A persistent worker pool runs
// the tasks; one parallel region runs at a time.
#include <algorithm>
#include <atomic>
#include <cmath>
#include <condition_variable>
#include <cstdint>
#include <cstring>
#include <exception>
#include <functional>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include <immintrin.h>

#include "spice_moe.h"

namespace spice {
spice_status_t set_error(spice_status_t st, const char* msg);
spice_status_t validate(const spice_moe_cfg_t* cfg, int32_t T);
}

namespace {

// ---------------------------------------------------------------- worker pool
class Pool {
   public:
    static Pool& get() {
        static Pool p;
        return p;
    }

    // Runs fn(task) for every task in [0, n_tasks) on at most `threads` threads
    // (the caller included).  A task that throws stops the handing out of further tasks;
    // run() returns only after every thread has left fn (which lives in the caller's
    // frame) and then rethrows the first exception on the calling thread.
    void run(int n_tasks, int threads, const std::function<void(int)>& fn) {
        std::lock_guard<std::mutex> region(region_mu_);
        threads = std::max(1, std::min(threads, n_tasks));
        ensure_workers(threads - 1);
        {
            std::lock_guard<std::mutex> lk(mu_);
            fn_ = &fn;
            n_tasks_ = n_tasks;
            next_.store(0);
            helpers_ = threads - 1;
            pending_ = threads - 1;
            error_ = nullptr;
            ++generation_;
        }
        cv_.notify_all();
        work();
        std::exception_ptr err;
        {
            std::unique_lock<std::mutex> lk(mu_);
            done_cv_.wait(lk, [&] { return pending_ == 0; });
            fn_ = nullptr;
            err = error_;
            error_ = nullptr;
        }
        if (err) std::rethrow_exception(err);
    }

    ~Pool() {
        {
            std::lock_guard<std::mutex> lk(mu_);
            stop_ = true;
            ++generation_;
        }
        cv_.notify_all();
        for (auto& t : workers_) t.join();
    }

   private:
    void work() {
        for (;;) {
            const int task = next_.fetch_add(1);
            if (task >= n_tasks_) break;
            try {
                (*fn_)(task);
            } catch (...) {
                std::lock_guard<std::mutex> lk(mu_);
                if (!error_) error_ = std::current_exception();
                next_.store(n_tasks_);  // hand out no further task
            }
        }
    }

    void ensure_workers(int n) {
        while ((int)workers_.size() < n) {
            const int id = (int)workers_.size();
            workers_.emplace_back([this, id] { loop(id); });
        }
    }

    void loop(int id) {
        uint64_t seen = 0;
        for (;;) {
            {
                std::unique_lock<std::mutex> lk(mu_);
                cv_.wait(lk, [&] { return stop_ || generation_ != seen; });
                if (stop_) return;
                seen = generation_;
                if (id >= helpers_) continue;
            }
            work();
            {
                std::lock_guard<std::mutex> lk(mu_);
                --pending_;
            }
            done_cv_.notify_all();
        }
    }

    std::mutex region_mu_, mu_;
    std::condition_variable cv_, done_cv_;
    std::vector<std::thread> workers_;
    const std::function<void(int)>* fn_ = nullptr;
    std::atomic<int> next_{0};
    int n_tasks_ = 0, helpers_ = 0, pending_ = 0;
    uint64_t generation_ = 0;
    bool stop_ = false;
    std::exception_ptr error_;  // first exception of the current region (guarded by mu_)
};

// ------------------------------------------------------------ dot products
// out[j] = sum_i w[i] * xs[j*ld + i] for j < n; w has `len` elements (dtype).
inline float load_w(const void* w, int dtype, size_t i) {
    if (dtype == SPICE_BF16) {
        uint32_t b = (uint32_t)static_cast<const uint16_t*>(w)[i] << 16;
        float f;
        std::memcpy(&f, &b, 4);
        return f;
    }
    return static_cast<const float*>(w)[i];
}

void dots_generic(const void* w, int dtype, size_t len, const float* xs, size_t ld, int n, float* out) {
    for (int j = 0; j < n; ++j) {
        float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        size_t i = 0;
        for (; i + 8 <= len; i += 8)
            for (int q = 0; q < 8; ++q) acc[q] += load_w(w, dtype, i + q) * xs[j * ld + i + q];
        for (; i < len; ++i) acc[0] += load_w(w, dtype, i) * xs[j * ld + i];
        out[j] = ((acc[0] + acc[1]) + (acc[2] + acc[3])) + ((acc[4] + acc[5]) + (acc[6] + acc[7]));
    }
}

__attribute__((target("avx512f,avx512bw,avx512vl,fma"))) inline __m512 load16_avx512(const void* w, int dtype,
                                                                                       size_t i) {
    if (dtype == SPICE_BF16) {
        const __m256i b = _mm256_loadu_si256(reinterpret_cast<const __m256i*>(static_cast<const uint16_t*>(w) + i));
        return _mm512_castsi512_ps(_mm512_slli_epi32(_mm512_cvtepu16_epi32(b), 16));
    }
    return _mm512_loadu_ps(static_cast<const float*>(w) + i);
}

// NT tokens at once, NA independent accumulators per token: each 16-element weight chunk
// is converted once and used NT times, and NA chains hide the FMA latency when NT is small.
template <int NT, int NA>
__attribute__((target("avx512f,avx512bw,avx512vl,fma"))) inline void dots_block_avx512(const void* w, int dtype,
                                                                                         size_t len, const float* xs,
                                                                                         size_t ld, float* out) {
    __m512 acc[NT][NA];
#pragma GCC unroll 8
    for (int q = 0; q < NT; ++q)
#pragma GCC unroll 4
        for (int c = 0; c < NA; ++c) acc[q][c] = _mm512_setzero_ps();
    size_t i = 0;
    for (; i + 16 * NA <= len; i += 16 * NA) {
#pragma GCC unroll 4
        for (int c = 0; c < NA; ++c) {
            const __m512 wv = load16_avx512(w, dtype, i + 16 * c);
#pragma GCC unroll 8
            for (int q = 0; q < NT; ++q)
                acc[q][c] = _mm512_fmadd_ps(wv, _mm512_loadu_ps(xs + (size_t)q * ld + i + 16 * c), acc[q][c]);
        }
    }
    for (; i + 16 <= len; i += 16) {
        const __m512 wv = load16_avx512(w, dtype, i);
#pragma GCC unroll 8
        for (int q = 0; q < NT; ++q) acc[q][0] = _mm512_fmadd_ps(wv, _mm512_loadu_ps(xs + (size_t)q * ld + i), acc[q][0]);
    }
#pragma GCC unroll 8
    for (int q = 0; q < NT; ++q) {
        __m512 t = acc[q][0];
#pragma GCC unroll 4
        for (int c = 1; c < NA; ++c) t = _mm512_add_ps(t, acc[q][c]);
        float sum = _mm512_reduce_add_ps(t);
        for (size_t k = i; k < len; ++k) sum += load_w(w, dtype, k) * xs[(size_t)q * ld + k];
        out[q] = sum;
    }
}

// Tokens in blocks of at most 8; fewer tokens take more accumulators per token.
__attribute__((target("avx512f,avx512bw,avx512vl,fma"))) void dots_avx512(const void* w, int dtype, size_t len,
                                                                            const float* xs, size_t ld, int n,
                                                                            float* out) {
    int j = 0;
    for (; j + 8 <= n; j += 8) dots_block_avx512<8, 1>(w, dtype, len, xs + (size_t)j * ld, ld, out + j);
    const float* x = xs + (size_t)j * ld;
    switch (n - j) {
        case 1: dots_block_avx512<1, 4>(w, dtype, len, x, ld, out + j); break;
        case 2: dots_block_avx512<2, 4>(w, dtype, len, x, ld, out + j); break;
        case 3: dots_block_avx512<3, 2>(w, dtype, len, x, ld, out + j); break;
        case 4: dots_block_avx512<4, 2>(w, dtype, len, x, ld, out + j); break;
        case 5: dots_block_avx512<5, 1>(w, dtype, len, x, ld, out + j); break;
        case 6: dots_block_avx512<6, 1>(w, dtype, len, x, ld, out + j); break;
        case 7: dots_block_avx512<7, 1>(w, dtype, len, x, ld, out + j); break;
        default: break;
    }
}

using DotsFn = void (*)(const void*, int, size_t, const float*, size_t, int, float*);

DotsFn pick_dots() {
    __builtin_cpu_init();
    if (__builtin_cpu_supports("avx512f") && __builtin_cpu_supports("avx512bw")) return dots_avx512;
    return dots_generic;
}

// ---- MXFP4 rows (OCP MX): 32-element blocks of E2M1 codes (low nibble first) and one
// E8M0 scale each.  out[j] = sum_i w[i] * xs[j*ld + i], len a multiple of 32.
const float kE2M1[16] = {0.0f, 0.5f, 1.0f, 1.5f, 2.0f, 3.0f, 4.0f, 6.0f,
                         -0.0f, -0.5f, -1.0f, -1.5f, -2.0f, -3.0f, -4.0f, -6.0f};

// E8M0 scale 2^(s - 127) from its bits: the exponent field for s >= 1, the subnormal 2^-127
// for s = 0, NaN for s = 255.
inline float e8m0(uint8_t s) {
    const uint32_t bits = s == 255 ? 0x7FC00000u : s == 0 ? 0x00400000u : (uint32_t)s << 23;
    float f;
    std::memcpy(&f, &bits, 4);
    return f;
}

void dots_mx_generic(const uint8_t* el, const uint8_t* sc, size_t len, const float* xs, size_t ld, int n,
                     float* out) {
    for (int j = 0; j < n; ++j) {
        float acc = 0.0f;
        for (size_t b = 0; b < len / 32; ++b) {
            const float s = e8m0(sc[b]);
            float blk = 0.0f;
            for (int i = 0; i < 16; ++i) {
                const uint8_t v = el[b * 16 + i];
                blk += kE2M1[v & 15] * xs[j * ld + b * 32 + 2 * i] + kE2M1[v >> 4] * xs[j * ld + b * 32 + 2 * i + 1];
            }
            acc += s * blk;
        }
        out[j] = acc;
    }
}

// NT tokens at once: each 32-element block is decoded once (table permute of the codes,
// with the table times the scale) and used NT times; two blocks per step and one
// accumulator per half block give 4 independent chains per token.
template <int NT>
__attribute__((target("avx512f,avx512bw,avx512vl,fma"))) inline void dots_mx_step(const uint8_t* el, const uint8_t* sc,
                                                                                    size_t blk, const float* xs,
                                                                                    size_t ld, __m512 (&acc)[NT][4],
                                                                                    int c0) {
    const __m512 lut = _mm512_loadu_ps(kE2M1);
    const __m128i low4 = _mm_set1_epi8(0x0F);
    const __m128i bytes = _mm_loadu_si128(reinterpret_cast<const __m128i*>(el + blk * 16));
    const __m128i lo = _mm_and_si128(bytes, low4), hi = _mm_and_si128(_mm_srli_epi16(bytes, 4), low4);
    const __m512 ls = _mm512_mul_ps(lut, _mm512_set1_ps(e8m0(sc[blk])));
    const __m512 w0 = _mm512_permutexvar_ps(_mm512_cvtepu8_epi32(_mm_unpacklo_epi8(lo, hi)), ls);
    const __m512 w1 = _mm512_permutexvar_ps(_mm512_cvtepu8_epi32(_mm_unpackhi_epi8(lo, hi)), ls);
#pragma GCC unroll 8
    for (int q = 0; q < NT; ++q) {
        const float* x = xs + (size_t)q * ld + blk * 32;
        acc[q][c0] = _mm512_fmadd_ps(w0, _mm512_loadu_ps(x), acc[q][c0]);
        acc[q][c0 + 1] = _mm512_fmadd_ps(w1, _mm512_loadu_ps(x + 16), acc[q][c0 + 1]);
    }
}

template <int NT>
__attribute__((target("avx512f,avx512bw,avx512vl,fma"))) inline void dots_mx_block_avx512(
    const uint8_t* el, const uint8_t* sc, size_t len, const float* xs, size_t ld, float* out) {
    __m512 acc[NT][4];
#pragma GCC unroll 8
    for (int q = 0; q < NT; ++q)
#pragma GCC unroll 4
        for (int c = 0; c < 4; ++c) acc[q][c] = _mm512_setzero_ps();
    const size_t nblk = len / 32;
    size_t b = 0;
    for (; b + 2 <= nblk; b += 2) {
        dots_mx_step<NT>(el, sc, b, xs, ld, acc, 0);
        dots_mx_step<NT>(el, sc, b + 1, xs, ld, acc, 2);
    }
    if (b < nblk) dots_mx_step<NT>(el, sc, b, xs, ld, acc, 0);
#pragma GCC unroll 8
    for (int q = 0; q < NT; ++q)
        out[q] = _mm512_reduce_add_ps(
            _mm512_add_ps(_mm512_add_ps(acc[q][0], acc[q][1]), _mm512_add_ps(acc[q][2], acc[q][3])));
}

__attribute__((target("avx512f,avx512bw,avx512vl,fma"))) void dots_mx_avx512(const uint8_t* el, const uint8_t* sc,
                                                                               size_t len, const float* xs,
                                                                               size_t ld, int n, float* out) {
    int j = 0;
    for (; j + 4 <= n; j += 4) dots_mx_block_avx512<4>(el, sc, len, xs + (size_t)j * ld, ld, out + j);
    const float* x = xs + (size_t)j * ld;
    switch (n - j) {
        case 1: dots_mx_block_avx512<1>(el, sc, len, x, ld, out + j); break;
        case 2: dots_mx_block_avx512<2>(el, sc, len, x, ld, out + j); break;
        case 3: dots_mx_block_avx512<3>(el, sc, len, x, ld, out + j); break;
        default: break;
    }
}

using DotsMxFn = void (*)(const uint8_t*, const uint8_t*, size_t, const float*, size_t, int, float*);

DotsMxFn pick_dots_mx() {
    __builtin_cpu_init();
    if (__builtin_cpu_supports("avx512f") && __builtin_cpu_supports("avx512bw")) return dots_mx_avx512;
    return dots_mx_generic;
}

inline float silu(float u) { return u / (1.0f + std::exp(-u)); }

}  // namespace

extern "C" spice_status_t moe_exact_residual_host(const spice_moe_cfg_t* cfg, int32_t T, const void* x_host,
                                                  const int32_t* topk_idx_host, const float* topk_w_host,
                                                  const uint8_t* slot_class_host, const void* const* w13_host,
                                                  const void* const* w2_host, float* resid_host,
                                                  int32_t n_threads) {
    try {
        const spice_status_t st = spice::validate(cfg, T);
        if (st != SPICE_OK) return st;
        const spice_moe_cfg_t& c = *cfg;
        if (T == 0) return SPICE_OK;
        if (!x_host || !topk_idx_host || !topk_w_host || !slot_class_host || !w13_host || !w2_host || !resid_host)
            return spice::set_error(SPICE_ERR_INVALID, "moe_exact_residual_host: a required pointer is NULL");
        const int N = c.n_experts, K = c.top_k, d = c.d, I = c.inter, dt = c.dtype;
        const size_t S = (size_t)T * K;

        // exact slots grouped by expert, ascending slot id inside a group
        std::vector<int> count(N, 0);
        for (size_t s = 0; s < S; ++s) {
            if (slot_class_host[s] > SPICE_CLASS_EXACT_GPU)
                return spice::set_error(SPICE_ERR_INVALID, "moe_exact_residual_host: slot_class out of range");
            if (slot_class_host[s] != SPICE_CLASS_EXACT) continue;
            const int e = topk_idx_host[s];
            if (e < 0 || e >= N) return spice::set_error(SPICE_ERR_INVALID, "moe_exact_residual_host: expert id out of range");
            if (!w13_host[e] || !w2_host[e])
                return spice::set_error(SPICE_ERR_INVALID, "moe_exact_residual_host: weights of an exact-miss expert are NULL");
            ++count[e];
        }
        std::vector<int> experts, first(N + 1, 0);
        for (int e = 0; e < N; ++e) {
            first[e + 1] = first[e] + count[e];
            if (count[e]) experts.push_back(e);
        }
        const int n_exact = first[N];
        std::vector<int> slot_of(n_exact), fill(N, 0), local_of(S, -1);
        for (size_t s = 0; s < S; ++s) {
            if (slot_class_host[s] != SPICE_CLASS_EXACT) continue;
            const int e = topk_idx_host[s];
            const int li = first[e] + fill[e]++;
            slot_of[li] = (int)s;
            local_of[s] = li;
        }

        int threads = n_threads > 0 ? n_threads : (int)std::max(1u, std::thread::hardware_concurrency());
        static const DotsFn dots = pick_dots();
        static const DotsMxFn dots_mx = pick_dots_mx();
        const bool mx = c.wfmt == SPICE_WFMT_MXFP4;
        Pool& pool = Pool::get();

        // x rows of the exact slots, widened to fp32 (one row per slot)
        std::vector<float> xs((size_t)n_exact * d), h((size_t)n_exact * I), y((size_t)n_exact * d);
        for (int li = 0; li < n_exact; ++li) {
            const size_t t = (size_t)slot_of[li] / K;
            for (int i = 0; i < d; ++i) xs[(size_t)li * d + i] = load_w(x_host, dt, t * d + i);
        }

        constexpr int kRows1 = 32, kRows2 = 64;
        const int nb1 = (I + kRows1 - 1) / kRows1, nb2 = (d + kRows2 - 1) / kRows2;
        const size_t es = dt == SPICE_BF16 ? 2 : 4;
        const int ne = (int)experts.size();

        pool.run(ne * nb1, threads, [&](int task) {
            const int e = experts[task / nb1], rb = task % nb1;
            const int n = count[e], base = first[e];
            const char* w13 = static_cast<const char*>(w13_host[e]);
            // MXFP4 blob of [2I][d]: codes, then the scales
            const uint8_t* el = reinterpret_cast<const uint8_t*>(w13);
            const uint8_t* sc = el + (size_t)2 * I * (d / 2);
            std::vector<float> gv(n), uv(n);
            for (int i = rb * kRows1; i < std::min(I, (rb + 1) * kRows1); ++i) {
                if (mx) {
                    dots_mx(el + (size_t)i * (d / 2), sc + (size_t)i * (d / 32), d, &xs[(size_t)base * d], d, n,
                            gv.data());
                    dots_mx(el + (size_t)(I + i) * (d / 2), sc + (size_t)(I + i) * (d / 32), d,
                            &xs[(size_t)base * d], d, n, uv.data());
                } else {
                    dots(w13 + (size_t)i * d * es, dt, d, &xs[(size_t)base * d], d, n, gv.data());
                    dots(w13 + (size_t)(I + i) * d * es, dt, d, &xs[(size_t)base * d], d, n, uv.data());
                }
                for (int j = 0; j < n; ++j) h[(size_t)(base + j) * I + i] = silu(gv[j]) * uv[j];
            }
        });
        pool.run(ne * nb2, threads, [&](int task) {
            const int e = experts[task / nb2], rb = task % nb2;
            const int n = count[e], base = first[e];
            const char* w2 = static_cast<const char*>(w2_host[e]);
            const uint8_t* el = reinterpret_cast<const uint8_t*>(w2);  // MXFP4 blob of [d][I]
            const uint8_t* sc = el + (size_t)d * (I / 2);
            std::vector<float> ov(n);
            for (int j = rb * kRows2; j < std::min(d, (rb + 1) * kRows2); ++j) {
                if (mx)
                    dots_mx(el + (size_t)j * (I / 2), sc + (size_t)j * (I / 32), I, &h[(size_t)base * I], I, n,
                            ov.data());
                else
                    dots(w2 + (size_t)j * I * es, dt, I, &h[(size_t)base * I], I, n, ov.data());
                for (int q = 0; q < n; ++q) y[(size_t)(base + q) * d + j] = ov[q];
            }
        });
        pool.run(T, threads, [&](int t) {
            float* r = resid_host + (size_t)t * d;
            std::fill(r, r + d, 0.0f);
            for (int k = 0; k < K; ++k) {
                const size_t s = (size_t)t * K + k;
                if (local_of[s] < 0) continue;
                const float g = topk_w_host[s];
                const float* ys = &y[(size_t)local_of[s] * d];
                for (int j = 0; j < d; ++j) r[j] += g * ys[j];
            }
        });
        return SPICE_OK;
    } catch (const std::exception& ex) {
        return spice::set_error(SPICE_ERR_INTERNAL, ex.what());
    } catch (...) {
        return spice::set_error(SPICE_ERR_INTERNAL, "unknown exception");
    }
}
