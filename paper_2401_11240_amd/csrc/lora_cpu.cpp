// CPU LoRA (Section 4.1 "CPU LoRA"; Section 4.2 "Profiling-guided LoRA
// parallelization"): the delta s ((x A) B) of a prompt's rows on host cores,
// the rows split into token slices, one thread per slice.  float32
// arithmetic, AVX2/FMA code paths (every x86-64 server core this library
// targets has them), with 32-column AVX-512F tiles where the host has them
// (the same fused multiply-adds in the same order: the same bits).  The
// factors are widened to float32 once per call, in parallel, B into blocks
// of columns so that a block's rank rows are contiguous.
#include <immintrin.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <condition_variable>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "lora.h"
#include "lora_coldstart.h"

namespace lora {
int set_error(int code, const std::string& msg);
}

namespace {

// C[i][0..32) (+)= sum_k X_i[k] Y[k][0..32) for four rows: the 4 x 32 tile of
// eight 16-wide accumulators (AVX-512F), each sum in k order with fused
// multiply-adds, as the 4 x 16 tile below, so the two give the same bits.
template <bool ACC>
__attribute__((target("avx512f"))) inline void tile4x32(const float* const X[4], const float* Y, int64_t ldy,
                                                        int32_t K, float* const C[4]) {
    __m512 c00, c01, c10, c11, c20, c21, c30, c31;
    if (ACC) {
        c00 = _mm512_loadu_ps(C[0]), c01 = _mm512_loadu_ps(C[0] + 16), c10 = _mm512_loadu_ps(C[1]);
        c11 = _mm512_loadu_ps(C[1] + 16), c20 = _mm512_loadu_ps(C[2]), c21 = _mm512_loadu_ps(C[2] + 16);
        c30 = _mm512_loadu_ps(C[3]), c31 = _mm512_loadu_ps(C[3] + 16);
    } else {
        c00 = c01 = c10 = c11 = c20 = c21 = c30 = c31 = _mm512_setzero_ps();
    }
    for (int32_t k = 0; k < K; ++k) {
        const float* y = Y + (int64_t)k * ldy;
        const __m512 y0 = _mm512_loadu_ps(y), y1 = _mm512_loadu_ps(y + 16);
        __m512 b = _mm512_set1_ps(X[0][k]);
        c00 = _mm512_fmadd_ps(b, y0, c00);
        c01 = _mm512_fmadd_ps(b, y1, c01);
        b = _mm512_set1_ps(X[1][k]);
        c10 = _mm512_fmadd_ps(b, y0, c10);
        c11 = _mm512_fmadd_ps(b, y1, c11);
        b = _mm512_set1_ps(X[2][k]);
        c20 = _mm512_fmadd_ps(b, y0, c20);
        c21 = _mm512_fmadd_ps(b, y1, c21);
        b = _mm512_set1_ps(X[3][k]);
        c30 = _mm512_fmadd_ps(b, y0, c30);
        c31 = _mm512_fmadd_ps(b, y1, c31);
    }
    _mm512_storeu_ps(C[0], c00);
    _mm512_storeu_ps(C[0] + 16, c01);
    _mm512_storeu_ps(C[1], c10);
    _mm512_storeu_ps(C[1] + 16, c11);
    _mm512_storeu_ps(C[2], c20);
    _mm512_storeu_ps(C[2] + 16, c21);
    _mm512_storeu_ps(C[3], c30);
    _mm512_storeu_ps(C[3] + 16, c31);
}

// AVX-512F on this host (decided once)
bool wide_tiles() {
    static const bool on = __builtin_cpu_supports("avx512f");
    return on;
}

}  // namespace

#pragma clang attribute push(__attribute__((target("avx2,fma,f16c"))), apply_to = function)

namespace {

// 16-bit storage to float32, n elements
void widen(const uint16_t* src, float* dst, int64_t n, int32_t dtype) {
    int64_t i = 0;
    if (dtype == LORA_F16) {
        for (; i + 8 <= n; i += 8)
            _mm256_storeu_ps(dst + i, _mm256_cvtph_ps(_mm_loadu_si128((const __m128i*)(src + i))));
        for (; i < n; ++i) dst[i] = _cvtsh_ss(src[i]);
    } else {
        for (; i + 8 <= n; i += 8) {
            const __m256i w = _mm256_cvtepu16_epi32(_mm_loadu_si128((const __m128i*)(src + i)));
            _mm256_storeu_ps(dst + i, _mm256_castsi256_ps(_mm256_slli_epi32(w, 16)));
        }
        for (; i < n; ++i) {
            const uint32_t b = (uint32_t)src[i] << 16;
            std::memcpy(dst + i, &b, 4);
        }
    }
}

struct Job;
typedef void (*TaskFn)(const Job&, int32_t);

struct Job {
    const uint16_t* x;
    int64_t ldx;
    int32_t h_in, h_out, rank, dtype;
    const float* A;        // [h_in, rank]
    const float* B;        // column blocks of B: block b is [rank][nbw] (columns b nbw .., zeros past h_out)
    int32_t nbw;           // columns per block
    float scale;
    float* delta;
    int64_t ld_delta;
    // the pool's work: task(job, i) for i < n_tasks
    TaskFn task;
    int32_t n_tasks, chunk, n_rows;
    // widening of the factors (16-bit input, float32 copies)
    const uint16_t* A16;
    const uint16_t* B16;
    int64_t widen_per_task;
};

// Float buffers kept across calls (each thread its own): fresh pages for
// every call cost more than a short prompt's arithmetic.  A buffer past
// kKeepFloats is given back after the call that needed it (release_big).
constexpr size_t kKeepFloats = (size_t)8 << 20;   // 32 MiB
float* scratch(std::vector<float>& v, size_t n) {
    if (v.size() < n) v.resize(n);
    return v.data();
}
void release_big(std::vector<float>& v) {
    if (v.size() > kKeepFloats) std::vector<float>().swap(v);
}

constexpr int32_t kKChunk = 128;   // rows of A kept in L1 while every row of a slice runs over them

// C[i][0..16) (+)= sum_k X_i[k] Y[k][0..16) for four rows X_0..X_3: a 4 x 16
// register tile of eight 8-wide accumulators, each sum taken in k order with
// fused multiply-adds, started from C (ACC) or from zero
template <bool ACC>
inline void tile4x16(const float* const X[4], const float* Y, int64_t ldy, int32_t K, float* const C[4]) {
    __m256 c00, c01, c10, c11, c20, c21, c30, c31;
    if (ACC) {
        c00 = _mm256_loadu_ps(C[0]), c01 = _mm256_loadu_ps(C[0] + 8), c10 = _mm256_loadu_ps(C[1]);
        c11 = _mm256_loadu_ps(C[1] + 8), c20 = _mm256_loadu_ps(C[2]), c21 = _mm256_loadu_ps(C[2] + 8);
        c30 = _mm256_loadu_ps(C[3]), c31 = _mm256_loadu_ps(C[3] + 8);
    } else {
        c00 = c01 = c10 = c11 = c20 = c21 = c30 = c31 = _mm256_setzero_ps();
    }
    for (int32_t k = 0; k < K; ++k) {
        const float* y = Y + (int64_t)k * ldy;
        const __m256 y0 = _mm256_loadu_ps(y), y1 = _mm256_loadu_ps(y + 8);
        __m256 b = _mm256_broadcast_ss(X[0] + k);
        c00 = _mm256_fmadd_ps(b, y0, c00);
        c01 = _mm256_fmadd_ps(b, y1, c01);
        b = _mm256_broadcast_ss(X[1] + k);
        c10 = _mm256_fmadd_ps(b, y0, c10);
        c11 = _mm256_fmadd_ps(b, y1, c11);
        b = _mm256_broadcast_ss(X[2] + k);
        c20 = _mm256_fmadd_ps(b, y0, c20);
        c21 = _mm256_fmadd_ps(b, y1, c21);
        b = _mm256_broadcast_ss(X[3] + k);
        c30 = _mm256_fmadd_ps(b, y0, c30);
        c31 = _mm256_fmadd_ps(b, y1, c31);
    }
    _mm256_storeu_ps(C[0], c00);
    _mm256_storeu_ps(C[0] + 8, c01);
    _mm256_storeu_ps(C[1], c10);
    _mm256_storeu_ps(C[1] + 8, c11);
    _mm256_storeu_ps(C[2], c20);
    _mm256_storeu_ps(C[2] + 8, c21);
    _mm256_storeu_ps(C[3], c30);
    _mm256_storeu_ps(C[3] + 8, c31);
}

// C[i][0..N) (+)= X_i . Y over k in [0, K) for the rows of a block (nt <= 4;
// missing rows repeat the last one and are not stored); columns past the
// last whole 16 one at a time, in the same k order
template <bool ACC>
void block_product(const float* const X[4], int nt, const float* Y, int64_t ldy, int32_t K, int32_t N,
                   float* const C[4]) {
    float scratch[4][32];
    int32_t n = 0;
    if (wide_tiles())
        for (; n + 32 <= N; n += 32) {
            float* dst[4];
            for (int i = 0; i < 4; ++i) {
                dst[i] = i < nt ? C[i] + n : scratch[i];
                if (ACC && i >= nt) std::memcpy(scratch[i], C[nt - 1] + n, 32 * sizeof(float));
            }
            tile4x32<ACC>(X, Y + n, ldy, K, dst);
        }
    for (; n + 16 <= N; n += 16) {
        float* dst[4];
        for (int i = 0; i < 4; ++i) {
            dst[i] = i < nt ? C[i] + n : scratch[i];
            if (ACC && i >= nt) std::memcpy(scratch[i], C[nt - 1] + n, 16 * sizeof(float));
        }
        tile4x16<ACC>(X, Y + n, ldy, K, dst);
    }
    for (; n < N; ++n)
        for (int i = 0; i < nt; ++i) {
            float c = ACC ? C[i][n] : 0.f;
            for (int32_t k = 0; k < K; ++k) c = std::fma(X[i][k], Y[(int64_t)k * ldy + n], c);
            C[i][n] = c;
        }
}

// rows [t0, t1): v = x[t] . A over chunks of kKChunk rows of A (every row of
// the slice runs over a chunk while it is in L1), then delta[t] = (s v) . B
// one 16-column block of B at a time (the block stays in L1 across the rows)
void run_rows(const Job& J, int32_t t0, int32_t t1) {
    const int32_t R = J.rank, n = t1 - t0;
    static thread_local std::vector<float> xbuf, vbuf;
    float* const xr = scratch(xbuf, (size_t)n * J.h_in);
    float* const vr = scratch(vbuf, (size_t)n * R);
    std::fill(vr, vr + (size_t)n * R, 0.f);
    for (int32_t i = 0; i < n; ++i) widen(J.x + (int64_t)(t0 + i) * J.ldx, xr + (size_t)i * J.h_in, J.h_in, J.dtype);
    auto rows = [&](int32_t tb, int nt, const float* base, size_t ld, int64_t off, const float* P[4]) {
        for (int i = 0; i < 4; ++i) P[i] = base + (size_t)(tb + std::min(i, nt - 1)) * ld + off;
    };
    for (int32_t k0 = 0; k0 < J.h_in; k0 += kKChunk) {
        const int32_t kc = std::min(kKChunk, J.h_in - k0);
        for (int32_t tb = 0; tb < n; tb += 4) {
            const int nt = std::min<int32_t>(4, n - tb);
            const float* X[4];
            rows(tb, nt, xr, J.h_in, k0, X);
            float* V[4];
            for (int i = 0; i < 4; ++i) V[i] = vr + (size_t)(tb + std::min(i, nt - 1)) * R;
            block_product<true>(X, nt, J.A + (int64_t)k0 * R, R, kc, R, V);
        }
    }
    for (size_t i = 0; i < (size_t)n * R; ++i) vr[i] *= J.scale;
    const int32_t nb = J.nbw;                // one block of B at a time (it stays in L1)
    for (int32_t n0 = 0; n0 < J.h_out; n0 += nb) {
        const int32_t nc = std::min<int32_t>(nb, J.h_out - n0);
        for (int32_t tb = 0; tb < n; tb += 4) {
            const int nt = std::min<int32_t>(4, n - tb);
            const float* Vr[4];
            rows(tb, nt, vr, R, 0, Vr);
            float* O[4];
            for (int i = 0; i < 4; ++i) O[i] = J.delta + (int64_t)(t0 + tb + std::min(i, nt - 1)) * J.ld_delta + n0;
            block_product<false>(Vr, nt, J.B + (size_t)(n0 / nb) * R * nb, nb, R, nc, O);
        }
    }
    release_big(xbuf);
    release_big(vbuf);
}

// B's rank rows [k0, k1) into the column blocks
void widen_b_rows(const Job& J, int32_t k0, int32_t k1) {
    const int32_t nbw = J.nbw, nblk = (J.h_out + nbw - 1) / nbw;
    float* const Bp = const_cast<float*>(J.B);
    for (int32_t k = k0; k < k1; ++k)
        for (int32_t b = 0; b < nblk; ++b) {
            const int32_t n0 = b * nbw, nc = std::min(nbw, J.h_out - n0);
            float* dst = Bp + ((size_t)b * J.rank + k) * nbw;
            widen(J.B16 + (int64_t)k * J.h_out + n0, dst, nc, J.dtype);
            for (int32_t j = nc; j < nbw; ++j) dst[j] = 0.f;
        }
}

// pool tasks: slice i of the rows; part i of the factors' widening (the
// first half of the tasks A's elements, the second half B's rank rows)
void rows_task(const Job& J, int32_t i) { run_rows(J, i * J.chunk, std::min(J.n_rows, (i + 1) * J.chunk)); }
void widen_task(const Job& J, int32_t i) {
    const int32_t half = J.n_tasks / 2;
    if (i < half) {
        const int64_t na = (int64_t)J.h_in * J.rank;
        const int64_t lo = i * J.widen_per_task, hi = std::min(na, lo + J.widen_per_task);
        if (lo < hi) widen(J.A16 + lo, const_cast<float*>(J.A) + lo, hi - lo, J.dtype);
    } else {
        const int32_t per = (J.rank + (J.n_tasks - half) - 1) / (J.n_tasks - half);
        const int32_t k0 = (i - half) * per;
        widen_b_rows(J, std::min(k0, J.rank), std::min(J.rank, k0 + per));
    }
}

}  // namespace

#pragma clang attribute pop

namespace {

// Worker threads kept across calls (starting threads costs tens of
// microseconds each, a fair part of a short prompt's layer).  A call posts its
// slices; the workers and the calling thread take them in turn; the call
// returns when every slice is done and no worker is still looking for one, so
// that the next call may rewrite the job.  Calls run one at a time.  The pool
// is never destroyed: its threads wait on it until the process ends.
struct Pool {
    std::mutex call_mu;                 // one call at a time
    std::mutex mu;                      // guards everything below but `next`
    std::condition_variable cv_work, cv_done;
    std::vector<std::thread> workers;
    const Job* job = nullptr;
    std::atomic<int32_t> next{0};
    int32_t done = 0;                   // tasks finished in this run
    int32_t active = 0;                 // workers between taking the job and reporting back
    uint64_t gen = 0;

    // tasks until none is left; returns how many this thread ran
    int32_t drain(const Job& J) {
        int32_t ran = 0;
        for (;;) {
            const int32_t i = next.fetch_add(1);
            if (i >= J.n_tasks) return ran;
            J.task(J, i);
            ++ran;
        }
    }

    void worker() {
        uint64_t seen = 0;
        for (;;) {
            const Job* J;
            {
                std::unique_lock<std::mutex> lk(mu);
                cv_work.wait(lk, [&] { return gen != seen && job != nullptr; });
                seen = gen;
                ++active;
                J = job;
            }
            const int32_t ran = drain(*J);
            std::lock_guard<std::mutex> lk(mu);
            done += ran;
            --active;
            cv_done.notify_all();
        }
    }

    // false when threads cannot be started
    bool ensure(int n) {
        try {
            while ((int)workers.size() < n) workers.emplace_back(&Pool::worker, this);
        } catch (...) {
            return false;
        }
        return true;
    }

    // J's tasks on the workers and the calling thread; returns when every
    // task is done and no worker is still looking for one
    void run(const Job& J) {
        {
            std::unique_lock<std::mutex> lk(mu);
            cv_done.wait(lk, [&] { return active == 0; });
            job = &J;
            next.store(0);
            done = 0;
            ++gen;
        }
        cv_work.notify_all();
        const int32_t ran = drain(J);
        std::unique_lock<std::mutex> lk(mu);
        done += ran;
        cv_done.wait(lk, [&] { return done == J.n_tasks && active == 0; });
        job = nullptr;
    }
};

Pool* pool() {
    static Pool* p = new Pool();
    return p;
}

}  // namespace

extern "C" int lora_cpu_delta(const void* x, int64_t ldx, int32_t n_rows, int32_t h_in, int32_t h_out, int32_t dtype,
                              const void* A, const void* B, int32_t rank, float scale, float* delta, int64_t ld_delta,
                              int32_t tokens_per_thread, int32_t max_threads) {
    if (n_rows < 0 || h_in < 1 || h_out < 1) return lora::set_error(LORA_E_ARG, "lora_cpu_delta: bad sizes");
    if (rank < 1 || rank > 256) return lora::set_error(LORA_E_RANK, "lora_cpu_delta: rank outside [1, 256]");
    if (dtype != LORA_F16 && dtype != LORA_BF16) return lora::set_error(LORA_E_ARG, "lora_cpu_delta: bad dtype");
    if (ldx < h_in || ld_delta < h_out) return lora::set_error(LORA_E_SHAPE, "lora_cpu_delta: ldx or ld_delta too small");
    if (n_rows == 0) return LORA_OK;
    if (!x || !A || !B || !delta) return lora::set_error(LORA_E_ARG, "lora_cpu_delta: NULL argument");
    if (max_threads < 1) max_threads = 1;
    const int32_t nbw = wide_tiles() ? 32 : 16;
    const int64_t na = (int64_t)h_in * rank, nb = (int64_t)rank * ((h_out + nbw - 1) / nbw) * nbw;
    static thread_local std::vector<float> abuf, bbuf;   // the caller's; workers fill them during the call
    float* const Af = scratch(abuf, (size_t)na);
    float* const Bf = scratch(bbuf, (size_t)nb);
    Job J{(const uint16_t*)x, ldx, h_in, h_out, rank, dtype, Af, Bf, nbw, scale, delta, ld_delta,
          nullptr, 0, 0, n_rows, (const uint16_t*)A, (const uint16_t*)B, 0};
    int32_t c = tokens_per_thread > 0 ? tokens_per_thread : (n_rows + max_threads - 1) / max_threads;
    int32_t n_thr = (n_rows + c - 1) / c;
    if (n_thr > max_threads) {
        n_thr = max_threads;
        c = (n_rows + n_thr - 1) / n_thr;
    }
    if (n_thr <= 1) {
        widen((const uint16_t*)A, Af, na, dtype);
        widen_b_rows(J, 0, rank);
        run_rows(J, 0, n_rows);
        release_big(abuf);
        release_big(bbuf);
        return LORA_OK;
    }
    Pool* P = pool();
    std::lock_guard<std::mutex> call(P->call_mu);
    if (!P->ensure(n_thr - 1)) return lora::set_error(LORA_E_NOMEM, "lora_cpu_delta: cannot start threads");
    // the factors widened by every thread, then the row slices
    J.task = widen_task;
    J.n_tasks = 2 * n_thr;
    J.widen_per_task = ((na + n_thr - 1) / n_thr + 7) / 8 * 8;
    P->run(J);
    J.task = rows_task;
    J.n_tasks = (n_rows + c - 1) / c;
    J.chunk = c;
    P->run(J);
    release_big(abuf);
    release_big(bbuf);
    return LORA_OK;
}
