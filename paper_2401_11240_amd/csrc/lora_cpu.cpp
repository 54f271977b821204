// CPU LoRA (Section 4.1 "CPU LoRA"; Section 4.2 "Profiling-guided LoRA
// parallelization"): the delta s ((x A) B) of a prompt's rows on host cores,
// the rows split into token slices, one thread per slice.  float32
// arithmetic, AVX2/FMA code paths (every x86-64 server core this library
// targets has them).
#include <immintrin.h>

#include <algorithm>
#include <cstdint>
#include <cstring>
#include <string>
#include <thread>
#include <vector>

#include "lora.h"
#include "lora_coldstart.h"

namespace lora {
int set_error(int code, const std::string& msg);
}

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

struct Job {
    const uint16_t* x;
    int64_t ldx;
    int32_t h_in, h_out, rank, dtype;
    const float* A;        // [h_in, rank]
    const float* B;        // [rank, h_out]
    float scale;
    float* delta;
    int64_t ld_delta;
};

// rows [t0, t1): v = x[t] . A (rank floats), then delta[t] = sum_j (s v_j) B[j]
void run_rows(const Job& J, int32_t t0, int32_t t1) {
    std::vector<float> xr(J.h_in), v(J.rank);
    for (int32_t t = t0; t < t1; ++t) {
        widen(J.x + (int64_t)t * J.ldx, xr.data(), J.h_in, J.dtype);
        std::fill(v.begin(), v.end(), 0.f);
        for (int32_t k = 0; k < J.h_in; ++k) {
            const float xk = xr[k];
            const float* a = J.A + (int64_t)k * J.rank;
            for (int32_t j = 0; j < J.rank; ++j) v[j] += xk * a[j];
        }
        float* out = J.delta + (int64_t)t * J.ld_delta;
        std::fill(out, out + J.h_out, 0.f);
        for (int32_t j = 0; j < J.rank; ++j) {
            const float sv = J.scale * v[j];
            const float* b = J.B + (int64_t)j * J.h_out;
            for (int32_t n = 0; n < J.h_out; ++n) out[n] += sv * b[n];
        }
    }
}

}  // namespace

#pragma clang attribute pop

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
    std::vector<float> Af((size_t)h_in * rank), Bf((size_t)rank * h_out);
    widen((const uint16_t*)A, Af.data(), (int64_t)h_in * rank, dtype);
    widen((const uint16_t*)B, Bf.data(), (int64_t)rank * h_out, dtype);
    const Job J{(const uint16_t*)x, ldx, h_in, h_out, rank, dtype, Af.data(), Bf.data(), scale, delta, ld_delta};
    int32_t c = tokens_per_thread > 0 ? tokens_per_thread : (n_rows + max_threads - 1) / max_threads;
    int32_t n_thr = (n_rows + c - 1) / c;
    if (n_thr > max_threads) {
        n_thr = max_threads;
        c = (n_rows + n_thr - 1) / n_thr;
    }
    if (n_thr <= 1) {
        run_rows(J, 0, n_rows);
        return LORA_OK;
    }
    std::vector<std::thread> pool;
    pool.reserve(n_thr - 1);
    try {
        for (int32_t i = 1; i < n_thr; ++i) {
            const int32_t t0 = i * c, t1 = std::min(n_rows, t0 + c);
            if (t0 < t1) pool.emplace_back(run_rows, std::cref(J), t0, t1);
        }
    } catch (...) {
        for (auto& th : pool) th.join();
        return lora::set_error(LORA_E_NOMEM, "lora_cpu_delta: cannot start threads");
    }
    run_rows(J, 0, std::min(n_rows, c));
    for (auto& th : pool) th.join();
    return LORA_OK;
}
