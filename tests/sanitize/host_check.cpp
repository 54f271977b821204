// Host-only exercise of the C ABI's planner and of the oracle, built with
// AddressSanitizer and UndefinedBehaviorSanitizer on the host code (the GPU
// code is compiled as usual and never launched: no call here reaches a HIP
// runtime function).  Random batches, shapes and ranks from a fixed seed:
//   * lora_group_rows equals the oracle's grouping, array for array;
//   * lora_plan_inspect lists a work list whose shrink K ranges, expand
//     column tiles and reduce slices cover each row block exactly once;
//   * malformed batches are refused with the documented codes;
//   * the oracle's apply equals its shrink followed by its expand, and its
//     one-row form equals the matching row of the full result.
// Any out-of-bounds access, use after free or undefined operation aborts
// the run with the sanitizer's report.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include <hip/hip_runtime.h>

#include "lora.h"
#include "lora_internal.h"
#include "lora_sched.h"
#include "lora_coldstart.h"

// The planner's launch functions live with the kernels, which this build
// leaves out: nothing here launches (every call exercised returns before any
// HIP call).  Stand-ins that report an error keep the link whole.
namespace lora {
hipError_t launch_shrink(const KernelArgs&, const uint32_t*, int, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_expand(const KernelArgs&, const uint32_t*, int, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_reduce(const KernelArgs&, const uint32_t*, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_step(const KernelArgs&, const uint32_t*, int, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_fill(uint32_t*, uint32_t, uint64_t, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_base(const BaseArgs&, int, hipStream_t) { return hipErrorNotSupported; }
}  // namespace lora

extern "C" {
int32_t oracle_group_rows(int32_t n_rows, int32_t n_segments, const int32_t* seg_offset,
                          const int32_t* seg_adapter, int32_t* perm, int32_t* group_off,
                          int32_t* group_adapter);
void oracle_lora_shrink(int32_t n_rows, int32_t n_segments, const int32_t* seg_offset,
                        const int32_t* seg_adapter, int32_t h_in, int dtype, const uint16_t* x, int64_t ldx,
                        const uint16_t* const* A, const int32_t* ranks, double* v, int64_t ldv);
void oracle_lora_expand(int32_t n_rows, int32_t n_segments, const int32_t* seg_offset,
                        const int32_t* seg_adapter, int32_t h_out, int dtype, const float* v, int64_t ldv,
                        const uint16_t* const* B, const int32_t* ranks, const float* scales, const uint16_t* y,
                        int64_t ldy, double* out, int64_t ldo);
int oracle_lora_apply(int32_t n_rows, int32_t n_segments, const int32_t* seg_offset, const int32_t* seg_adapter,
                      int32_t h_in, int32_t h_out, int dtype, const uint16_t* x, int64_t ldx,
                      const uint16_t* const* A, const uint16_t* const* B, const int32_t* ranks,
                      const float* scales, int32_t r_max, const uint16_t* y, int64_t ldy, double* out,
                      int64_t ldo);
int oracle_lora_apply_row(int32_t t, int32_t n_segments, const int32_t* seg_offset, const int32_t* seg_adapter,
                          int32_t h_in, int32_t h_out, int dtype, const uint16_t* x, int64_t ldx,
                          const uint16_t* const* A, const uint16_t* const* B, const int32_t* ranks,
                          const float* scales, const uint16_t* y, int64_t ldy, double* out);
}

namespace {

uint64_t g_state = 0x9e3779b97f4a7c15ull;
uint32_t rnd() {                      // xorshift64*
    g_state ^= g_state >> 12;
    g_state ^= g_state << 25;
    g_state ^= g_state >> 27;
    return (uint32_t)((g_state * 0x2545f4914f6cdd1dull) >> 32);
}
int rint_in(int lo, int hi) { return lo + (int)(rnd() % (uint32_t)(hi - lo + 1)); }

int failures = 0;
#define CHECK(cond, ...)                                   \
    do {                                                   \
        if (!(cond)) {                                     \
            std::fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__); \
            std::fprintf(stderr, __VA_ARGS__);             \
            std::fprintf(stderr, "\n");                    \
            ++failures;                                    \
        }                                                  \
    } while (0)

struct Batch {
    std::vector<int32_t> off, ad;
    lora_batch_t c() const { return lora_batch_t{off.back(), (int32_t)ad.size(), off.data(), ad.data()}; }
};

Batch random_batch(int n_adapters) {
    Batch b;
    b.off.push_back(0);
    const int nseg = rint_in(0, 90);
    for (int s = 0; s < nseg; ++s) {
        const int len = rnd() % 4 == 0 ? rint_in(0, 150) : 1;
        b.off.push_back(b.off.back() + len);
        b.ad.push_back(rint_in(-1, n_adapters - 1));
    }
    return b;
}

void check_grouping(const Batch& b, int n_adapters) {
    const lora_batch_t c = b.c();
    const int T = c.n_rows;
    std::vector<int32_t> p1(T + 1), o1(T + 2), a1(T + 1), p2(T + 1), o2(T + 2), a2(T + 1);
    int32_t G1 = -1;
    const int rc = lora_group_rows(&c, n_adapters, p1.data(), o1.data(), a1.data(), &G1);
    CHECK(rc == LORA_OK, "lora_group_rows rc %d: %s", rc, lora_last_error());
    const int32_t G2 = oracle_group_rows(T, c.n_segments, c.seg_offset, c.seg_adapter, p2.data(), o2.data(), a2.data());
    CHECK(G1 == G2, "groups %d vs %d", G1, G2);
    if (G1 != G2) return;
    for (int g = 0; g <= G1; ++g) CHECK(o1[g] == o2[g], "group_off[%d]", g);
    for (int g = 0; g < G1; ++g) CHECK(a1[g] == a2[g], "group_adapter[%d]", g);
    for (int i = 0; i < o1[G1]; ++i) CHECK(p1[i] == p2[i], "perm[%d]", i);
}

void check_plan(const Batch& b, int n_adapters) {
    std::vector<int32_t> ranks(n_adapters);
    for (auto& r : ranks) r = rnd() % 3 == 0 ? rint_in(1, 256) : (8 << rint_in(0, 4));
    const int h_in = 8 * rint_in(1, 1200), h_out = 8 * rint_in(1, 1200);
    const int n_xcd = rnd() % 2 ? 8 : 1;
    const lora_batch_t c = b.c();
    int32_t n = -1;
    int rc = lora_plan_inspect(&c, h_in, h_out, n_adapters, ranks.data(), n_xcd, nullptr, 0, &n);
    CHECK(rc == LORA_OK, "inspect size rc %d: %s", rc, lora_last_error());
    if (rc != LORA_OK) return;
    std::vector<lora_item_info_t> it(n > 0 ? n : 1);
    if (n > 0) {
        rc = lora_plan_inspect(&c, h_in, h_out, n_adapters, ranks.data(), n_xcd, it.data(), 0, &n);
        CHECK(rc == LORA_E_ARG, "capacity 0 must be refused (rc %d)", rc);
    }
    rc = lora_plan_inspect(&c, h_in, h_out, n_adapters, ranks.data(), n_xcd, it.data(), (int32_t)it.size(), &n);
    CHECK(rc == LORA_OK, "inspect rc %d: %s", rc, lora_last_error());
    if (rc != LORA_OK) return;
    // per row block: K covered once by its shrink items, h_out by its expand
    // tiles, its v block by its lora_shrink reduce slices
    int n_rb = 0;
    for (int i = 0; i < n; ++i) n_rb = std::max(n_rb, it[i].row_block + 1);
    std::vector<std::vector<int>> kcov(n_rb), ncov(n_rb), vcov(n_rb);
    std::vector<int> pstride(n_rb, 0);
    int grid_items = 0;
    for (int i = 0; i < n; ++i) {
        const auto& q = it[i];
        CHECK(q.kind >= 0 && q.kind <= 3, "kind %d", q.kind);
        if (q.kind == 0) continue;
        CHECK(q.row_block >= 0 && q.row_block < n_rb, "row block %d", q.row_block);
        CHECK(q.nrows >= 1 && q.nrows <= 64, "nrows %d", q.nrows);
        CHECK(q.rank >= 1 && q.rank <= 256, "rank %d", q.rank);
        auto& cov = q.kind == 1 ? kcov[q.row_block] : (q.kind == 2 ? ncov[q.row_block] : vcov[q.row_block]);
        const int lim = q.kind == 1 ? h_in : (q.kind == 2 ? h_out : q.pstride);
        if (q.kind == 3) {
            if (q.grid_pos >= 0) continue;        // the step launch's own reduce items: a subset
            pstride[q.row_block] = q.pstride;
        }
        if (q.grid_pos >= 0) ++grid_items;
        CHECK(q.lo >= 0 && q.len > 0 && q.lo + q.len <= lim, "range [%d,+%d) of %d (kind %d)", q.lo, q.len, lim, q.kind);
        if ((int)cov.size() < lim) cov.resize(lim, 0);
        for (int k = q.lo; k < q.lo + q.len && k < lim; ++k) ++cov[k];
    }
    for (int r = 0; r < n_rb; ++r) {
        for (size_t k = 0; k < kcov[r].size(); ++k) CHECK(kcov[r][k] == 1, "rb %d k %zu covered %d times", r, k, kcov[r][k]);
        CHECK((int)kcov[r].size() == h_in, "rb %d K coverage %zu of %d", r, kcov[r].size(), h_in);
        for (size_t k = 0; k < ncov[r].size(); ++k) CHECK(ncov[r][k] == 1, "rb %d col %zu covered %d times", r, k, ncov[r][k]);
        CHECK((int)ncov[r].size() == h_out, "rb %d column coverage %zu of %d", r, ncov[r].size(), h_out);
        for (size_t k = 0; k < vcov[r].size(); ++k) CHECK(vcov[r][k] == 1, "rb %d v float %zu covered %d times", r, k, vcov[r][k]);
        CHECK((int)vcov[r].size() == pstride[r], "rb %d v coverage", r);
    }
    (void)grid_items;
}

void check_errors(int n_adapters) {
    std::vector<int32_t> perm(16), off(17), ad(16);
    int32_t G = 0;
    {
        int32_t so[] = {0, 3, 2}, sa[] = {0, 1};
        lora_batch_t b{2, 2, so, sa};
        CHECK(lora_group_rows(&b, n_adapters, perm.data(), off.data(), ad.data(), &G) == LORA_E_SHAPE, "decreasing");
    }
    {
        int32_t so[] = {0, 1, 2}, sa[] = {0, n_adapters};
        lora_batch_t b{2, 2, so, sa};
        CHECK(lora_group_rows(&b, n_adapters, perm.data(), off.data(), ad.data(), &G) == LORA_E_INDEX, "index");
    }
    {
        int32_t so[] = {0, 1, 2}, sa[] = {0, -2};
        lora_batch_t b{2, 2, so, sa};
        CHECK(lora_group_rows(&b, n_adapters, perm.data(), off.data(), ad.data(), &G) == LORA_E_INDEX, "index -2");
    }
    {
        int32_t so[] = {0, 1, 2}, sa[] = {0, 0};
        lora_batch_t b{3, 2, so, sa};
        CHECK(lora_group_rows(&b, n_adapters, perm.data(), off.data(), ad.data(), &G) == LORA_E_SHAPE, "n_rows");
        CHECK(lora_group_rows(nullptr, n_adapters, perm.data(), off.data(), ad.data(), &G) == LORA_E_ARG, "null");
        int32_t r[1] = {0};
        int32_t n = 0;
        lora_batch_t ok{2, 2, so, sa};
        CHECK(lora_plan_inspect(&ok, 64, 64, 1, r, 1, nullptr, 0, &n) == LORA_E_RANK, "rank 0");
        r[0] = 8;
        CHECK(lora_plan_inspect(&ok, 60, 64, 1, r, 1, nullptr, 0, &n) == LORA_E_SHAPE, "h_in 60");
    }
}

void check_oracle() {
    for (int rep = 0; rep < 40; ++rep) {
        const int n_ad = rint_in(1, 5);
        const int h_in = rint_in(1, 40), h_out = rint_in(1, 40);
        const int dtype = rep & 1;
        std::vector<int32_t> ranks(n_ad);
        int r_max = 1;
        for (auto& r : ranks) r_max = std::max(r_max, r = rint_in(1, 9));
        Batch b;
        b.off.push_back(0);
        for (int s = rint_in(0, 6); s > 0; --s) {
            b.off.push_back(b.off.back() + rint_in(0, 3));
            b.ad.push_back(rint_in(-1, n_ad - 1));
        }
        const lora_batch_t c = b.c();
        const int T = c.n_rows;
        auto bits = [&](size_t n) {     // finite values of modest size in either format
            std::vector<uint16_t> v(n);
            for (auto& e : v) e = dtype == 0 ? (uint16_t)((rnd() & 0x83ff) | (rint_in(10, 18) << 10))
                                             : (uint16_t)((rnd() & 0x807f) | (rint_in(120, 130) << 7));
            return v;
        };
        std::vector<uint16_t> x = bits((size_t)T * h_in + 1), y = bits((size_t)T * h_out + 1);
        std::vector<std::vector<uint16_t>> A(n_ad), B(n_ad);
        std::vector<const uint16_t*> Ap(n_ad), Bp(n_ad);
        std::vector<float> scales(n_ad);
        for (int g = 0; g < n_ad; ++g) {
            A[g] = bits((size_t)h_in * ranks[g]);
            B[g] = bits((size_t)ranks[g] * h_out);
            Ap[g] = A[g].data();
            Bp[g] = B[g].data();
            scales[g] = 0.25f * rint_in(1, 8);
        }
        std::vector<double> out((size_t)T * h_out + 1), out2((size_t)T * h_out + 1), v((size_t)T * r_max + 1);
        CHECK(oracle_lora_apply(T, c.n_segments, c.seg_offset, c.seg_adapter, h_in, h_out, dtype, x.data(), h_in,
                                Ap.data(), Bp.data(), ranks.data(), scales.data(), r_max, y.data(), h_out,
                                out.data(), h_out) == 0, "oracle apply");
        oracle_lora_shrink(T, c.n_segments, c.seg_offset, c.seg_adapter, h_in, dtype, x.data(), h_in, Ap.data(),
                           ranks.data(), v.data(), r_max);
        std::vector<float> vf(v.size());
        for (size_t i = 0; i < v.size(); ++i) vf[i] = (float)v[i];
        oracle_lora_expand(T, c.n_segments, c.seg_offset, c.seg_adapter, h_out, dtype, vf.data(), r_max, Bp.data(),
                           ranks.data(), scales.data(), y.data(), h_out, out2.data(), h_out);
        auto widen = [&](uint16_t h) {  // binary16 or bfloat16 to double, for the error bound only
            if (dtype == 1) {
                uint32_t u = (uint32_t)h << 16;
                float f;
                std::memcpy(&f, &u, 4);
                return (double)f;
            }
            const int e = (h >> 10) & 31, m = h & 1023;
            const double v = e ? std::ldexp(1024 + m, e - 25) : std::ldexp(m, -24);
            return (h >> 15) ? -v : v;
        };
        std::vector<int32_t> row_ad(T, -1);
        for (int s = 0; s < c.n_segments; ++s)
            for (int t = c.seg_offset[s]; t < c.seg_offset[s + 1]; ++t) row_ad[t] = c.seg_adapter[s];
        for (int t = 0; t < T; ++t) {
            std::vector<double> row(h_out);
            CHECK(oracle_lora_apply_row(t, c.n_segments, c.seg_offset, c.seg_adapter, h_in, h_out, dtype, x.data(),
                                        h_in, Ap.data(), Bp.data(), ranks.data(), scales.data(), y.data(), h_out,
                                        row.data()) == 0, "apply_row");
            const int g = row_ad[t];
            for (int n = 0; n < h_out; ++n) {
                const double a = out[(size_t)t * h_out + n], e = out2[(size_t)t * h_out + n];
                CHECK(row[n] == a, "apply_row differs at %d,%d", t, n);
                // the expand took v rounded to float32: |error| <= s 2^-24 sum |v_j B_jn|
                double bound = 0.0;
                if (g >= 0)
                    for (int j = 0; j < ranks[g]; ++j)
                        bound += std::fabs(v[(size_t)t * r_max + j] * widen(B[g][(size_t)j * h_out + n]));
                bound = bound * scales[g >= 0 ? g : 0] * 0x1p-23 + 1e-300;
                CHECK(std::fabs(a - e) <= bound, "apply vs shrink+expand at %d,%d: %g %g (bound %g)", t, n, a, e,
                      bound);
            }
        }
    }
}

// the scheduler's simulator and cost score on random traces: every request
// routed to a valid instance, times ordered, no memory error
void check_sched(int reps) {
    for (int rep = 0; rep < reps; ++rep) {
        const int n = rint_in(0, 400);
        std::vector<lora_sim_req_t> q(n);
        double t = 0.0;
        for (int j = 0; j < n; ++j) {
            t += (double)rint_in(0, 50) * 0.1;
            q[j] = lora_sim_req_t{t, 8 << rint_in(0, 3), rint_in(1, 300), rint_in(1, 40), 0, (double)rint_in(0, 999) / 1000.0};
        }
        lora_sim_config_t c{};
        c.pre = lora_perf_model_t{LORA_PERF_TOKENS, 0, 0.01, 0.5};
        c.dec = lora_perf_model_t{rint_in(0, 1), 0, 0.002, 3.0};
        c.n_instances = rint_in(1, 12);
        c.max_batch = rint_in(1, 20);
        c.policy = rint_in(0, 3);
        c.avg_resp_len = 20.0;
        c.slo = 4.0;
        c.penalty = 100.0;
        std::vector<lora_sim_out_t> o(n);
        const int rc = lora_sim_run(&c, q.data(), n, o.data());
        CHECK(rc == LORA_OK, "lora_sim_run: %d %s", rc, lora_last_error());
        for (int j = 0; j < n; ++j) {
            CHECK(o[j].instance >= 0 && o[j].instance < c.n_instances, "request %d on instance %d", j, o[j].instance);
            CHECK(o[j].first_token >= q[j].arrival && o[j].finish >= o[j].first_token, "request %d times", j);
        }
        std::vector<lora_req_t> run(rint_in(0, 30)), qq(rint_in(0, 5));
        for (auto& r : run) r = lora_req_t{rint_in(1, 256), rint_in(1, 100)};
        for (auto& r : qq) r = lora_req_t{rint_in(1, 256), rint_in(1, 100)};
        const lora_req_t req{rint_in(1, 256), rint_in(1, 100)};
        const double cost = lora_sched_cost(&c.pre, &c.dec, &req, run.data(), (int32_t)run.size(), qq.data(),
                                            (int32_t)qq.size(), 10.0, 5.0, 1.0);
        CHECK(cost == cost, "lora_sched_cost gave NaN");
    }
    CHECK(lora_sim_run(nullptr, nullptr, 0, nullptr) == LORA_E_ARG, "NULL configuration accepted");
}

// the CPU LoRA kernel on random shapes and thread splits: no memory error,
// the same result for every split
void check_cpu_delta(int reps) {
    for (int rep = 0; rep < reps; ++rep) {
        const int T = rint_in(0, 40), h_in = 8 * rint_in(1, 40), h_out = 8 * rint_in(1, 40), r = rint_in(1, 64);
        const int dtype = rint_in(0, 1);
        std::vector<uint16_t> x((size_t)T * h_in + 1), A((size_t)h_in * r), Bm((size_t)r * h_out);
        for (auto& e : x) e = (uint16_t)(dtype ? 0x3c00 + rint_in(0, 255) : 0x3800 + rint_in(0, 511));
        for (auto& e : A) e = (uint16_t)(dtype ? 0x3c00 + rint_in(0, 255) : 0x3800 + rint_in(0, 511));
        for (auto& e : Bm) e = (uint16_t)(dtype ? 0x3c00 + rint_in(0, 255) : 0x3800 + rint_in(0, 511));
        std::vector<float> d1((size_t)T * h_out + 1), d2((size_t)T * h_out + 1);
        int rc = lora_cpu_delta(x.data(), h_in, T, h_in, h_out, dtype, A.data(), Bm.data(), r, 0.5f, d1.data(), h_out, 0, 1);
        CHECK(rc == LORA_OK, "lora_cpu_delta: %d %s", rc, lora_last_error());
        rc = lora_cpu_delta(x.data(), h_in, T, h_in, h_out, dtype, A.data(), Bm.data(), r, 0.5f, d2.data(), h_out,
                            rint_in(1, 9), rint_in(1, 8));
        CHECK(rc == LORA_OK, "lora_cpu_delta threads: %d %s", rc, lora_last_error());
        CHECK(std::memcmp(d1.data(), d2.data(), sizeof(float) * (size_t)T * h_out) == 0, "thread split changed the result");
    }
}

}  // namespace

int main() {
    for (int rep = 0; rep < 300; ++rep) {
        const int n_adapters = rint_in(1, 300);
        const Batch b = random_batch(n_adapters);
        check_grouping(b, n_adapters);
        check_plan(b, n_adapters);
    }
    check_errors(7);
    check_oracle();
    check_sched(200);
    check_cpu_delta(60);
    if (failures) {
        std::fprintf(stderr, "%d checks failed\n", failures);
        return 1;
    }
    std::printf("host_check: all checks passed\n");
    return 0;
}
