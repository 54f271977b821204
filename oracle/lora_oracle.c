/*
 * Plain CPU oracle for the batched, heterogeneous-rank LoRA delta.
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product path may call, link or
 * load this file or the library built from it; only the tests, the smoke
 * check and the benchmark's CPU-baseline leg do.  It shares no code, header
 * or table with the HIP library.
 *
 * What it computes (paper, Section 2.1 "LLM adaption", Eq. 1): a weight
 * W in R^{H1 x H2} adapted by A in R^{H1 x r}, B in R^{r x H2} gives
 * y' = xW + xAB, in the row-vector convention y = xW.  Section 2.2 ("The need
 * of LLM-multiplexing") computes xAB on the fly for every request and adds it
 * to the shared base output xW; Section 2.3 (C2) and Section 4.1 ("GPU LoRA")
 * batch many requests, each gathering its own adapter, in one step.  So for
 * every row t of a segment whose adapter is g >= 0:
 *
 *     v[j]     = sum_k x[t,k] * A_g[k,j]              j < r_g
 *     d[n]     = s_g * sum_j v[j] * B_g[j,n]
 *     out[t,n] = y[t,n] + d[n]
 *
 * and rows with adapter -1 keep y unchanged.  The per-adapter scale s_g is
 * this build's reading (Eq. 1 has none; s = 1 recovers it).
 *
 * Arithmetic is IEEE double, sums in ascending index order, no blocking, no
 * fusion, built without fast-math or FP contraction.  Inputs are 16-bit
 * floats (binary16 or bfloat16) held as raw bits and widened exactly.
 * Rows may be spread over OpenMP threads; every element's summation order is
 * fixed and independent of the thread count.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_F16 0
#define ORACLE_BF16 1

/* ---------------------------------------------------------------------- */
/* 16-bit float formats (IEEE 754-2008 binary16; bfloat16 = upper half of  */
/* binary32)                                                                */
/* ---------------------------------------------------------------------- */

static double widen_f16(uint16_t h) {
    int sign = h >> 15;
    int e = (h >> 10) & 0x1f;
    int m = h & 0x3ff;
    double v;
    if (e == 0)
        v = ldexp((double)m, -24);                 /* subnormal: m * 2^-24 */
    else if (e == 31)
        v = m ? NAN : INFINITY;
    else
        v = ldexp((double)(m | 0x400), e - 25);    /* 1.m * 2^(e-15) */
    return sign ? -v : v;
}

static double widen_bf16(uint16_t b) {
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

static double widen(uint16_t bits, int dtype) {
    return dtype == ORACLE_F16 ? widen_f16(bits) : widen_bf16(bits);
}

/* Round a double to a binary format with p significand bits, minimum normal
 * exponent emin, maximum exponent emax and exponent bias, nearest-even,
 * directly from the double (no intermediate rounding). */
static uint16_t round_to_format(double x, int p, int emin, int emax, int bias, int exp_bits) {
    const uint16_t sign = signbit(x) ? (uint16_t)(1u << 15) : 0;
    const int mbits = p - 1;
    const uint16_t exp_all = (uint16_t)(((1u << exp_bits) - 1u) << mbits);
    if (isnan(x))
        return (uint16_t)(sign | exp_all | (1u << (mbits - 1)));
    double a = fabs(x);
    if (a == 0.0)
        return sign;
    if (isinf(a))
        return (uint16_t)(sign | exp_all);
    int e2;
    frexp(a, &e2);                      /* a = f * 2^e2, f in [0.5, 1) */
    int E = e2 - 1;                     /* a in [2^E, 2^(E+1)) */
    int qexp = (E < emin ? emin : E) - mbits;      /* exponent of one unit in the last place */
    double n = rint(ldexp(a, -qexp));   /* nearest-even count of units */
    double r = ldexp(n, qexp);
    double max_finite = ldexp(2.0 - ldexp(1.0, -mbits), emax);
    if (r > max_finite)
        return (uint16_t)(sign | exp_all);
    if (r < ldexp(1.0, emin))           /* subnormal (or rounded up to the smallest normal below) */
        return (uint16_t)(sign | (uint16_t)n);
    frexp(r, &e2);
    E = e2 - 1;
    uint32_t mant = (uint32_t)ldexp(r, mbits - E) - (1u << mbits);
    return (uint16_t)(sign | (uint16_t)((uint32_t)(E + bias) << mbits) | (uint16_t)mant);
}

uint16_t oracle_round_one(double x, int dtype) {
    if (dtype == ORACLE_F16)
        return round_to_format(x, 11, -14, 15, 15, 5);
    return round_to_format(x, 8, -126, 127, 127, 8);
}

void oracle_widen(const uint16_t* src, int dtype, double* dst, int64_t n) {
    for (int64_t i = 0; i < n; ++i) dst[i] = widen(src[i], dtype);
}

void oracle_round(const double* src, int dtype, uint16_t* dst, int64_t n) {
    for (int64_t i = 0; i < n; ++i) dst[i] = oracle_round_one(src[i], dtype);
}

int oracle_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads later calls use (n >= 1); the arithmetic does not depend on it. */
void oracle_set_num_threads(int n) {
#ifdef _OPENMP
    if (n >= 1) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* ---------------------------------------------------------------------- */
/* Batch bookkeeping                                                        */
/* ---------------------------------------------------------------------- */

/* Adapter of row t: the adapter of the segment that holds it. */
static int32_t row_adapter(int32_t t, int32_t n_segments, const int32_t* seg_offset,
                           const int32_t* seg_adapter) {
    for (int32_t s = 0; s < n_segments; ++s)
        if (t >= seg_offset[s] && t < seg_offset[s + 1]) return seg_adapter[s];
    return -1;
}

/* Group the rows of a step by adapter (the gather of Section 2.3 C2 / 4.1).
 * Groups are ordered by the first row that uses the adapter; rows inside a
 * group ascend; rows with adapter -1 belong to no group.  Writes perm[] (the
 * grouped row list), group_off[0..G] and group_adapter[0..G-1]; returns G.
 * Quadratic on purpose: every adapter is searched for over all rows. */
int32_t oracle_group_rows(int32_t n_rows, int32_t n_segments, const int32_t* seg_offset,
                          const int32_t* seg_adapter, int32_t* perm, int32_t* group_off,
                          int32_t* group_adapter) {
    int32_t G = 0;
    for (int32_t t = 0; t < n_rows; ++t) {
        int32_t a = row_adapter(t, n_segments, seg_offset, seg_adapter);
        if (a < 0) continue;
        int seen = 0;
        for (int32_t g = 0; g < G; ++g)
            if (group_adapter[g] == a) seen = 1;
        if (!seen) group_adapter[G++] = a;
    }
    int32_t p = 0;
    group_off[0] = 0;
    for (int32_t g = 0; g < G; ++g) {
        for (int32_t t = 0; t < n_rows; ++t)
            if (row_adapter(t, n_segments, seg_offset, seg_adapter) == group_adapter[g])
                perm[p++] = t;
        group_off[g + 1] = p;
    }
    return G;
}

/* ---------------------------------------------------------------------- */
/* The delta                                                                */
/* ---------------------------------------------------------------------- */

/* v[t, j] = sum_k x[t,k] * A_g[k,j] for every row t with adapter g >= 0,
 * j < r_g (the shrink half of xAB).  A_g is [h_in, r_g] row-major. Rows with
 * adapter -1 are not written. */
void oracle_lora_shrink(int32_t n_rows, int32_t n_segments, const int32_t* seg_offset,
                        const int32_t* seg_adapter, int32_t h_in, int dtype,
                        const uint16_t* x, int64_t ldx, const uint16_t* const* A,
                        const int32_t* ranks, double* v, int64_t ldv) {
    int32_t t;
#pragma omp parallel for schedule(dynamic, 1)
    for (t = 0; t < n_rows; ++t) {
        int32_t g = row_adapter(t, n_segments, seg_offset, seg_adapter);
        if (g < 0) continue;
        const int32_t r = ranks[g];
        for (int32_t j = 0; j < r; ++j) {
            double acc = 0.0;
            for (int32_t k = 0; k < h_in; ++k)
                acc += widen(x[(int64_t)t * ldx + k], dtype) * widen(A[g][(int64_t)k * r + j], dtype);
            v[(int64_t)t * ldv + j] = acc;
        }
    }
}

/* out[t, n] = y[t,n] + s_g * sum_j v[t,j] * B_g[j,n] (the expand half and the
 * add into the base output).  v is given in double; B_g is [r_g, h_out]
 * row-major.  Rows with adapter -1 get out = y. */
static void expand_rows(int32_t n_rows, int32_t n_segments, const int32_t* seg_offset,
                        const int32_t* seg_adapter, int32_t h_out, int dtype, const double* v,
                        int64_t ldv, const uint16_t* const* B, const int32_t* ranks,
                        const float* scales, const uint16_t* y, int64_t ldy, double* out,
                        int64_t ldo) {
    int32_t t;
#pragma omp parallel for schedule(dynamic, 1)
    for (t = 0; t < n_rows; ++t) {
        int32_t g = row_adapter(t, n_segments, seg_offset, seg_adapter);
        for (int32_t n = 0; n < h_out; ++n) {
            double base = widen(y[(int64_t)t * ldy + n], dtype);
            if (g < 0) {
                out[(int64_t)t * ldo + n] = base;
                continue;
            }
            const int32_t r = ranks[g];
            double acc = 0.0;
            for (int32_t j = 0; j < r; ++j)
                acc += v[(int64_t)t * ldv + j] * widen(B[g][(int64_t)j * h_out + n], dtype);
            out[(int64_t)t * ldo + n] = base + (double)scales[g] * acc;
        }
    }
}

/* Expand from a float32 v (the boundary type of the shrink result). */
void oracle_lora_expand(int32_t n_rows, int32_t n_segments, const int32_t* seg_offset,
                        const int32_t* seg_adapter, int32_t h_out, int dtype, const float* v,
                        int64_t ldv, const uint16_t* const* B, const int32_t* ranks,
                        const float* scales, const uint16_t* y, int64_t ldy, double* out,
                        int64_t ldo) {
    double* vd = (double*)malloc(sizeof(double) * (size_t)(n_rows > 0 ? n_rows : 1) * (size_t)(ldv > 0 ? ldv : 1));
    if (!vd) return;
    for (int64_t i = 0; i < (int64_t)n_rows * ldv; ++i) vd[i] = (double)v[i];
    expand_rows(n_rows, n_segments, seg_offset, seg_adapter, h_out, dtype, vd, ldv, B, ranks,
                scales, y, ldy, out, ldo);
    free(vd);
}

/* The whole delta: shrink in double, then expand and add. */
int oracle_lora_apply(int32_t n_rows, int32_t n_segments, const int32_t* seg_offset,
                      const int32_t* seg_adapter, int32_t h_in, int32_t h_out, int dtype,
                      const uint16_t* x, int64_t ldx, const uint16_t* const* A,
                      const uint16_t* const* B, const int32_t* ranks, const float* scales,
                      int32_t r_max, const uint16_t* y, int64_t ldy, double* out, int64_t ldo) {
    int64_t ldv = r_max > 0 ? r_max : 1;
    double* v = (double*)calloc((size_t)(n_rows > 0 ? n_rows : 1) * (size_t)ldv, sizeof(double));
    if (!v) return -1;
    oracle_lora_shrink(n_rows, n_segments, seg_offset, seg_adapter, h_in, dtype, x, ldx, A, ranks,
                       v, ldv);
    expand_rows(n_rows, n_segments, seg_offset, seg_adapter, h_out, dtype, v, ldv, B, ranks,
                scales, y, ldy, out, ldo);
    free(v);
    return 0;
}

/* Eq. 1 whole (Section 2.1): y' = xW + xAB, the base projection and the
 * adapter delta together, with the per-adapter scale:
 *     out[t, n] = sum_k x[t,k] W[k,n]  +  s_g sum_j v[t,j] B_g[j,n],
 *     v[t, j]   = sum_k x[t,k] A_g[k,j]
 * W is the paper's H1 x H2 weight, [h_in, h_out] row-major with leading
 * dimension ldw.  Rows with adapter -1 get x.W alone.  Double, k and j
 * ascending, the base sum and the delta added once at the end. */
int oracle_base_lora_apply(int32_t n_rows, int32_t n_segments, const int32_t* seg_offset,
                           const int32_t* seg_adapter, int32_t h_in, int32_t h_out, int dtype,
                           const uint16_t* x, int64_t ldx, const uint16_t* W, int64_t ldw,
                           const uint16_t* const* A, const uint16_t* const* B, const int32_t* ranks,
                           const float* scales, int32_t r_max, double* out, int64_t ldo) {
    int64_t ldv = r_max > 0 ? r_max : 1;
    double* v = (double*)calloc((size_t)(n_rows > 0 ? n_rows : 1) * (size_t)ldv, sizeof(double));
    if (!v) return -1;
    oracle_lora_shrink(n_rows, n_segments, seg_offset, seg_adapter, h_in, dtype, x, ldx, A, ranks,
                       v, ldv);
    int32_t t;
#pragma omp parallel for schedule(dynamic, 1)
    for (t = 0; t < n_rows; ++t) {
        const int32_t g = row_adapter(t, n_segments, seg_offset, seg_adapter);
        for (int32_t n = 0; n < h_out; ++n) {
            double base = 0.0;
            for (int32_t k = 0; k < h_in; ++k)
                base += widen(x[(int64_t)t * ldx + k], dtype) * widen(W[(int64_t)k * ldw + n], dtype);
            double delta = 0.0;
            if (g >= 0) {
                double acc = 0.0;
                for (int32_t j = 0; j < ranks[g]; ++j)
                    acc += v[(int64_t)t * ldv + j] * widen(B[g][(int64_t)j * h_out + n], dtype);
                delta = (double)scales[g] * acc;
            }
            out[(int64_t)t * ldo + n] = base + delta;
        }
    }
    free(v);
    return 0;
}

/* One output row only (for sampled checks at full size): out[0..h_out). */
int oracle_lora_apply_row(int32_t t, int32_t n_segments, const int32_t* seg_offset,
                          const int32_t* seg_adapter, int32_t h_in, int32_t h_out, int dtype,
                          const uint16_t* x, int64_t ldx, const uint16_t* const* A,
                          const uint16_t* const* B, const int32_t* ranks, const float* scales,
                          const uint16_t* y, int64_t ldy, double* out) {
    int32_t g = row_adapter(t, n_segments, seg_offset, seg_adapter);
    if (g < 0) {
        for (int32_t n = 0; n < h_out; ++n) out[n] = widen(y[(int64_t)t * ldy + n], dtype);
        return 0;
    }
    const int32_t r = ranks[g];
    double* v = (double*)calloc((size_t)(r > 0 ? r : 1), sizeof(double));
    if (!v) return -1;
    for (int32_t j = 0; j < r; ++j) {
        double acc = 0.0;
        for (int32_t k = 0; k < h_in; ++k)
            acc += widen(x[(int64_t)t * ldx + k], dtype) * widen(A[g][(int64_t)k * r + j], dtype);
        v[j] = acc;
    }
    for (int32_t n = 0; n < h_out; ++n) {
        double acc = 0.0;
        for (int32_t j = 0; j < r; ++j) acc += v[j] * widen(B[g][(int64_t)j * h_out + n], dtype);
        out[n] = widen(y[(int64_t)t * ldy + n], dtype) + (double)scales[g] * acc;
    }
    free(v);
    return 0;
}
