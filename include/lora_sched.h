/*
 * Rank-aware request scheduling (Section 5): the linear performance models of
 * a batch of heterogeneous adapters, their least-squares fit to measured
 * latencies, the cost score of Algorithm 1 and a discrete-time simulator of
 * instances under continuous batching that routes requests with Algorithm 1
 * or with the baselines of Section 7.4.
 *
 * Host code only: nothing here touches a GPU, allocates device memory or
 * synchronises a stream.  All arithmetic is IEEE double, evaluated in the
 * order written below (no fused multiply-add), so that a second
 * implementation following the same definitions reproduces every result bit
 * for bit.  Return codes are the LORA_* codes of lora.h; lora_last_error()
 * holds the message of the last failure on the calling thread.
 */
#ifndef LORA_SCHED_H
#define LORA_SCHED_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* One request as a batch sees it: its adapter's rank and the tokens it brings
 * to the iteration (its prompt length in a prefill, 1 in a decode step). */
typedef struct lora_req_s {
    int32_t rank;
    int32_t tokens;
} lora_req_t;

/* Feature of a batch S that a model is linear in (Section 5, "Performance
 * modeling"):
 *   LORA_PERF_PADDED    |S| * max_i rank(i)   (padded batched gather, BGMV)
 *   LORA_PERF_SUM_RANK  sum_i rank(i)         (padding-free, MBGMV; also this
 *                                              library's rank-bucketed kernels)
 *   LORA_PERF_TOKENS    sum_i tokens(i)       (a prompt batch, whose cost the
 *                                              base projection's token count
 *                                              sets; the paper gives no form
 *                                              for prefill, this is a reading)
 * The empty batch has feature 0 and costs 0 (no launch). */
enum { LORA_PERF_PADDED = 0, LORA_PERF_SUM_RANK = 1, LORA_PERF_TOKENS = 2 };

/* Perf(S) = alpha * feature(S) + beta for non-empty S, 0 for empty S. */
typedef struct lora_perf_model_s {
    int32_t kind;
    int32_t pad;
    double alpha;
    double beta;
} lora_perf_model_t;

/* feature(S) of n requests (n >= 0; reqs may be NULL when n == 0).  Returns
 * -1.0 for an unknown kind, a negative n or NULL reqs with n > 0. */
double lora_perf_feature(int32_t kind, const lora_req_t* reqs, int32_t n);

/* Perf(S) as above; -1.0 on the errors of lora_perf_feature. */
double lora_perf_eval(const lora_perf_model_t* m, const lora_req_t* reqs, int32_t n);

/* Ordinary least squares of t ~ alpha f + beta over n >= 2 samples with at
 * least two distinct f: alpha = S_ft / S_ff, beta = mean(t) - alpha mean(f),
 * r2 = 1 - SS_res / SS_tot (1 when SS_tot is 0).  out->kind = kind.  r2 may
 * be NULL.  LORA_E_ARG for NULL arrays or n < 2, LORA_E_SHAPE when every f is
 * equal. */
int lora_perf_fit(int32_t kind, const double* f, const double* t, int32_t n, lora_perf_model_t* out,
                  double* r2);

/* CalcCost of Algorithm 1 for request req on an instance with the given
 * running batch and queue:
 *   exists    = running + queue (decode form: tokens taken as 1)
 *   d_prefill = PrePerf(queue + req) - PrePerf(queue)   (prompt tokens)
 *   d_decode  = DecPerf(exists + req) - DecPerf(exists)
 *   cost      = d_prefill / avg_resp_len + d_decode
 *               (+ penalty when DecPerf(exists + req) > slo)
 * Returns the cost; NaN on NULL arguments or avg_resp_len <= 0. */
double lora_sched_cost(const lora_perf_model_t* pre, const lora_perf_model_t* dec, const lora_req_t* req,
                       const lora_req_t* running, int32_t n_running, const lora_req_t* queue, int32_t n_queue,
                       double avg_resp_len, double slo, double penalty);

/* Routing policies: Algorithm 1 and the three baselines of Section 7.4. */
enum {
    LORA_SCHED_RANK_AWARE = 0, /* minimum cost * (len(running) + len(queue)) over the candidates */
    LORA_SCHED_MOST_IDLE = 1,  /* fewest running + queued requests */
    LORA_SCHED_RANDOM = 2,     /* instance floor(u * n_instances) of the request's own uniform u */
    LORA_SCHED_FIRST_FIT = 3   /* first instance below max_batch, else the most idle */
};

typedef struct lora_sim_config_s {
    lora_perf_model_t pre;     /* prompt batch latency, kind LORA_PERF_TOKENS or another */
    lora_perf_model_t dec;     /* decode step latency */
    int32_t n_instances;       /* >= 1 */
    int32_t max_batch;         /* running + queued requests an instance takes before it stops being a
                                  candidate (>= 1) */
    int32_t policy;            /* LORA_SCHED_* */
    int32_t pad;
    double avg_resp_len;       /* Algorithm 1's average response length, > 0 */
    double slo;                /* time-per-token objective */
    double penalty;            /* added to the cost score of an instance the request would push past slo */
} lora_sim_config_t;

/* A request of the simulated trace.  Arrivals must not decrease along the
 * array; output >= 1 tokens (the first comes out of the prefill). */
typedef struct lora_sim_req_s {
    double arrival;
    int32_t rank;
    int32_t prompt;
    int32_t output;
    int32_t pad;
    double u;                  /* uniform [0, 1) draw used by LORA_SCHED_RANDOM */
} lora_sim_req_t;

typedef struct lora_sim_out_s {
    int32_t instance;
    int32_t pad;
    double first_token;        /* end of the prefill iteration that took the request */
    double finish;             /* end of the iteration that produced its last token */
    double tpot;               /* (finish - first_token) / (output - 1); 0 when output == 1 */
} lora_sim_out_t;

/*
 * Simulates the trace.  Each instance runs iterations back to back while it
 * has work (continuous batching, Section 2.2): when its queue is not empty, a
 * prefill iteration of the whole queue lasting PrePerf(queue), after which the
 * queued requests join the running batch in arrival order with their first
 * token; otherwise a decode iteration lasting DecPerf(running) that gives every
 * running request one token, requests with all their tokens leaving at its
 * end.  Before request j is routed, every instance runs the iterations that
 * start before its arrival to their end; the policy then sees each instance's
 * running batch and queue (Algorithm 1's GetStats), and the request joins the
 * chosen instance's queue (an idle instance's clock moves up to the arrival).
 * Ties between instances go to the lower index.  out[j] describes request j.
 * LORA_E_ARG for NULL pointers, n < 0, a bad policy or configuration, or
 * decreasing arrivals.
 */
int lora_sim_run(const lora_sim_config_t* c, const lora_sim_req_t* reqs, int32_t n, lora_sim_out_t* out);

#ifdef __cplusplus
}
#endif

#endif /* LORA_SCHED_H */
