// Rank-aware scheduling of Section 5: linear performance models of a batch of
// heterogeneous adapters, their least-squares fit, Algorithm 1's cost score,
// and a discrete-time simulator of instances under continuous batching.
// Host code; every floating-point result is a plain IEEE double operation in
// the order written, with contraction into fused multiply-adds switched off,
// so that another implementation of the same definitions agrees bit for bit.
#include <cmath>
#include <cstdint>
#include <limits>
#include <string>
#include <vector>

#include "lora.h"
#include "lora_sched.h"

#pragma clang fp contract(off)

namespace lora {
int set_error(int code, const std::string& msg);
}

namespace {

bool kind_ok(int32_t kind) { return kind == LORA_PERF_PADDED || kind == LORA_PERF_SUM_RANK || kind == LORA_PERF_TOKENS; }

// feature(S): integers summed exactly (they stay far below 2^53), then one
// conversion
double feature(int32_t kind, const lora_req_t* r, int32_t n) {
    if (n == 0) return 0.0;
    if (kind == LORA_PERF_PADDED) {
        int64_t mx = 0;
        for (int32_t i = 0; i < n; ++i) mx = r[i].rank > mx ? r[i].rank : mx;
        return (double)((int64_t)n * mx);
    }
    int64_t s = 0;
    for (int32_t i = 0; i < n; ++i) s += kind == LORA_PERF_SUM_RANK ? r[i].rank : r[i].tokens;
    return (double)s;
}

double eval(const lora_perf_model_t& m, const lora_req_t* r, int32_t n) {
    if (n == 0) return 0.0;
    const double f = feature(m.kind, r, n);
    return m.alpha * f + m.beta;
}

// CalcCost of Algorithm 1 over prepared request lists
double calc_cost(const lora_perf_model_t& pre, const lora_perf_model_t& dec, const lora_req_t& req,
                 const std::vector<lora_req_t>& run, const std::vector<lora_req_t>& queue, double avg_resp_len,
                 double slo, double penalty) {
    // queue + req, prompt form
    std::vector<lora_req_t> q1(queue);
    q1.push_back(req);
    const double d_prefill = eval(pre, q1.data(), (int32_t)q1.size()) - eval(pre, queue.data(), (int32_t)queue.size());
    // exists = running + queue, decode form (one token each)
    std::vector<lora_req_t> ex;
    ex.reserve(run.size() + queue.size() + 1);
    for (const lora_req_t& r : run) ex.push_back(lora_req_t{r.rank, 1});
    for (const lora_req_t& r : queue) ex.push_back(lora_req_t{r.rank, 1});
    const double dec0 = eval(dec, ex.data(), (int32_t)ex.size());
    ex.push_back(lora_req_t{req.rank, 1});
    const double dec1 = eval(dec, ex.data(), (int32_t)ex.size());
    const double d_decode = dec1 - dec0;
    double cost = d_prefill / avg_resp_len + d_decode;
    if (dec1 > slo) cost = cost + penalty;
    return cost;
}

struct Instance {
    double clock = 0.0;
    std::vector<int32_t> run;     // request indices, in the order they joined
    std::vector<int32_t> queue;
    std::vector<int32_t> left;    // tokens still to produce, per running request (parallel to run)
    bool idle() const { return run.empty() && queue.empty(); }
    int32_t load() const { return (int32_t)(run.size() + queue.size()); }
};

struct Sim {
    const lora_sim_config_t& c;
    const lora_sim_req_t* reqs;
    lora_sim_out_t* out;
    std::vector<Instance> inst;

    std::vector<lora_req_t> as_prompt(const std::vector<int32_t>& ids) const {
        std::vector<lora_req_t> v;
        v.reserve(ids.size());
        for (int32_t j : ids) v.push_back(lora_req_t{reqs[j].rank, reqs[j].prompt});
        return v;
    }
    std::vector<lora_req_t> as_decode(const std::vector<int32_t>& ids) const {
        std::vector<lora_req_t> v;
        v.reserve(ids.size());
        for (int32_t j : ids) v.push_back(lora_req_t{reqs[j].rank, 1});
        return v;
    }

    void finish(int32_t j, double t) {
        out[j].finish = t;
        const int32_t o = reqs[j].output;
        out[j].tpot = o > 1 ? (t - out[j].first_token) / (double)(o - 1) : 0.0;
    }

    // one iteration of instance i
    void iterate(Instance& I) {
        if (!I.queue.empty()) {
            const std::vector<lora_req_t> q = as_prompt(I.queue);
            I.clock = I.clock + eval(c.pre, q.data(), (int32_t)q.size());
            for (int32_t j : I.queue) {
                out[j].first_token = I.clock;
                if (reqs[j].output <= 1) {
                    finish(j, I.clock);
                } else {
                    I.run.push_back(j);
                    I.left.push_back(reqs[j].output - 1);
                }
            }
            I.queue.clear();
            return;
        }
        const std::vector<lora_req_t> r = as_decode(I.run);
        I.clock = I.clock + eval(c.dec, r.data(), (int32_t)r.size());
        size_t k = 0;
        for (size_t i = 0; i < I.run.size(); ++i) {
            const int32_t j = I.run[i];
            const int32_t left = I.left[i] - 1;
            if (left == 0) {
                finish(j, I.clock);
            } else {
                I.run[k] = j;
                I.left[k] = left;
                ++k;
            }
        }
        I.run.resize(k);
        I.left.resize(k);
    }

    // run the iterations that start before time `until`
    void advance(Instance& I, double until) {
        while (!I.idle() && I.clock < until) iterate(I);
    }

    int32_t most_idle() const {
        int32_t best = 0;
        for (int32_t i = 1; i < c.n_instances; ++i)
            if (inst[i].load() < inst[best].load()) best = i;
        return best;
    }

    int32_t pick(int32_t j) const {
        const int32_t m = c.n_instances;
        switch (c.policy) {
            case LORA_SCHED_MOST_IDLE:
                return most_idle();
            case LORA_SCHED_RANDOM: {
                const double u = reqs[j].u;
                int32_t i = (int32_t)std::floor(u * (double)m);
                if (i < 0) i = 0;
                if (i >= m) i = m - 1;
                return i;
            }
            case LORA_SCHED_FIRST_FIT:
                for (int32_t i = 0; i < m; ++i)
                    if (inst[i].load() < c.max_batch) return i;
                return most_idle();
            default: {
                // Algorithm 1: the candidates are the instances with room; with
                // none, every instance
                bool any = false;
                for (int32_t i = 0; i < m; ++i) any = any || inst[i].load() < c.max_batch;
                const lora_req_t req{reqs[j].rank, reqs[j].prompt};
                int32_t best = -1;
                double best_cost = 0.0;
                for (int32_t i = 0; i < m; ++i) {
                    const Instance& I = inst[i];
                    if (any && I.load() >= c.max_batch) continue;
                    const double cost = calc_cost(c.pre, c.dec, req, as_prompt(I.run), as_prompt(I.queue),
                                                  c.avg_resp_len, c.slo, c.penalty);
                    const double total = cost * (double)I.load();
                    if (best < 0 || total < best_cost) {
                        best = i;
                        best_cost = total;
                    }
                }
                return best;
            }
        }
    }
};

bool model_ok(const lora_perf_model_t& m) { return kind_ok(m.kind); }

}  // namespace

extern "C" {

double lora_perf_feature(int32_t kind, const lora_req_t* reqs, int32_t n) {
    if (!kind_ok(kind) || n < 0 || (n > 0 && !reqs)) return -1.0;
    return feature(kind, reqs, n);
}

double lora_perf_eval(const lora_perf_model_t* m, const lora_req_t* reqs, int32_t n) {
    if (!m || !kind_ok(m->kind) || n < 0 || (n > 0 && !reqs)) return -1.0;
    return eval(*m, reqs, n);
}

int lora_perf_fit(int32_t kind, const double* f, const double* t, int32_t n, lora_perf_model_t* out, double* r2) {
    if (!f || !t || !out) return lora::set_error(LORA_E_ARG, "lora_perf_fit: NULL argument");
    if (n < 2) return lora::set_error(LORA_E_ARG, "lora_perf_fit: needs at least two samples");
    if (!kind_ok(kind)) return lora::set_error(LORA_E_ARG, "lora_perf_fit: unknown model kind");
    double sf = 0.0, st = 0.0;
    for (int32_t i = 0; i < n; ++i) {
        sf = sf + f[i];
        st = st + t[i];
    }
    const double mf = sf / (double)n, mt = st / (double)n;
    double sff = 0.0, sft = 0.0, stt = 0.0;
    for (int32_t i = 0; i < n; ++i) {
        const double df = f[i] - mf, dt = t[i] - mt;
        sff = sff + df * df;
        sft = sft + df * dt;
        stt = stt + dt * dt;
    }
    if (!(sff > 0.0)) return lora::set_error(LORA_E_SHAPE, "lora_perf_fit: every feature value is equal");
    const double alpha = sft / sff;
    const double beta = mt - alpha * mf;
    double ssr = 0.0;
    for (int32_t i = 0; i < n; ++i) {
        const double e = t[i] - (alpha * f[i] + beta);
        ssr = ssr + e * e;
    }
    out->kind = kind;
    out->pad = 0;
    out->alpha = alpha;
    out->beta = beta;
    if (r2) *r2 = stt > 0.0 ? 1.0 - ssr / stt : 1.0;
    return LORA_OK;
}

double lora_sched_cost(const lora_perf_model_t* pre, const lora_perf_model_t* dec, const lora_req_t* req,
                       const lora_req_t* running, int32_t n_running, const lora_req_t* queue, int32_t n_queue,
                       double avg_resp_len, double slo, double penalty) {
    const double nan = std::numeric_limits<double>::quiet_NaN();
    if (!pre || !dec || !req || !model_ok(*pre) || !model_ok(*dec) || n_running < 0 || n_queue < 0 ||
        (n_running > 0 && !running) || (n_queue > 0 && !queue) || !(avg_resp_len > 0.0))
        return nan;
    const std::vector<lora_req_t> run(running, running + n_running), q(queue, queue + n_queue);
    return calc_cost(*pre, *dec, *req, run, q, avg_resp_len, slo, penalty);
}

int lora_sim_run(const lora_sim_config_t* c, const lora_sim_req_t* reqs, int32_t n, lora_sim_out_t* out) {
    if (!c || n < 0 || (n > 0 && (!reqs || !out))) return lora::set_error(LORA_E_ARG, "lora_sim_run: NULL argument");
    if (c->n_instances < 1 || c->max_batch < 1 || c->policy < 0 || c->policy > LORA_SCHED_FIRST_FIT ||
        !model_ok(c->pre) || !model_ok(c->dec) || !(c->avg_resp_len > 0.0))
        return lora::set_error(LORA_E_ARG, "lora_sim_run: bad configuration");
    for (int32_t j = 0; j < n; ++j) {
        if (reqs[j].output < 1 || reqs[j].rank < 1 || reqs[j].prompt < 1)
            return lora::set_error(LORA_E_ARG, "lora_sim_run: request " + std::to_string(j) +
                                                   " needs rank, prompt and output >= 1");
        if (j > 0 && reqs[j].arrival < reqs[j - 1].arrival)
            return lora::set_error(LORA_E_ARG, "lora_sim_run: arrivals decrease at request " + std::to_string(j));
    }
    Sim S{*c, reqs, out, std::vector<Instance>(c->n_instances)};
    for (int32_t j = 0; j < n; ++j) {
        out[j] = lora_sim_out_t{-1, 0, 0.0, 0.0, 0.0};
        const double a = reqs[j].arrival;
        for (Instance& I : S.inst) S.advance(I, a);
        const int32_t i = S.pick(j);
        Instance& I = S.inst[i];
        if (I.idle() && I.clock < a) I.clock = a;
        I.queue.push_back(j);
        out[j].instance = i;
    }
    for (Instance& I : S.inst) S.advance(I, std::numeric_limits<double>::infinity());
    return LORA_OK;
}

}  // extern "C"
