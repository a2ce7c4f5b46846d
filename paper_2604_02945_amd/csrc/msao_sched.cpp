// msao_sched.cpp -- host side of MSAO's adaptive speculative edge-cloud
// offloading (Sec. 4.2): the latency model (Eq. 8, 12-14) and Algorithm 1's
// per-request initialisation and per-step threshold logic, driven by the
// normalised entropies that msao_draft_entropy computes on the GPU.
//
// Everything is double precision with no contraction of multiply-adds, so
// that a decision at the threshold is reproducible bit for bit.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <vector>

#include "../../include/msao.h"

#pragma clang fp contract(off)

namespace {

bool is_finite(double x) { return std::isfinite(x); }

bool params_ok(const msao_sched_params* p)
{
    return p && p->p_target > 0.0 && p->p_target < 1.0 && p->n_max >= 1 && p->quantile >= 0.0 &&
           p->quantile <= 1.0 && p->delta > 0.0 && p->delta <= 1.0 && p->theta_min >= 0.0 &&
           is_finite(p->theta_min) && p->alpha >= 0.0 && p->alpha <= 1.0;
}

// Algorithm 1, line 3, with the draft length kept in [1, N_max].
int32_t draft_length(double p_conf, double p_target, int32_t n_max)
{
    if (p_conf >= 1.0) return n_max;
    if (p_conf <= 0.0) return 1;
    const double len = std::floor(std::log(1.0 - p_target) / std::log(p_conf));
    if (len >= (double)n_max) return n_max;
    return len < 1.0 ? 1 : (int32_t)len;
}

}  // namespace

extern "C" {

msao_sched_params msao_sched_default_params(void)
{
    msao_sched_params p;
    p.p_target = 0.8;
    p.n_max = 5;
    p.quantile = 0.7;
    p.delta = 0.95;
    p.theta_min = 0.05;
    p.alpha = 0.1;
    return p;
}

double msao_comm_latency(double data_bytes, double bandwidth_bytes_per_s, double rtt_s)
{
    return data_bytes / bandwidth_bytes_per_s + rtt_s;
}

double msao_p_conf(const float* h_norm, int64_t n, double theta)
{
    if (!h_norm || n < 1) return 0.0;
    int64_t below = 0;
    for (int64_t i = 0; i < n; ++i) below += (double)h_norm[i] <= theta ? 1 : 0;
    return (double)below / (double)n;
}

double msao_expected_spec_tokens(double p_conf) { return p_conf >= 1.0 ? INFINITY : 1.0 / (1.0 - p_conf); }

double msao_expected_e2e_latency(const msao_latency_model* m)
{
    if (!m) return NAN;
    const double cloud = m->prefill_cloud + m->comm_offloaded;
    const double prefill = std::max(m->prefill_edge, cloud);
    const double draft = (double)m->n_draft * m->t_draft;
    const double verify = (double)m->n_draft * m->t_verify;
    const double spec = msao_expected_spec_tokens(m->p_conf) * (draft + m->p_conf * verify);
    return prefill + spec + (1.0 - m->p_conf) * m->t_offload;
}

msao_status msao_retention_floor(const float* mas, int n, float* beta)
{
    if (n < 0 || (n > 0 && (!mas || !beta))) return MSAO_ERR_INVALID_ARG;
    for (int m = 0; m < n; ++m) beta[m] = (float)(1.0 - (double)mas[m]);
    return MSAO_OK;
}

msao_status msao_sched_init(const float* calib_h_norm, int64_t n, const msao_sched_params* params,
                            msao_sched_state* state)
{
    if (!calib_h_norm || n < 1 || !state || !params_ok(params)) return MSAO_ERR_INVALID_ARG;
    std::vector<double> h((size_t)n);
    for (int64_t i = 0; i < n; ++i) {
        h[(size_t)i] = (double)calib_h_norm[i];
        if (!is_finite(h[(size_t)i])) return MSAO_ERR_INVALID_ARG;
    }
    // line 2: the inverse empirical CDF at `quantile` (the lower quantile)
    int64_t at = (int64_t)std::ceil(params->quantile * (double)n) - 1;
    at = std::min<int64_t>(std::max<int64_t>(at, 0), n - 1);
    std::nth_element(h.begin(), h.begin() + at, h.end());
    const double theta = h[(size_t)at];
    *state = msao_sched_state{};
    state->theta = theta;
    state->p_conf = msao_p_conf(calib_h_norm, n, theta);  // Eq. 12
    state->n_draft = draft_length(state->p_conf, params->p_target, params->n_max);
    return MSAO_OK;
}

msao_status msao_sched_step(msao_sched_state* state, const msao_sched_params* params, float h_norm,
                            int32_t* decision)
{
    if (!state || !params || !decision) return MSAO_ERR_INVALID_ARG;
    const double h = (double)h_norm;
    state->steps += 1;
    if (h <= state->theta) {  // Eq. 10: confident, speculate
        state->cache += 1;
        state->cache_h += h;
        if (state->cache >= state->n_draft) {
            const double mean = state->cache_h / (double)state->cache;
            state->theta = (1.0 - params->alpha) * state->theta + params->alpha * mean;
            state->tokens_sent += state->cache;
            state->sends += 1;
            state->cache = 0;
            state->cache_h = 0.0;
            *decision = MSAO_DECIDE_SEND;
        } else {
            state->held += 1;
            *decision = MSAO_DECIDE_HOLD;
        }
    } else {
        const double decayed = state->theta * params->delta;
        state->theta = decayed > params->theta_min ? decayed : params->theta_min;
        state->offloads += 1;
        state->cache = 0;
        state->cache_h = 0.0;
        *decision = MSAO_DECIDE_OFFLOAD;
    }
    return MSAO_OK;
}

msao_status msao_sched_run(msao_sched_state* state, const msao_sched_params* params, const float* h_norm,
                           int64_t steps, int8_t* decisions, double* theta_after)
{
    if (!state || !params || steps < 0 || (steps > 0 && !h_norm)) return MSAO_ERR_INVALID_ARG;
    for (int64_t i = 0; i < steps; ++i) {
        int32_t d = 0;
        const msao_status st = msao_sched_step(state, params, h_norm[i], &d);
        if (st != MSAO_OK) return st;
        if (decisions) decisions[i] = (int8_t)d;
        if (theta_after) theta_after[i] = state->theta;
    }
    return MSAO_OK;
}

}  // extern "C"
