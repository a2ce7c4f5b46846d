/*
 * msao_oracle_decode.c -- plain CPU oracle of the decoding-side quantities of
 * MSAO's adaptive speculative offloading (Sec. 4.2): the draft model's
 * confidence (Eq. 9) and speculation test (Eq. 10), the communication latency
 * (Eq. 8), the empirical speculation probability (Eq. 12), the expected
 * speculative run length (Eq. 13), the expected end-to-end latency (Eq. 14),
 * and the per-request and per-step logic of Algorithm 1.
 *
 * TEST INFRASTRUCTURE ONLY. This is the slow, obviously-correct reference the
 * library is checked against. Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load it; the product path never calls it.
 * It shares no code, header, table or helper with the library.
 *
 * Arithmetic: logits are widened exactly to float (bf16 -> float is a 16-bit
 * shift) and then to double; everything else is double, each formula written
 * out as the paper states it.
 *
 * Readings taken where the paper is silent (listed with their reasons in the
 * design notes):
 *  - entropy is in nats; the confidence threshold, which the paper keeps in
 *    [0, 1], applies to the entropy divided by its maximum ln|V|;
 *  - the draft token is the arg max of the logits (greedy drafting), the
 *    first index among equal maxima; a logit of -inf has probability 0;
 *  - the inverse empirical CDF of Algorithm 1 is the lower quantile
 *    sorted[ceil(q n) - 1];
 *  - the draft length of Algorithm 1 is clamped to [1, N_max] (P_conf = 1
 *    gives N_max, P_conf = 0 gives 1);
 *  - the retention of Algorithm 1 sits at the floor of Eq. 11:
 *    beta_m = 1 - MAS_m;
 *  - "cache" counts the drafted tokens held on the edge; a confident step adds
 *    its token, and when the cache holds N_draft tokens they are sent for
 *    verification and the threshold moves by an EMA (weight alpha) toward
 *    the mean normalised entropy of those tokens; an unconfident step
 *    offloads (the held tokens travel with the offloaded state, emptying the
 *    cache) and decays the threshold to max(theta * delta, theta_min).
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { ORC_F32 = 0, ORC_BF16 = 1 };
enum { ORC_HOLD = 0, ORC_SEND = 1, ORC_OFFLOAD = 2 };

static double logit_at(const void* row, int dtype, int64_t v)
{
    if (dtype == ORC_F32) return (double)((const float*)row)[v];
    uint32_t bits = (uint32_t)((const uint16_t*)row)[v] << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

/* Eq. 9 for every row: H = -sum_v p_v log p_v with p the softmax of the row's
 * logits (0 log 0 = 0), and the first index of the largest logit. A row with
 * a NaN or +inf logit, or with no finite logit, gets H = NaN. */
void orc_entropy_rows(const void* logits, int64_t rows, int64_t vocab, int64_t row_stride, int dtype,
                      double* H, int32_t* argmax)
{
    const size_t es = dtype == ORC_F32 ? 4 : 2;
    for (int64_t r = 0; r < rows; ++r) {
        const void* row = (const uint8_t*)logits + (size_t)r * (size_t)row_stride * es;
        double m = -INFINITY;
        int64_t am = 0;
        int bad = 0;
        for (int64_t v = 0; v < vocab; ++v) {
            const double x = logit_at(row, dtype, v);
            if (isnan(x) || (isinf(x) && x > 0)) bad = 1;
            if (x > m) {
                m = x;
                am = v;
            }
        }
        argmax[r] = (int32_t)am;
        if (bad || !(m > -INFINITY)) {
            H[r] = NAN;
            continue;
        }
        double S = 0.0;
        for (int64_t v = 0; v < vocab; ++v) S += exp(logit_at(row, dtype, v) - m);
        double h = 0.0;
        for (int64_t v = 0; v < vocab; ++v) {
            const double p = exp(logit_at(row, dtype, v) - m) / S;
            if (p > 0.0) h -= p * log(p);
        }
        H[r] = h;
    }
}

/* The entropy divided by its maximum ln|V| (the threshold's scale). */
double orc_entropy_normalized(double H, int64_t vocab) { return H / log((double)vocab); }

/* Eq. 10: speculate iff the (normalised) entropy is at most theta. */
int orc_speculate(double h_norm, double theta) { return h_norm <= theta; }

/* Eq. 8: transfer time of one modality plus the round trip. */
double orc_comm_latency(double data_bytes, double bandwidth_bytes_per_s, double rtt_s)
{
    return data_bytes / bandwidth_bytes_per_s + rtt_s;
}

/* Eq. 12: fraction of steps whose entropy is at most theta. */
double orc_p_conf(const double* h, int64_t n, double theta)
{
    int64_t c = 0;
    for (int64_t i = 0; i < n; ++i)
        if (h[i] <= theta) ++c;
    return n > 0 ? (double)c / (double)n : 0.0;
}

/* Eq. 13, closed form: E[N_spec] = 1 / (1 - P_conf) (infinite at P_conf = 1). */
double orc_expected_spec(double p_conf) { return p_conf >= 1.0 ? INFINITY : 1.0 / (1.0 - p_conf); }

/* Eq. 14. comm_offloaded is the sum over offloaded modalities of Eq. 8. */
double orc_expected_e2e(double prefill_edge, double prefill_cloud, double comm_offloaded, double p_conf,
                        int n_draft, double t_draft, double t_verify, double t_offload)
{
    const double prefill = prefill_edge > prefill_cloud + comm_offloaded ? prefill_edge
                                                                          : prefill_cloud + comm_offloaded;
    const double T_draft = (double)n_draft * t_draft;
    const double T_verify = (double)n_draft * t_verify;
    return prefill + orc_expected_spec(p_conf) * (T_draft + p_conf * T_verify) + (1.0 - p_conf) * t_offload;
}

static int cmp_double(const void* a, const void* b)
{
    const double x = *(const double*)a, y = *(const double*)b;
    return (x > y) - (x < y);
}

/* Inverse empirical CDF of Algorithm 1 (line 2): sorted[ceil(q n) - 1]. */
double orc_entropy_quantile(const double* h, int64_t n, double q)
{
    if (n <= 0) return NAN;
    double* s = (double*)malloc(sizeof(double) * (size_t)n);
    memcpy(s, h, sizeof(double) * (size_t)n);
    qsort(s, (size_t)n, sizeof(double), cmp_double);
    int64_t i = (int64_t)ceil(q * (double)n) - 1;
    if (i < 0) i = 0;
    if (i > n - 1) i = n - 1;
    const double v = s[i];
    free(s);
    return v;
}

/* Algorithm 1, line 3: N_draft = min(floor(log(1 - P_target) / log P_conf), N_max), at least 1. */
int orc_n_draft(double p_conf, double p_target, int n_max)
{
    if (p_conf >= 1.0) return n_max;
    if (p_conf <= 0.0) return 1;
    const double n = floor(log(1.0 - p_target) / log(p_conf));
    if (n >= (double)n_max) return n_max;
    if (n < 1.0) return 1;
    return (int)n;
}

/* Algorithm 1, line 1 at the floor of Eq. 11: beta_m = 1 - MAS_m. */
void orc_retention(const double* mas, int k, double* beta)
{
    for (int m = 0; m < k; ++m) beta[m] = 1.0 - mas[m];
}

/* Algorithm 1, lines 4-12, over a trace of normalised entropies. theta starts
 * at theta0; decisions[i] is HOLD, SEND or OFFLOAD and theta_after[i] the
 * threshold after step i. counts = {held, sent batches, offloads, tokens sent}. */
void orc_sched_run(const double* h_norm, int64_t steps, double theta0, int n_draft, double delta,
                   double theta_min, double alpha, int8_t* decisions, double* theta_after, int64_t* counts)
{
    double theta = theta0;
    int64_t cache = 0;
    double cache_h = 0.0;
    int64_t held = 0, sends = 0, offloads = 0, tokens_sent = 0;
    for (int64_t i = 0; i < steps; ++i) {
        const double h = h_norm[i];
        int8_t d;
        if (h <= theta) {
            cache += 1;
            cache_h += h;
            if (cache >= n_draft) {
                d = ORC_SEND;
                theta = (1.0 - alpha) * theta + alpha * (cache_h / (double)cache);
                tokens_sent += cache;
                sends += 1;
                cache = 0;
                cache_h = 0.0;
            } else {
                d = ORC_HOLD;
                held += 1;
            }
        } else {
            d = ORC_OFFLOAD;
            offloads += 1;
            cache = 0;
            cache_h = 0.0;
            theta = theta * delta > theta_min ? theta * delta : theta_min;
        }
        decisions[i] = d;
        theta_after[i] = theta;
    }
    counts[0] = held;
    counts[1] = sends;
    counts[2] = offloads;
    counts[3] = tokens_sent;
}
