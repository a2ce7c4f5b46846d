/*
 * msao_oracle.c -- plain CPU oracle of MSAO's fine-grained sparsity analysis
 * (Sec. 4.1: spatial sparsity Eq. 3-4, temporal sparsity Eq. 5, modal
 * sparsity Eq. 6, MAS Eq. 7) and of the MAS-guided token selection and
 * compaction that the analysis drives (the retention floor of Eq. 11 and the
 * pruning of low-importance patches in Sec. 4.1.1).
 *
 * TEST INFRASTRUCTURE ONLY. This is the slow, obviously-correct reference the
 * GPU path is checked against. Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load it; the product path never calls it.
 * It shares no code, header, table or helper with the GPU path.
 *
 * Arithmetic: inputs are widened exactly to float (bf16 -> float is a 16-bit
 * shift); sums are accumulated in double and rounded once to float; counts
 * are exact integers; everything derived from counts is computed in double
 * and rounded once to float. No blocking, fusion or reordering: each step is
 * a plain loop in the order the method states it.
 *
 * Readings taken where the paper is silent (each one is listed with its
 * justification in the design notes of this repository):
 *  - the learned spatial head of Eq. 3 is replaced by a parameter-free
 *    importance: the fraction of a token's channels that are active;
 *  - a channel is active iff NOT(|x| <= tau) (so NaN counts as active);
 *  - the hash family of Eq. 5 is bit sampling over the activity bits, every
 *    channel sampled once (K = C per token, K = P*C per frame);
 *  - frame 0 is compared with an all-zero predecessor and excluded from the
 *    averages; a clip with one frame has no temporal term;
 *  - MAS uses the redundancy 1 - gamma_avg by default (flag LITERAL uses
 *    gamma_avg as printed); the inner bracket is clamped to [0, 1];
 *  - a token's selection key is the exact integer
 *        Ls*z + Lt*(C - d)   with Ls = rne(lambda_s * 2^24), Lt likewise,
 *    the keep count is k = min(N, ceil(kappa * N)) and the k smallest
 *    (key, index) pairs of each segment are kept, ties by ascending index.
 *
 * Parity pins for every function below live in the CPU test suite.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { ORC_TEXT = 0, ORC_IMAGE = 1, ORC_VIDEO = 2, ORC_AUDIO = 3, ORC_NMOD = 4 };
enum { ORC_F32 = 0, ORC_BF16 = 1 };
enum { ORC_FLAG_TEMPORAL_LITERAL = 1 };

typedef struct {
    const void* data;          /* row (t*P + p) starts at data + (t*P+p)*row_stride elements */
    int64_t row_stride;        /* elements */
    int32_t request;
    int32_t modality;
    int32_t n_frames;          /* T */
    int32_t tokens_per_frame;  /* P */
    int32_t hidden;            /* C */
    int32_t dtype;
    float keep_ratio;          /* kappa in [0,1]; negative: kappa = 1 - MAS */
} orc_segment;

typedef struct {
    float tau;
    float tau_s;
    float lambda_s[ORC_NMOD];
    float lambda_t[ORC_NMOD];
    uint32_t flags;
} orc_params;

typedef struct {
    /* per token, indexed by global token id (segments in table order) */
    uint32_t* z;      /* inactive channel count */
    float* l1;        /* sum |x| */
    float* l2;        /* sum x^2 */
    float* info;      /* 1 - (lambda_s z + lambda_t e)/C */
    uint32_t* d;      /* activity-bit Hamming distance to the previous frame (0 if not temporal) */
    float* res;       /* sum (x_t - x_{t-1})^2 (0 if not temporal) */
    /* per frame of temporal segments (VIDEO, T >= 2, P > 0), frames in table order */
    uint64_t* dframe; /* D_t = sum_p d */
    float* sim;       /* Eq. 5 */
    float* gamma;     /* 1 - sim */
    /* per (request, modality), index r*4 + m */
    uint64_t* agg;    /* [R*4*4]: Ntok, Nsparse, Dsum, Qbits */
    float* rho;       /* Eq. 4 over the modality */
    float* temporal;  /* temporal term used in Eq. 7 (0 when absent) */
    float* beta;      /* modal softmax (Sec. 4.1.3) */
    float* mas;       /* Eq. 7 */
    uint8_t* present;
    /* selection */
    int32_t* k;       /* [n] keep count per segment */
    uint8_t* keep;    /* [Ntot] */
    int32_t* kept_idx;/* [Ntot]: segment s owns [tok_off_s, tok_off_s + N_s); its first k_s
                         entries are the kept local indices in ascending order, the rest -1 */
} orc_outputs;

/* ---------------------------------------------------------------- O1 widen */
/* Element c of a row as float: fp32 as is, bf16 by placing its 16 bits in the
 * high half of a float (exact). */
static float widen(const void* row, int dtype, int c)
{
    if (dtype == ORC_F32) return ((const float*)row)[c];
    uint32_t bits = (uint32_t)((const uint16_t*)row)[c] << 16;
    float v;
    memcpy(&v, &bits, sizeof v);
    return v;
}

static const void* row_ptr(const orc_segment* s, int64_t token)
{
    size_t esize = s->dtype == ORC_F32 ? 4 : 2;
    return (const char*)s->data + (size_t)token * (size_t)s->row_stride * esize;
}

static size_t elt_size(int dtype) { return dtype == ORC_F32 ? 4 : 2; }

/* ------------------------------------------------------------- O2 activity */
/* A channel is active unless its magnitude is at most tau. */
static int active(float v, float tau) { return !(fabsf(v) <= tau); }

/* ---------------------------------------------------------- O3 token stats */
/* Per token: active count a, L1 and L2 energy (double sums). The token's
 * importance (stand-in for one entry of M_spatial, Eq. 3) is a / C. */
static void token_stats(const void* row, int dtype, int C, float tau,
                        uint32_t* a, double* l1, double* l2)
{
    uint32_t cnt = 0;
    double s1 = 0.0, s2 = 0.0;
    for (int c = 0; c < C; ++c) {
        float v = widen(row, dtype, c);
        cnt += (uint32_t)active(v, tau);
        s1 += fabs((double)v);
        s2 += (double)v * (double)v;
    }
    *a = cnt;
    *l1 = s1;
    *l2 = s2;
}

/* ------------------------------------------------------ O4 temporal (Eq. 5) */
/* Bit-sampling LSH with every channel sampled: h_c(f) = active(f_c). The
 * number of differing hash values is the Hamming distance d of the two
 * activity patterns; res is the energy of the frame difference. A NULL
 * predecessor is the all-zero vector. */
static void temporal_pair(const void* cur, const void* prev, int dtype, int C, float tau,
                          uint32_t* d, double* res)
{
    uint32_t diff = 0;
    double e = 0.0;
    for (int c = 0; c < C; ++c) {
        float v = widen(cur, dtype, c);
        float u = prev ? widen(prev, dtype, c) : 0.0f;
        diff += (uint32_t)(active(v, tau) != active(u, tau));
        double delta = (double)v - (double)u;
        e += delta * delta;
    }
    *d = diff;
    *res = e;
}

/* Eq. 4: a token is sparse iff its importance a/C is below tau_s (strict). */
static int is_sparse(uint32_t a, int C, float tau_s)
{
    return (double)a / (double)C < (double)tau_s;
}

/* Eq. 5 for one frame: sim = (1/K) sum_k [h_k equal], K = P*C. */
static double frame_similarity(uint64_t D, int64_t P, int64_t C)
{
    return 1.0 - (double)D / (double)(P * C);
}

/* Sec. 4.1.3: softmax of the relevance logits over the modalities present in
 * the request. */
static void modal_softmax(const double alpha[ORC_NMOD], const int present[ORC_NMOD],
                          double beta[ORC_NMOD])
{
    double mx = -INFINITY;
    for (int m = 0; m < ORC_NMOD; ++m)
        if (present[m] && alpha[m] > mx) mx = alpha[m];
    double den = 0.0;
    for (int m = 0; m < ORC_NMOD; ++m)
        if (present[m]) den += exp(alpha[m] - mx);
    for (int m = 0; m < ORC_NMOD; ++m)
        beta[m] = present[m] ? exp(alpha[m] - mx) / den : 0.0;
}

/* Eq. 7: MAS = 1 - beta * (1 - lambda_s * rho - lambda_t * temporal), the
 * bracket clamped to [0, 1]; the temporal term only where the modality has one. */
static double mas_value(double beta, double lam_s, double rho, double lam_t, double tterm, int has_t)
{
    double inner = 1.0 - lam_s * rho;
    if (has_t) inner = inner - lam_t * tterm;
    if (inner < 0.0) inner = 0.0;
    if (inner > 1.0) inner = 1.0;
    return 1.0 - beta * inner;
}

static int is_temporal(const orc_segment* s)
{
    return s->modality == ORC_VIDEO && s->n_frames >= 2 && s->tokens_per_frame > 0;
}

/* Q24 fixed-point weight: round-to-nearest-even of lambda * 2^24. */
static uint64_t q24(float lambda)
{
    return (uint64_t)nearbyint((double)lambda * 16777216.0);
}

/* Keep count: k = min(N, ceil(kappa * N)). */
static int64_t keep_count(double kappa, int64_t N)
{
    double k = ceil(kappa * (double)N);
    if (k > (double)N) k = (double)N;
    if (k < 0.0) k = 0.0;
    return (int64_t)k;
}

typedef struct { uint64_t key; int64_t idx; } orc_pair;

static int pair_cmp(const void* a, const void* b)
{
    const orc_pair* x = (const orc_pair*)a;
    const orc_pair* y = (const orc_pair*)b;
    if (x->key != y->key) return x->key < y->key ? -1 : 1;
    if (x->idx != y->idx) return x->idx < y->idx ? -1 : 1;
    return 0;
}

/* Selection of one segment: sort (key, index) ascending, keep the first k. */
static int select_segment(const orc_segment* s, const orc_params* p, const uint32_t* z,
                          const uint32_t* d, int64_t k, uint8_t* keep, int32_t* kept_idx)
{
    int64_t N = (int64_t)s->n_frames * s->tokens_per_frame;
    int64_t C = s->hidden;
    uint64_t Ls = q24(p->lambda_s[s->modality]);
    uint64_t Lt = q24(p->lambda_t[s->modality]);
    int temporal = is_temporal(s);
    orc_pair* pairs = (orc_pair*)malloc(sizeof(orc_pair) * (size_t)(N > 0 ? N : 1));
    if (!pairs) return -1;
    for (int64_t i = 0; i < N; ++i) {
        uint64_t key = Ls * (uint64_t)z[i];
        if (temporal) key += Lt * (uint64_t)(C - (int64_t)d[i]);
        pairs[i].key = key;
        pairs[i].idx = i;
    }
    qsort(pairs, (size_t)N, sizeof(orc_pair), pair_cmp);
    for (int64_t i = 0; i < N; ++i) keep[i] = 0;
    for (int64_t j = 0; j < k; ++j) keep[pairs[j].idx] = 1;
    int64_t w = 0;
    for (int64_t i = 0; i < N; ++i)
        if (keep[i]) kept_idx[w++] = (int32_t)i;
    for (; w < N; ++w) kept_idx[w] = -1;
    free(pairs);
    return 0;
}

/* Selection over all segments from given per-token z, d and per-(request,
 * modality) MAS (used only by segments with a negative keep ratio). */
int orc_select(const orc_segment* segs, int n, int R, const orc_params* p,
               const uint32_t* z, const uint32_t* d, const float* mas,
               int32_t* k_out, uint8_t* keep, int32_t* kept_idx)
{
    int64_t off = 0;
    for (int s = 0; s < n; ++s) {
        const orc_segment* sg = &segs[s];
        int64_t N = (int64_t)sg->n_frames * sg->tokens_per_frame;
        double kappa;
        if (sg->keep_ratio < 0.0f) {
            if (!mas || sg->request < 0 || sg->request >= R) return -2;
            kappa = 1.0 - (double)mas[sg->request * ORC_NMOD + sg->modality];
        } else {
            kappa = (double)sg->keep_ratio;
        }
        int64_t k = keep_count(kappa, N);
        k_out[s] = (int32_t)k;
        if (select_segment(sg, p, z + off, d ? d + off : NULL, k, keep + off, kept_idx + off))
            return -1;
        off += N;
    }
    return 0;
}

/* The whole analysis, step by step. Returns 0 on success. */
int orc_run(const orc_segment* segs, int n, int R, const orc_params* p,
            const float* alpha, orc_outputs* o)
{
    /* O3/O4: per-token statistics and per-frame similarity */
    int64_t tok = 0, frame = 0;
    for (int s = 0; s < n; ++s) {
        const orc_segment* sg = &segs[s];
        int64_t T = sg->n_frames, P = sg->tokens_per_frame, C = sg->hidden;
        int temporal = is_temporal(sg);
        for (int64_t t = 0; t < T; ++t) {
            uint64_t D = 0;
            for (int64_t q = 0; q < P; ++q) {
                int64_t i = t * P + q, g = tok + i;
                const void* row = row_ptr(sg, i);
                uint32_t a;
                double l1, l2;
                token_stats(row, sg->dtype, (int)C, p->tau, &a, &l1, &l2);
                uint32_t z = (uint32_t)C - a;
                uint32_t dd = 0;
                double res = 0.0;
                if (temporal) {
                    const void* prev = t > 0 ? row_ptr(sg, i - P) : NULL;
                    temporal_pair(row, prev, sg->dtype, (int)C, p->tau, &dd, &res);
                    D += dd;
                }
                double lam_s = (double)p->lambda_s[sg->modality];
                double lam_t = (double)p->lambda_t[sg->modality];
                double redundant = lam_s * (double)z;
                if (temporal) redundant += lam_t * (double)((uint32_t)C - dd);
                o->z[g] = z;
                o->l1[g] = (float)l1;
                o->l2[g] = (float)l2;
                o->info[g] = (float)(1.0 - redundant / (double)C);
                o->d[g] = dd;
                o->res[g] = (float)res;
            }
            if (temporal) {
                double sim = frame_similarity(D, P, C);
                o->dframe[frame + t] = D;
                o->sim[frame + t] = (float)sim;
                o->gamma[frame + t] = (float)(1.0 - sim);
            }
        }
        if (temporal) frame += T;
        tok += T * P;
    }

    /* O5: integer aggregates per (request, modality) */
    for (int i = 0; i < R * ORC_NMOD * 4; ++i) o->agg[i] = 0;
    tok = 0;
    frame = 0;
    for (int s = 0; s < n; ++s) {
        const orc_segment* sg = &segs[s];
        int64_t T = sg->n_frames, P = sg->tokens_per_frame, C = sg->hidden, N = T * P;
        uint64_t* ag = &o->agg[(sg->request * ORC_NMOD + sg->modality) * 4];
        ag[0] += (uint64_t)N;
        for (int64_t i = 0; i < N; ++i) {
            uint32_t a = (uint32_t)C - o->z[tok + i];
            ag[1] += (uint64_t)is_sparse(a, (int)C, p->tau_s);
        }
        if (is_temporal(sg)) {
            for (int64_t t = 1; t < T; ++t) ag[2] += o->dframe[frame + t];
            ag[3] += (uint64_t)((T - 1) * P * C);
            frame += T;
        }
        tok += N;
    }

    /* O6/O7: modal softmax and MAS per request */
    for (int r = 0; r < R; ++r) {
        int present[ORC_NMOD];
        double al[ORC_NMOD], beta[ORC_NMOD];
        for (int m = 0; m < ORC_NMOD; ++m) {
            present[m] = o->agg[(r * ORC_NMOD + m) * 4 + 0] > 0;
            al[m] = alpha ? (double)alpha[r * ORC_NMOD + m] : 0.0;
        }
        modal_softmax(al, present, beta);
        for (int m = 0; m < ORC_NMOD; ++m) {
            int x = r * ORC_NMOD + m;
            const uint64_t* ag = &o->agg[x * 4];
            if (!present[m]) {
                o->rho[x] = o->temporal[x] = o->beta[x] = o->mas[x] = 0.0f;
                o->present[x] = 0;
                continue;
            }
            double rho = (double)ag[1] / (double)ag[0];
            int has_t = ag[3] > 0;
            double tterm = 0.0;
            if (has_t) {
                double gamma_avg = (double)ag[2] / (double)ag[3];
                tterm = (p->flags & ORC_FLAG_TEMPORAL_LITERAL) ? gamma_avg : 1.0 - gamma_avg;
            }
            double mas = mas_value(beta[m], (double)p->lambda_s[m], rho,
                                   (double)p->lambda_t[m], tterm, has_t);
            o->rho[x] = (float)rho;
            o->temporal[x] = (float)tterm;
            o->beta[x] = (float)beta[m];
            o->mas[x] = (float)mas;
            o->present[x] = 1;
        }
    }

    /* O8-O10: keys, keep counts, selection */
    return orc_select(segs, n, R, p, o->z, o->d, o->mas, o->k, o->keep, o->kept_idx);
}

/* O11: compaction, a byte copy of each kept row into packed per-segment
 * outputs: segment s's rows go to out + out_off[s], one after another. */
void orc_compact(const orc_segment* segs, int n, const int32_t* k, const int32_t* kept_idx,
                 void* out, const int64_t* out_off)
{
    int64_t tok = 0;
    for (int s = 0; s < n; ++s) {
        const orc_segment* sg = &segs[s];
        int64_t N = (int64_t)sg->n_frames * sg->tokens_per_frame;
        size_t row_bytes = (size_t)sg->hidden * elt_size(sg->dtype);
        char* dst = (char*)out + out_off[s];
        for (int64_t j = 0; j < k[s]; ++j)
            memcpy(dst + (size_t)j * row_bytes, row_ptr(sg, kept_idx[tok + j]), row_bytes);
        tok += N;
    }
}

/* Exposed single steps, for pinning each step on its own. */
void orc_token_stats(const void* row, int dtype, int C, float tau, uint32_t* a, double* l1, double* l2)
{
    token_stats(row, dtype, C, tau, a, l1, l2);
}

void orc_temporal_pair(const void* cur, const void* prev, int dtype, int C, float tau,
                       uint32_t* d, double* res)
{
    temporal_pair(cur, prev, dtype, C, tau, d, res);
}

int orc_is_sparse(uint32_t a, int C, float tau_s) { return is_sparse(a, C, tau_s); }

void orc_modal_softmax(const double* alpha, const int* present, double* beta)
{
    modal_softmax(alpha, present, beta);
}

double orc_mas_value(double beta, double lam_s, double rho, double lam_t, double tterm, int has_t)
{
    return mas_value(beta, lam_s, rho, lam_t, tterm, has_t);
}

int64_t orc_keep_count(double kappa, int64_t N) { return keep_count(kappa, N); }

uint64_t orc_q24(float lambda) { return q24(lambda); }
