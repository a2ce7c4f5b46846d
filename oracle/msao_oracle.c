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
 *        Ls*z*E + Lt*(E - d)*C   with Ls = rne(lambda_s * 2^24), Lt likewise
 *    and E the bits d compares per token (E = C for bit sampling), i.e.
 *    C E (Ls z / C + Lt e / E) with e = E - d;
 *    the keep count is k = min(N, ceil(kappa * N)) and the k smallest
 *    (key, index) pairs of each segment are kept, ties by ascending index;
 *    with the per-frame scope flag each frame of P tokens is its own
 *    selection, k_f = min(P, ceil(kappa * P)) tokens per frame;
 *  - the SimHash variant of Eq. 5 hashes each token with K caller
 *    hyperplanes r_k: bit k is 1 iff r_k . f >= 0 (Charikar's hash); frame
 *    0 is compared with the all-zero frame, whose bits are all 1. Run with
 *    SimHash (orc_run_simhash), its d (E = K bits per token) replaces bit
 *    sampling's in every later step: D_t, sim, Qbits, the temporal term,
 *    informativeness and the selection key.
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
enum { ORC_FLAG_TEMPORAL_LITERAL = 1, ORC_FLAG_SELECT_PER_FRAME = 2 };

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
    float* info;      /* 1 - (lambda_s z/C + lambda_t e/E), e = E - d */
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

/* Eq. 5 for one frame: sim = (1/K) sum_k [h_k equal] over its K = P*E hash
 * functions (E per token: C activity bits, or K SimHash bits). */
static double frame_similarity(uint64_t D, int64_t P, int64_t E)
{
    return 1.0 - (double)D / (double)(P * E);
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

/* Selection among tokens [i0, i0 + n) of a segment: sort (key, index)
 * ascending, keep the first k (keep flags set for the range only). E is the
 * number of bits d compares per token (C for bit sampling, K for SimHash);
 * the key is C E 2^24 (lambda_s z / C + lambda_t (E - d) / E) with the
 * weights in Q24, an exact integer (the temporal term only for temporal
 * segments). */
static int select_range(const orc_segment* s, const orc_params* p, const uint32_t* z,
                        const uint32_t* d, int64_t E, int64_t i0, int64_t n, int64_t k, uint8_t* keep)
{
    int64_t C = s->hidden;
    uint64_t Ls = q24(p->lambda_s[s->modality]);
    uint64_t Lt = q24(p->lambda_t[s->modality]);
    int temporal = is_temporal(s);
    orc_pair* pairs = (orc_pair*)malloc(sizeof(orc_pair) * (size_t)(n > 0 ? n : 1));
    if (!pairs) return -1;
    for (int64_t j = 0; j < n; ++j) {
        int64_t i = i0 + j;
        uint64_t key = Ls * (uint64_t)z[i] * (uint64_t)E;
        if (temporal) key += Lt * (uint64_t)(E - (int64_t)d[i]) * (uint64_t)C;
        pairs[j].key = key;
        pairs[j].idx = i;
    }
    qsort(pairs, (size_t)n, sizeof(orc_pair), pair_cmp);
    for (int64_t j = 0; j < n; ++j) keep[i0 + j] = 0;
    for (int64_t j = 0; j < k; ++j) keep[pairs[j].idx] = 1;
    free(pairs);
    return 0;
}

typedef struct { double m; int64_t idx; } orc_imp_pair;

/* The more important token first: larger importance, then smaller index. */
static int imp_cmp(const void* a, const void* b)
{
    const orc_imp_pair* x = (const orc_imp_pair*)a;
    const orc_imp_pair* y = (const orc_imp_pair*)b;
    if (x->m != y->m) return x->m > y->m ? -1 : 1;
    if (x->idx != y->idx) return x->idx < y->idx ? -1 : 1;
    return 0;
}

/* Selection among tokens [i0, i0 + n) of a segment by a learned importance
 * (Sec. 4.1.1: the patches of low Eq. 3 importance are pruned): the k of
 * largest importance, ties by ascending index; an importance that is NaN or
 * not above 0 counts as 0, the least important. */
static int select_range_importance(const double* imp, int64_t i0, int64_t n, int64_t k, uint8_t* keep)
{
    orc_imp_pair* pairs = (orc_imp_pair*)malloc(sizeof(orc_imp_pair) * (size_t)(n > 0 ? n : 1));
    if (!pairs) return -1;
    for (int64_t j = 0; j < n; ++j) {
        const double m = imp[i0 + j];
        pairs[j].m = (m > 0.0) ? m : 0.0;  /* NaN compares false */
        pairs[j].idx = i0 + j;
    }
    qsort(pairs, (size_t)n, sizeof(orc_imp_pair), imp_cmp);
    for (int64_t j = 0; j < n; ++j) keep[i0 + j] = 0;
    for (int64_t j = 0; j < k; ++j) keep[pairs[j].idx] = 1;
    free(pairs);
    return 0;
}

/* Selection of one segment with keep ratio kappa: the whole segment, or
 * (per-frame scope) each of its T frames of P tokens on its own. imp (the
 * segment's tokens' learned importance) or NULL (the redundancy key). Kept
 * indices ascending, then -1. Returns the keep count. */
static int64_t select_segment(const orc_segment* s, const orc_params* p, const uint32_t* z,
                              const uint32_t* d, int64_t E, double kappa, const double* imp, uint8_t* keep,
                              int32_t* kept_idx)
{
    int64_t T = s->n_frames, P = s->tokens_per_frame, N = T * P, k = 0;
    if (p->flags & ORC_FLAG_SELECT_PER_FRAME) {
        int64_t kf = keep_count(kappa, P);
        for (int64_t t = 0; t < T; ++t) {
            const int rc = imp ? select_range_importance(imp, t * P, P, kf, keep)
                               : select_range(s, p, z, d, E, t * P, P, kf, keep);
            if (rc) return -1;
        }
        k = kf * T;
    } else {
        k = keep_count(kappa, N);
        const int rc = imp ? select_range_importance(imp, 0, N, k, keep) : select_range(s, p, z, d, E, 0, N, k, keep);
        if (rc) return -1;
    }
    int64_t w = 0;
    for (int64_t i = 0; i < N; ++i)
        if (keep[i]) kept_idx[w++] = (int32_t)i;
    for (; w < N; ++w) kept_idx[w] = -1;
    return k;
}

/* Selection over all segments from per-token z, d (E[s]: bits compared per
 * token of segment s) and per-(request, modality) MAS (used only by segments
 * with a negative keep ratio). by_imp (may be NULL): segments s with
 * by_imp[s] set are ranked by the per-token importance imp instead. */
static int select_all(const orc_segment* segs, int n, int R, const orc_params* p,
                      const uint32_t* z, const uint32_t* d, const int64_t* E, const float* mas,
                      const double* imp, const int* by_imp, int32_t* k_out, uint8_t* keep, int32_t* kept_idx)
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
        const double* im = (by_imp && by_imp[s]) ? imp + off : NULL;
        int64_t k = select_segment(sg, p, z + off, d ? d + off : NULL, E[s], kappa, im, keep + off, kept_idx + off);
        if (k < 0) return -1;
        k_out[s] = (int32_t)k;
        off += N;
    }
    return 0;
}

/* Selection over all segments from given per-token z, d (activity-bit
 * distances, E = C) and per-(request, modality) MAS. */
int orc_select(const orc_segment* segs, int n, int R, const orc_params* p,
               const uint32_t* z, const uint32_t* d, const float* mas,
               int32_t* k_out, uint8_t* keep, int32_t* kept_idx)
{
    int64_t* E = (int64_t*)malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    if (!E) return -1;
    for (int s = 0; s < n; ++s) E[s] = segs[s].hidden;
    int rc = select_all(segs, n, R, p, z, d, E, mas, NULL, NULL, k_out, keep, kept_idx);
    free(E);
    return rc;
}

/* SimHash hyperplanes of one segment (the SimHash variant of Eq. 5, below). */
typedef struct {
    const void* planes; /* [bits][hidden] in the segment's dtype: hyperplane r_k is row k */
    int32_t bits;       /* K hash functions per token, 1..64 */
} orc_simhash;

static uint64_t simhash_token(const void* row, const void* planes, int dtype, int C, int K);
static uint32_t popcount64(uint64_t v);

/* The whole analysis, step by step. h == NULL: Eq. 5 by bit sampling over
 * the activity bits (E = C bits compared per token). Otherwise the temporal
 * segments hash with SimHash (h[s], E = K): their signatures go to sig, and
 * d is the number of signature bits that differ from the same patch in the
 * previous frame (frame 0: from the all-zero frame, all bits 1); every step
 * after Eq. 5 then uses that d and E. Returns 0 on success. */
static int run_impl(const orc_segment* segs, int n, int R, const orc_params* p,
                    const float* alpha, const orc_simhash* h, uint64_t* sig, orc_outputs* o)
{
    int64_t* E = (int64_t*)malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    if (!E) return -1;
    /* O3/O4: per-token statistics and per-frame similarity */
    int64_t tok = 0, frame = 0;
    for (int s = 0; s < n; ++s) {
        const orc_segment* sg = &segs[s];
        int64_t T = sg->n_frames, P = sg->tokens_per_frame, C = sg->hidden;
        int temporal = is_temporal(sg);
        int hashed = temporal && h != NULL;
        E[s] = C;
        uint64_t all = 0;
        if (hashed) {
            if (!h[s].planes || h[s].bits < 1 || h[s].bits > 64) {
                free(E);
                return -1;
            }
            E[s] = h[s].bits;
            all = h[s].bits == 64 ? ~(uint64_t)0 : (((uint64_t)1 << h[s].bits) - 1);
            for (int64_t i = 0; i < T * P; ++i)
                sig[tok + i] = simhash_token(row_ptr(sg, i), h[s].planes, sg->dtype, (int)C, h[s].bits);
        } else if (sig) {
            for (int64_t i = 0; i < T * P; ++i) sig[tok + i] = 0;
        }
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
                    if (hashed) dd = popcount64(sig[g] ^ (t > 0 ? sig[g - P] : all));
                    D += dd;
                }
                double lam_s = (double)p->lambda_s[sg->modality];
                double lam_t = (double)p->lambda_t[sg->modality];
                double redundant = lam_s * (double)z / (double)C;
                if (temporal) redundant += lam_t * (double)((uint32_t)E[s] - dd) / (double)E[s];
                o->z[g] = z;
                o->l1[g] = (float)l1;
                o->l2[g] = (float)l2;
                o->info[g] = (float)(1.0 - redundant);
                o->d[g] = dd;
                o->res[g] = (float)res;
            }
            if (temporal) {
                double sim = frame_similarity(D, P, E[s]);
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
            ag[3] += (uint64_t)((T - 1) * P * E[s]);
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
    int rc = select_all(segs, n, R, p, o->z, o->d, E, o->mas, NULL, NULL, o->k, o->keep, o->kept_idx);
    free(E);
    return rc;
}

/* The whole analysis with bit sampling in Eq. 5. Returns 0 on success. */
int orc_run(const orc_segment* segs, int n, int R, const orc_params* p,
            const float* alpha, orc_outputs* o)
{
    return run_impl(segs, n, R, p, alpha, NULL, NULL, o);
}

/* The whole analysis with SimHash in Eq. 5 (h[s] for every temporal
 * segment; sig [Ntot] receives the signatures, 0 outside temporal segments).
 * Returns 0 on success, -1 for a missing or invalid hash. */
int orc_run_simhash(const orc_segment* segs, int n, int R, const orc_params* p, const orc_simhash* h,
                    const float* alpha, uint64_t* sig, orc_outputs* o)
{
    if (!h || !sig) return -1;
    return run_impl(segs, n, R, p, alpha, h, sig, o);
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

/* ==================================================================
 * Learned probe heads with caller weights (Sec. 4.1.1 Eq. 3 and
 * Sec. 4.1.3 Eq. 6), in place of the parameter-free stand-ins.
 * ================================================================ */

typedef struct {
    const void* weight; /* [hidden], segment dtype: the 1x1 convolution to one logit; NULL: no head */
    float bias;
    int32_t grid_w;     /* patches per grid row of a frame; grid (P / grid_w) x grid_w; 0: one row */
    int32_t pool;       /* odd AvgPool window; 1: none */
} orc_head;

#define ORC_DESC 8      /* entries of the modality descriptor z_m */

typedef struct {
    const float* w1;    /* [hidden][prompt_dim + ORC_DESC], row-major */
    const float* b1;    /* [hidden] */
    const float* w2;    /* [hidden] */
    float b2;
    int32_t hidden, prompt_dim;
    const float* prompt; /* [R][prompt_dim]: the prompt embedding p of each request */
} orc_mlp;

static double sigmoid(double v) { return 1.0 / (1.0 + exp(-v)); }

/* Eq. 3 for one frame of a segment with a head (P tokens from token t0, on
 * an H x W grid, token q at row q / W, column q % W):
 *     M = sigmoid(Conv1x1(AvgPool(F))),  Conv1x1(f) = w . f + b.
 * The window of a patch is the pool x pool square around it, cut to the grid;
 * its average is over the patches inside. The convolution is linear, so the
 * average of the projections w . f over the window equals the projection of
 * the averaged features. */
static void head_frame(const orc_segment* s, const orc_head* h, int64_t t0, double* M)
{
    const int64_t P = s->tokens_per_frame, C = s->hidden;
    const int64_t W = h->grid_w > 0 ? h->grid_w : P, H = P / W, r = (h->pool - 1) / 2;
    double* y = (double*)malloc(sizeof(double) * (size_t)(P > 0 ? P : 1));
    for (int64_t q = 0; q < P; ++q) {
        const void* row = row_ptr(s, t0 + q);
        double acc = 0.0;
        for (int64_t c = 0; c < C; ++c)
            acc += (double)widen(h->weight, s->dtype, (int)c) * (double)widen(row, s->dtype, (int)c);
        y[q] = acc;
    }
    for (int64_t q = 0; q < P; ++q) {
        const int64_t i = q / W, j = q % W;
        double sum = 0.0;
        int64_t cnt = 0;
        for (int64_t ii = i - r; ii <= i + r; ++ii)
            for (int64_t jj = j - r; jj <= j + r; ++jj)
                if (ii >= 0 && ii < H && jj >= 0 && jj < W) {
                    sum += y[ii * W + jj];
                    cnt += 1;
                }
        M[q] = sigmoid(sum / (double)cnt + (double)h->bias);
    }
    free(y);
}

/* The analysis of orc_run with learned heads:
 *  - importance[g] of every token: Eq. 3 where the segment has a head, its
 *    activity density a / C otherwise;
 *  - Nsparse of Eq. 4 counts importance < tau_s (the density test of orc_run
 *    where there is no head);
 *  - per (request, modality) the descriptor z_m (desc[x * 8 + 0..7]):
 *    1, rho (Eq. 4), sum a / sum C, sum L1 / sum C, sqrt(sum L2 / sum C),
 *    the temporal term of Eq. 7 (0 if none), 1 if that term exists,
 *    ln(1 + Ntok) / 16, the sums over the modality's tokens (L1, L2 as the
 *    per-token float values);
 *  - Eq. 6: alpha = w2 . relu(W1 [p; z_m] + b1) + b2 (alpha = 0 without an
 *    MLP), then the softmax over the modalities present and Eq. 7;
 *  - the selection (Sec. 4.1.1 pruning): a segment with a head keeps its k
 *    tokens of largest Eq. 3 importance M (ties by ascending index, a NaN M
 *    as 0); a segment without one keeps the k smallest (key, index) pairs of
 *    orc_run; k from the keep ratio, or from this MAS when it is negative;
 *    the per-frame scope as in orc_run.
 * heads may be NULL (no head anywhere), heads[s].weight NULL for no head on
 * segment s. o receives the token, frame and request outputs of orc_run with
 * agg[.][1], rho, beta and mas replaced, and the selection above. */
int orc_run_learned(const orc_segment* segs, int n, int R, const orc_params* p, const orc_head* heads,
                    const orc_mlp* mlp, orc_outputs* o, double* importance, double* alpha_out, double* desc)
{
    int rc = orc_run(segs, n, R, p, NULL, o);
    if (rc) return rc;
    const int X = R * ORC_NMOD;
    double* A = (double*)calloc((size_t)(X > 0 ? X : 1), sizeof(double));
    double* CC = (double*)calloc((size_t)(X > 0 ? X : 1), sizeof(double));
    double* L1 = (double*)calloc((size_t)(X > 0 ? X : 1), sizeof(double));
    double* L2 = (double*)calloc((size_t)(X > 0 ? X : 1), sizeof(double));
    for (int x = 0; x < X; ++x) o->agg[x * 4 + 1] = 0;
    int64_t tok = 0;
    for (int s = 0; s < n; ++s) {
        const orc_segment* sg = &segs[s];
        const int64_t T = sg->n_frames, P = sg->tokens_per_frame, C = sg->hidden, N = T * P;
        const int x = sg->request * ORC_NMOD + sg->modality;
        const orc_head* h = heads && heads[s].weight ? &heads[s] : NULL;
        double* M = (double*)malloc(sizeof(double) * (size_t)(P > 0 ? P : 1));
        for (int64_t t = 0; t < T; ++t) {
            if (h) head_frame(sg, h, t * P, M);
            for (int64_t q = 0; q < P; ++q) {
                const int64_t g = tok + t * P + q;
                const uint32_t a = (uint32_t)C - o->z[g];
                if (h) {
                    importance[g] = M[q];
                    o->agg[x * 4 + 1] += M[q] < (double)p->tau_s;
                } else {
                    importance[g] = (double)a / (double)C;
                    o->agg[x * 4 + 1] += (uint64_t)is_sparse(a, (int)C, p->tau_s);
                }
                A[x] += (double)a;
                CC[x] += (double)C;
                L1[x] += (double)o->l1[g];
                L2[x] += (double)o->l2[g];
            }
        }
        free(M);
        tok += N;
    }
    for (int r = 0; r < R; ++r) {
        int present[ORC_NMOD];
        double al[ORC_NMOD], beta[ORC_NMOD], rho[ORC_NMOD], tterm[ORC_NMOD];
        int has_t[ORC_NMOD];
        for (int m = 0; m < ORC_NMOD; ++m) {
            const int x = r * ORC_NMOD + m;
            const uint64_t* ag = &o->agg[x * 4];
            present[m] = ag[0] > 0;
            rho[m] = present[m] ? (double)ag[1] / (double)ag[0] : 0.0;
            has_t[m] = ag[3] > 0;
            tterm[m] = 0.0;
            if (has_t[m]) {
                const double gamma_avg = (double)ag[2] / (double)ag[3];
                tterm[m] = (p->flags & ORC_FLAG_TEMPORAL_LITERAL) ? gamma_avg : 1.0 - gamma_avg;
            }
            double* z = &desc[x * ORC_DESC];
            for (int k = 0; k < ORC_DESC; ++k) z[k] = 0.0;
            if (present[m]) {
                z[0] = 1.0;
                z[1] = rho[m];
                z[2] = A[x] / CC[x];
                z[3] = L1[x] / CC[x];
                z[4] = sqrt(L2[x] / CC[x]);
                z[5] = tterm[m];
                z[6] = has_t[m] ? 1.0 : 0.0;
                z[7] = log(1.0 + (double)ag[0]) / 16.0;
            }
            al[m] = 0.0;
            if (mlp && present[m]) {
                const int in = mlp->prompt_dim + ORC_DESC;
                double out = (double)mlp->b2;
                for (int j = 0; j < mlp->hidden; ++j) {
                    double hsum = (double)mlp->b1[j];
                    for (int k = 0; k < in; ++k) {
                        const double v = k < mlp->prompt_dim ? (double)mlp->prompt[r * mlp->prompt_dim + k]
                                                             : z[k - mlp->prompt_dim];
                        hsum += (double)mlp->w1[j * in + k] * v;
                    }
                    out += (double)mlp->w2[j] * (hsum > 0.0 ? hsum : 0.0);
                }
                al[m] = out;
            }
            alpha_out[x] = al[m];
        }
        modal_softmax(al, present, beta);
        for (int m = 0; m < ORC_NMOD; ++m) {
            const int x = r * ORC_NMOD + m;
            if (!present[m]) continue;
            o->rho[x] = (float)rho[m];
            o->beta[x] = (float)beta[m];
            o->mas[x] = (float)mas_value(beta[m], (double)p->lambda_s[m], rho[m], (double)p->lambda_t[m], tterm[m],
                                         has_t[m]);
        }
    }
    free(A);
    free(CC);
    free(L1);
    free(L2);
    /* selection with the learned MAS; segments with a head by importance */
    int64_t* E = (int64_t*)malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    int* by_imp = (int*)calloc((size_t)(n > 0 ? n : 1), sizeof(int));
    if (!E || !by_imp) {
        free(E);
        free(by_imp);
        return -1;
    }
    for (int s = 0; s < n; ++s) {
        E[s] = segs[s].hidden;
        by_imp[s] = heads && heads[s].weight ? 1 : 0;
    }
    rc = select_all(segs, n, R, p, o->z, o->d, E, o->mas, importance, by_imp, o->k, o->keep, o->kept_idx);
    free(E);
    free(by_imp);
    return rc;
}

/* ==================================================================
 * SimHash variant of Eq. 5 (Sec. 4.1.2): Charikar's random-hyperplane
 * hash in place of bit sampling over the activity bits.
 * ================================================================ */

/* Signature of one token: bit k is 1 iff r_k . f >= 0, the dot product
 * summed in double over the channels in order (NaN compares false: 0). */
static uint64_t simhash_token(const void* row, const void* planes, int dtype, int C, int K)
{
    uint64_t sig = 0;
    for (int k = 0; k < K; ++k) {
        const void* r = (const char*)planes + (size_t)k * (size_t)C * elt_size(dtype);
        double y = 0.0;
        for (int c = 0; c < C; ++c) y += (double)widen(r, dtype, c) * (double)widen(row, dtype, c);
        if (y >= 0.0) sig |= (uint64_t)1 << k;
    }
    return sig;
}

static uint32_t popcount64(uint64_t v)
{
    uint32_t n = 0;
    for (; v; v &= v - 1) ++n;
    return n;
}

/* Eq. 5 with K hyperplanes per token (K P hash functions per frame):
 *   sig[g]  the token's signature (0 outside temporal segments);
 *   d[g]    the number of its K bits that differ from the same patch in the
 *           previous frame (frame 0: from the all-zero frame, all bits 1);
 *   D_t = sum_p d, sim_t = 1 - D_t / (P K), gamma_t = 1 - sim_t;
 *   per (request, modality) x: dq[2x] = sum of D_t over frames 1..T-1,
 *   dq[2x+1] = (T - 1) P K, and the temporal term of Eq. 7 (1 - Dsum/Qbits,
 *   or Dsum/Qbits with the literal flag; 0 where there is none).
 * Every temporal segment needs planes (else -1). */
int orc_temporal_simhash(const orc_segment* segs, int n, int R, const orc_params* p, const orc_simhash* h,
                         uint64_t* sig, uint32_t* d, uint64_t* dframe, float* sim, float* gamma, uint64_t* dq,
                         float* temporal)
{
    for (int i = 0; i < R * ORC_NMOD * 2; ++i) dq[i] = 0;
    int64_t tok = 0, frame = 0;
    for (int s = 0; s < n; ++s) {
        const orc_segment* sg = &segs[s];
        int64_t T = sg->n_frames, P = sg->tokens_per_frame, N = T * P;
        if (!is_temporal(sg)) {
            for (int64_t i = 0; i < N; ++i) {
                sig[tok + i] = 0;
                d[tok + i] = 0;
            }
            tok += N;
            continue;
        }
        if (!h || !h[s].planes || h[s].bits < 1 || h[s].bits > 64) return -1;
        const int K = h[s].bits;
        const uint64_t all = K == 64 ? ~(uint64_t)0 : (((uint64_t)1 << K) - 1);
        for (int64_t i = 0; i < N; ++i)
            sig[tok + i] = simhash_token(row_ptr(sg, i), h[s].planes, sg->dtype, sg->hidden, K);
        uint64_t* x = &dq[(sg->request * ORC_NMOD + sg->modality) * 2];
        for (int64_t t = 0; t < T; ++t) {
            uint64_t D = 0;
            for (int64_t q = 0; q < P; ++q) {
                const int64_t g = tok + t * P + q;
                const uint64_t prev = t > 0 ? sig[g - P] : all;
                d[g] = popcount64(sig[g] ^ prev);
                D += d[g];
            }
            const double sm = 1.0 - (double)D / (double)(P * K);
            dframe[frame + t] = D;
            sim[frame + t] = (float)sm;
            gamma[frame + t] = (float)(1.0 - sm);
            if (t >= 1) x[0] += D;
        }
        x[1] += (uint64_t)((T - 1) * P * K);
        frame += T;
        tok += N;
    }
    for (int x = 0; x < R * ORC_NMOD; ++x) {
        temporal[x] = 0.0f;
        if (dq[2 * x + 1] == 0) continue;
        const double gamma_avg = (double)dq[2 * x] / (double)dq[2 * x + 1];
        temporal[x] = (float)((p->flags & ORC_FLAG_TEMPORAL_LITERAL) ? gamma_avg : 1.0 - gamma_avg);
    }
    return 0;
}
