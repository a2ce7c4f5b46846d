/*
 * msao.h -- C ABI of the MI355X (gfx950) implementation of MSAO's
 * fine-grained sparsity analysis: per-token activation-sparsity statistics,
 * the temporal-redundancy term between consecutive video frames, per-modality
 * aggregation into MAS (Modal Activation Sparsity), and the MAS-guided
 * selection and compaction of the tokens that are kept. Also the decoding
 * side of its speculative offloading (Sec. 4.2): the draft model's
 * confidence per generation step on the GPU (Eq. 9-10), and on the host the
 * latency model (Eq. 8, 12-14) and Algorithm 1's threshold logic.
 *
 * Paper: "MSAO" (arXiv 2604.02945). Sec. 4.1 defines the probing module:
 * spatial sparsity (Sec. 4.1.1, Eq. 3-4), temporal sparsity (Sec. 4.1.2,
 * Eq. 5), modal sparsity (Sec. 4.1.3, Eq. 6 and the softmax after it) and
 * MAS (Sec. 4.1.4, Eq. 7). Eq. 11's last constraint (retained proportion at
 * least 1 - MAS) sets the MAS-guided keep ratio; Sec. 4.1.1 prunes the patches
 * of low importance.
 *
 * Stand-ins for what the paper leaves open (all exact and parameter-free):
 *  - importance of a token = fraction of its C channels that are active, a
 *    channel being active iff NOT(|x| <= tau) (NaN is active, -0 is not);
 *  - the LSH of Eq. 5 = bit sampling over the activity bits, every channel
 *    sampled once; frame 0 is compared with an all-zero frame and left out of
 *    the averages; a clip with one frame has no temporal term;
 *  - the temporal term of Eq. 7 is the redundancy 1 - gamma_avg, or gamma_avg
 *    as printed under MSAO_FLAG_TEMPORAL_LITERAL; the bracket of Eq. 7 is
 *    clamped to [0, 1];
 *  - relevance logits alpha (Eq. 6) are supplied by the caller (0 if absent);
 *  - a token's redundancy key is the exact integer
 *        key = Ls*z + Lt*e,  Ls = rne(lambda_s[m] * 2^24), Lt = rne(lambda_t[m] * 2^24),
 *    z = inactive channels, e = C - d (channels whose activity equals the
 *    previous frame's; temporal segments only, else the term is absent);
 *    each segment keeps its k smallest (key, index) pairs, ties by ascending
 *    index, with k = min(N, ceil(kappa * N)) computed in double from the
 *    float keep ratio kappa (kappa = 1 - MAS of the segment's request and
 *    modality when the keep ratio is negative).
 *
 * Conventions
 *  - Every data pointer is HIP device memory owned by the caller unless it is
 *    marked "host". The library allocates no device memory: scratch comes
 *    from the caller's workspace (size from msao_workspace_size), except for
 *    msao_run_noalloc, which uses the library's own static array. The context
 *    owns host state only (pinned staging for the small per-call tables, HIP
 *    events, the last error message).
 *  - Calls are asynchronous: they enqueue on `stream` (a hipStream_t; NULL is
 *    the null stream) and return; outputs are valid once the caller has
 *    synchronised with that stream. Pointers are not retained after return.
 *  - Validation runs entirely on the host before anything is enqueued: an
 *    invalid call returns a specific status, writes nothing and records a
 *    message for msao_last_error. Runtime and launch failures return
 *    MSAO_ERR_HIP.
 *  - One context per concurrently used stream (a context is not thread-safe).
 *  - Token t*P + p of a segment is row (t*P + p) of its data; global token ids
 *    concatenate the segments in table order. Per-token outputs are indexed by
 *    global token id. Frames are numbered over the temporal segments only
 *    (VIDEO, n_frames >= 2, tokens_per_frame > 0), in table order.
 *    Per-(request, modality) outputs are indexed r*4 + m.
 *  - Layout: data and row_stride*element_size must be multiples of 16 bytes;
 *    hidden a multiple of 8 (bf16) or 4 (fp32), at most 65536; n_frames > 1
 *    only for VIDEO; total tokens below 2^31.
 */
#ifndef MSAO_H
#define MSAO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MSAO_NUM_MODALITIES 4
#define MSAO_MAX_HIDDEN 65536

typedef enum {
    MSAO_OK = 0,
    MSAO_ERR_INVALID_ARG = 1,   /* bad pointer, size, enum value, parameter or output set */
    MSAO_ERR_ALIGNMENT = 2,     /* data, row pitch or output not aligned as required */
    MSAO_ERR_WORKSPACE = 3,     /* workspace missing, not 256-byte aligned or too small */
    MSAO_ERR_UNSUPPORTED = 4,   /* valid request outside what the library handles (sizes, pitches) */
    MSAO_ERR_HIP = 5            /* a HIP runtime call or a kernel launch failed */
} msao_status;

typedef enum { MSAO_TEXT = 0, MSAO_IMAGE = 1, MSAO_VIDEO = 2, MSAO_AUDIO = 3 } msao_modality;
typedef enum { MSAO_F32 = 0, MSAO_BF16 = 1 } msao_dtype;

/* Eq. 7 takes gamma_avg itself as the temporal term (default: 1 - gamma_avg). */
#define MSAO_FLAG_TEMPORAL_LITERAL 1u
/* Per-frame selection scope (the alternative to one selection per segment
 * that Sec. 4.1.1's pruning leaves open): every frame of a segment with
 * T >= 2 keeps its own k_f = min(P, ceil(kappa P)) tokens, the k_f smallest
 * (key, index) pairs of the frame (a MAS-guided kappa = 1 - MAS of the
 * segment's request and modality for every frame); kept_count = T k_f and
 * the kept indices stay ascending over the segment. */
#define MSAO_FLAG_SELECT_PER_FRAME 2u

typedef struct msao_ctx msao_ctx;

/* One modality-tagged activation tensor of one request (Sec. 3 Eq. 1-2, the
 * early-layer features F of Eq. 3 and f_t of Eq. 5). */
typedef struct {
    const void* data;          /* device; row i at data + i*row_stride elements */
    int64_t row_stride;        /* elements between consecutive rows, >= hidden */
    int32_t request;           /* 0 .. n_requests-1 */
    int32_t modality;          /* msao_modality */
    int32_t n_frames;          /* T >= 1 (> 1 only for VIDEO) */
    int32_t tokens_per_frame;  /* P >= 0; the segment has N = T*P tokens */
    int32_t hidden;            /* C */
    int32_t dtype;             /* msao_dtype */
    float keep_ratio;          /* kappa in [0, 1]; negative: MAS-guided, kappa = 1 - MAS */
} msao_segment;

/* Thresholds and weights (Sec. 5.1.4 defaults from msao_default_params). */
typedef struct {
    float tau;                          /* channel activity threshold, >= 0, finite (-0 is 0) */
    float tau_s;                        /* Eq. 4 importance threshold, in [0, 1] */
    float lambda_s[MSAO_NUM_MODALITIES];/* Eq. 7 spatial weight per modality, in [0, 1] */
    float lambda_t[MSAO_NUM_MODALITIES];/* Eq. 7 temporal weight per modality, in [0, 1] */
    uint32_t flags;                     /* MSAO_FLAG_* */
} msao_params;

/* Per-token outputs, [total tokens] each; any pointer may be NULL (not written)
 * unless the entry point says otherwise. d and res are 0 for tokens of
 * non-temporal segments. */
typedef struct {
    uint32_t* z;     /* inactive channels (importance = 1 - z/C, Eq. 3 stand-in) */
    float* l1;       /* sum |x| */
    float* l2;       /* sum x^2 */
    float* info;     /* 1 - (lambda_s*z + lambda_t*e)/C: informativeness, orders like -key
                        (with SimHash: 1 - lambda_s*z/C - lambda_t*(K - d)/K) */
    uint32_t* d;     /* Hamming distance of activity bits to the previous frame (Eq. 5;
                        with SimHash: of the K signature bits) */
    float* res;      /* sum (x_t - x_{t-1})^2, the residual energy of Sec. 4.1.2 */
} msao_token_out;

/* Per-frame outputs of temporal segments, [total temporal frames] each; NULL skips. */
typedef struct {
    uint64_t* dframe;/* D_t = sum over the frame's tokens of d */
    float* sim;      /* Eq. 5: 1 - D_t/(P*C) (P*K with SimHash) */
    float* gamma;    /* 1 - sim (Sec. 4.1.2) */
} msao_frame_out;

/* Per-(request, modality) outputs, index r*4 + m; NULL skips. */
typedef struct {
    uint64_t* agg;   /* [R*4*4]: Ntok, Nsparse (Eq. 4 count), Dsum, Qbits (hash bits compared) */
    float* rho;      /* Eq. 4 over the modality: Nsparse/Ntok */
    float* temporal; /* temporal term of Eq. 7 (0 where absent) */
    float* beta;     /* softmax of alpha over the modalities present (Sec. 4.1.3) */
    float* mas;      /* Eq. 7 */
    uint8_t* present;/* 1 if the request has tokens of the modality */
} msao_req_out;

/* Selection outputs. kept_idx is [total tokens]: segment s owns the range
 * starting at its global token offset; its first kept_count[s] entries are the
 * kept token indices (local to the segment) in ascending order, the rest -1. */
typedef struct {
    uint8_t* keep;       /* [total tokens] 1 kept / 0 dropped; may be NULL */
    int32_t* kept_idx;   /* [total tokens], required */
    int32_t* kept_count; /* [n segments], required */
} msao_select_out;

/* ---- context and helpers (host only) ------------------------------------ */

/* Create a context bound to HIP device `device`. MSAO_ERR_HIP if it is absent.
 * Tuning read from the environment at creation (launch shapes only: every
 * output is the same for any value): MSAO_ROW_ITEM_BYTES (bytes of rows per
 * scoring wavefront, 8192), MSAO_CHAIN_FRAMES (frames per wavefront of the
 * chain pass over clips, 0 = automatic), MSAO_XCD_ORDER (scoring block order:
 * -1 automatic, 0 dispatch order, 1 one range per XCD), MSAO_CLIP_FUSE (1:
 * the run with SimHash scores and hashes its clips in one pass), MSAO_PAIR
 * (1: bf16 clips with rows of 512 to 2,048 bytes take the paired pass) and
 * MSAO_POST_BIG_SEGMENT (selections of at least this many tokens take
 * 1,024-thread blocks, 4096: lower latency per batch; a larger value favours
 * throughput with several batches in flight). */
msao_status msao_create(msao_ctx** ctx, int device);
/* Destroy a context (NULL is ignored). Waits for the context's pending uploads. */
void msao_destroy(msao_ctx* ctx);
/* Message of the last failed call on this context ("" if none). */
const char* msao_last_error(const msao_ctx* ctx);
/* Message of the last failed context-free call in this thread ("" if none). */
const char* msao_last_error_global(void);
/* Static name of a status code. */
const char* msao_status_string(msao_status s);
/* tau 0.1, tau_s 0.3, lambda_s {0, .6, .6, .6}, lambda_t {0, 0, .4, 0}, flags 0. */
msao_params msao_default_params(void);

/* Check a segment table and parameters without touching any device. */
msao_status msao_validate(const msao_segment* segs, int n, int n_requests, const msao_params* params);
/* Total tokens and total temporal frames of a segment table (host only). */
msao_status msao_count(const msao_segment* segs, int n, int64_t* n_tokens, int64_t* n_frames);
/* Workspace bytes any entry point needs for this table (host only). */
msao_status msao_workspace_size(const msao_segment* segs, int n, int n_requests, size_t* bytes);
/* Default packed compaction layout (host only): out_byte_off[s] (host, [n]) is
 * where segment s's kept rows start; a segment with a fixed keep ratio gets
 * room for its kept rows under either selection scope (max(ceil(kappa N),
 * T ceil(kappa P))), a MAS-guided one for all N rows; offsets are 256-byte
 * aligned. *total_bytes receives the buffer size needed. */
msao_status msao_compact_layout(const msao_segment* segs, int n, int64_t* out_byte_off, int64_t* total_bytes);

/* ---- entry points (enqueue on `stream`) ---------------------------------- */

/* Sec. 4.1.1-4.1.4: per-token statistics, per-frame similarity, per-modality
 * aggregation, softmax and MAS. alpha is host [n_requests*4] logits or NULL. */
msao_status msao_mas_score(msao_ctx* ctx, const msao_segment* segs, int n, int n_requests,
                           const msao_params* params, const float* alpha,
                           const msao_token_out* tok, const msao_frame_out* frm, const msao_req_out* req,
                           void* workspace, size_t workspace_bytes, void* stream);

/* Sec. 4.1.2 Eq. 5 only: d and res per token (0 outside temporal segments),
 * per-frame D_t, sim and gamma, and the temporal term of Eq. 7 per (request,
 * modality) (`temporal`, device [n_requests*4], may be NULL). */
msao_status msao_temporal_redundancy(msao_ctx* ctx, const msao_segment* segs, int n, int n_requests,
                                     const msao_params* params, uint32_t* d, float* res,
                                     const msao_frame_out* frm, float* temporal,
                                     void* workspace, size_t workspace_bytes, void* stream);

/* Sec. 4.1.1 pruning with the Eq. 11 floor: per-segment top-k selection from
 * per-token z (and d for temporal segments; may be NULL if there are none).
 * mas (device [n_requests*4]) is read for segments with a negative keep ratio
 * and may be NULL if there are none. */
msao_status msao_select_tokens(msao_ctx* ctx, const msao_segment* segs, int n, int n_requests,
                               const msao_params* params, const uint32_t* z, const uint32_t* d,
                               const float* mas, const msao_select_out* sel,
                               void* workspace, size_t workspace_bytes, void* stream);

/* Packed copy of each segment's kept rows: row j of segment s (j <
 * kept_count[s]) is row kept_idx[off_s + j] of its data, written bitwise at
 * out + out_byte_off[s] + j*hidden*element_size. out_byte_off is host [n],
 * 16-byte aligned; each segment needs room for its kept rows under either
 * selection scope, max(ceil(kappa N), T ceil(kappa P)) for a fixed keep ratio
 * (the room msao_compact_layout gives), or N rows if its keep ratio is
 * negative; out_bytes bounds every write. */
msao_status msao_compact(msao_ctx* ctx, const msao_segment* segs, int n,
                         const int32_t* kept_idx, const int32_t* kept_count,
                         void* out, const int64_t* out_byte_off, int64_t out_bytes,
                         void* workspace, size_t workspace_bytes, void* stream);

/* All of the above in one call: scoring, MAS, selection and (if out != NULL)
 * compaction. tok->z is required, and tok->d if any segment is temporal. */
msao_status msao_run(msao_ctx* ctx, const msao_segment* segs, int n, int n_requests,
                     const msao_params* params, const float* alpha,
                     const msao_token_out* tok, const msao_frame_out* frm, const msao_req_out* req,
                     const msao_select_out* sel, void* out, const int64_t* out_byte_off, int64_t out_bytes,
                     void* workspace, size_t workspace_bytes, void* stream);

/* ---- msao_run for callers that cannot allocate device memory -------------- */

/* Limits of msao_run_noalloc: its scratch (per-call tables, then one 16-byte
 * integer partial per scoring work item) and, within it, its tables. */
#define MSAO_NOALLOC_SCRATCH_BYTES 16777216
#define MSAO_NOALLOC_TABLE_BYTES 2097152

/* msao_run with no workspace argument, for callers that cannot call hipMalloc
 * or anything that allocates device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid it): it allocates nothing, host
 * pinned memory included. Its scratch is the library's own array of
 * MSAO_NOALLOC_SCRATCH_BYTES, one per GPU, held from the first msao_create on
 * that GPU until the process ends; msao_create also reserves the context's
 * pinned staging for tables of up to MSAO_NOALLOC_TABLE_BYTES. Every other
 * argument, the outputs and the errors are those of msao_run, plus
 * MSAO_ERR_UNSUPPORTED (nothing enqueued) when the call's tables or scratch
 * exceed those limits (msao_workspace_size bounds the scratch a table needs;
 * the five benchmark workloads need at most about 4.4 MB). Every call on a
 * GPU shares that GPU's array and overwrites all of it that the call uses
 * before reading it: calls that overlap on one GPU (other streams, other
 * contexts, other threads) race on it and must be ordered by the caller. */
msao_status msao_run_noalloc(msao_ctx* ctx, const msao_segment* segs, int n, int n_requests,
                             const msao_params* params, const float* alpha,
                             const msao_token_out* tok, const msao_frame_out* frm, const msao_req_out* req,
                             const msao_select_out* sel, void* out, const int64_t* out_byte_off, int64_t out_bytes,
                             void* stream);

/* ---- plans: tables uploaded once, runs with no host-to-device copy -------- */

/* A plan holds the per-call tables of msao_run (offsets, work items, integer
 * thresholds, Q24 weights, keep counts, data pointers) for one segment table.
 * msao_plan_create validates, builds the tables and enqueues their upload into
 * `workspace` on `stream`; msao_plan_run then enqueues the three launches of
 * msao_run with no host-to-device copy, so a fixed-shape serving loop (new
 * data written into the same input buffers each time) pays no per-call
 * upload. The workspace must stay allocated and must not be written by the
 * caller while the plan exists; runs on other streams must be ordered after
 * `stream`. out_byte_off (host [n], may be NULL if no run compacts) is copied.
 * Runs of one plan that overlap on the GPU race on the workspace. */
typedef struct msao_plan msao_plan;
msao_status msao_plan_create(msao_ctx* ctx, const msao_segment* segs, int n, int n_requests,
                             const msao_params* params, const float* alpha, const int64_t* out_byte_off,
                             void* workspace, size_t workspace_bytes, void* stream, msao_plan** plan);
/* Same outputs and rules as msao_run. */
msao_status msao_plan_run(msao_plan* plan, const msao_token_out* tok, const msao_frame_out* frm,
                          const msao_req_out* req, const msao_select_out* sel, void* out, int64_t out_bytes,
                          void* stream);
/* Free a plan (NULL is ignored); the caller must have synchronised its runs. */
void msao_plan_destroy(msao_plan* plan);

/* ---- Sec. 4.1.1 Eq. 3 and Sec. 4.1.3 Eq. 6 with caller weights ------------ */

/* A learned spatial probing head for one segment (Eq. 3):
 *     M = sigmoid(Conv1x1(AvgPool(F)))
 * with the 1x1 convolution w . f + bias to one importance logit. AvgPool
 * averages over the pool x pool square around each patch of a frame's grid
 * (grid_w patches per row, tokens_per_frame / grid_w rows), cut to the grid.
 * A token is sparse (Eq. 4) iff M < tau_s. weight: device [hidden] in the
 * segment's dtype, 16-byte aligned; NULL means no head (the density
 * importance a / C is used). pool: odd, 1..15. grid_w: 0 (one row) or a
 * divisor of tokens_per_frame; tokens_per_frame <= 16384 with a head. */
typedef struct {
    const void* weight;
    float bias;
    int32_t grid_w;
    int32_t pool;
} msao_spatial_head;

/* Entries of the modality descriptor z_m fed to the relevance MLP: 1, rho
 * (Eq. 4), sum a / sum C (active fraction), sum L1 / sum C, sqrt(sum L2 /
 * sum C), the temporal term of Eq. 7 (0 if none), 1 if that term exists,
 * ln(1 + Ntok) / 16, all over the modality's tokens in the request. */
#define MSAO_MODAL_DESC 8

/* The relevance MLP of Eq. 6, shared by the modalities:
 *     alpha_m = w2 . relu(W1 [p; z_m] + b1) + b2
 * with p the request's prompt embedding. All pointers device, fp32, 4-byte
 * aligned: w1 [hidden][prompt_dim + MSAO_MODAL_DESC] row-major, b1 and w2
 * [hidden], prompt [n_requests][prompt_dim] (may be NULL when prompt_dim is
 * 0). 1 <= hidden <= 4096, 0 <= prompt_dim <= 16384. */
typedef struct {
    const float* w1;
    const float* b1;
    const float* w2;
    float b2;
    int32_t hidden;
    int32_t prompt_dim;
    const float* prompt;
} msao_modal_mlp;

/* Sec. 4.1.1-4.1.4 with learned heads: msao_mas_score's outputs, where a
 * segment with a head (heads[s].weight non-NULL; heads may be NULL) counts
 * Eq. 4 on its Eq. 3 importance, and beta is the softmax of the MLP's alpha
 * (of the host logits alpha, or 0, when mlp is NULL). importance (device
 * [total tokens] or NULL): M for tokens of segments with a head, a / C for
 * the others. alpha_out (device [n_requests*4]) and desc (device
 * [n_requests*4*MSAO_MODAL_DESC]) may be NULL; absent modalities get 0.
 * The workspace is the one msao_workspace_size gives. Errors as
 * msao_mas_score, plus MSAO_ERR_INVALID_ARG / MSAO_ERR_ALIGNMENT for the
 * head and MLP rules above. */
msao_status msao_mas_score_learned(msao_ctx* ctx, const msao_segment* segs, int n, int n_requests,
                                   const msao_params* params, const msao_spatial_head* heads,
                                   const msao_modal_mlp* mlp, const float* alpha, const msao_token_out* tok,
                                   float* importance, const msao_frame_out* frm, const msao_req_out* req,
                                   float* alpha_out, float* desc, void* ws, size_t ws_bytes, void* stream);

/* Sec. 4.1 with learned heads through to the kept tokens: the outputs of
 * msao_mas_score_learned, then the selection and compaction of msao_run,
 * where the pruning of Sec. 4.1.1 follows the learned importance:
 *   - a segment with a head keeps its k tokens of largest Eq. 3 importance M
 *     (ties by ascending index; an M that is NaN or not above 0 counts as 0,
 *     the least important);
 *   - a segment without a head keeps the k smallest (key, index) pairs of
 *     msao_run (activity and temporal redundancy);
 *   - k = min(N, ceil(kappa N)) from the keep ratio, or, for a negative keep
 *     ratio, kappa = 1 - MAS with the learned MAS (the MLP's beta and the
 *     heads' rho); the per-frame scope as in msao_run.
 * M is the float32 value the library computes (it is written to importance
 * when that is not NULL), so a token whose importance is within rounding of
 * the k-th one may fall on either side compared with an exact evaluation.
 * tok->z is required, and tok->d if any segment is temporal; sel, out,
 * out_byte_off and out_bytes as for msao_run. The workspace is the one
 * msao_workspace_size gives. Errors: those of msao_mas_score_learned and of
 * msao_run. */
msao_status msao_run_learned(msao_ctx* ctx, const msao_segment* segs, int n, int n_requests,
                             const msao_params* params, const msao_spatial_head* heads, const msao_modal_mlp* mlp,
                             const float* alpha, const msao_token_out* tok, float* importance,
                             const msao_frame_out* frm, const msao_req_out* req, float* alpha_out, float* desc,
                             const msao_select_out* sel, void* out, const int64_t* out_byte_off, int64_t out_bytes,
                             void* ws, size_t ws_bytes, void* stream);

/* ---- the SimHash variant of Eq. 5 ----------------------------------------- */

/* Random hyperplanes of one segment for Charikar's hash (Sec. 4.1.2 Eq. 5
 * with h_k(f) = 1 iff r_k . f >= 0). planes: device [bits][hidden] in the
 * segment's dtype (row k is r_k), 16-byte aligned; bits: 16, 32, 48 or 64.
 * The caller draws the hyperplanes (e.g. N(0, 1) entries). */
typedef struct {
    const void* planes;
    int32_t bits;
} msao_simhash;

/* Sec. 4.1.2 Eq. 5 with SimHash instead of bit sampling. hashes (host, [n]):
 * the entry of every temporal segment (VIDEO, n_frames >= 2,
 * tokens_per_frame > 0) is required, the others are ignored.
 *   sig (device [total tokens] u64, required): the token's K-bit signature
 *     (bit k for r_k; 0 outside temporal segments);
 *   d (device [total tokens], required): the number of its K bits that
 *     differ from the same patch in the previous frame; frame 0 is compared
 *     with the all-zero frame, whose bits are all 1; 0 outside temporal
 *     segments;
 *   frm: D_t = sum of d over the frame, sim = 1 - D_t/(P K), gamma = 1 - sim;
 *   temporal (device [n_requests*4] or NULL): the temporal term of Eq. 7
 *     from frames 1..T-1 (1 - gamma_avg, or gamma_avg under
 *     MSAO_FLAG_TEMPORAL_LITERAL).
 * The projections are fp32 sums of exact bf16 products (fp32 products for
 * fp32 data) on the matrix cores, so a bit whose projection is within
 * rounding of 0 may differ from an exact evaluation. Workspace from
 * msao_workspace_size. Errors: those of msao_temporal_redundancy, plus
 * MSAO_ERR_INVALID_ARG for a missing hash entry or bits not in {16, 32, 48,
 * 64}, MSAO_ERR_ALIGNMENT for planes, sig or d, MSAO_ERR_UNSUPPORTED for a
 * row pitch of 64 MiB or more (32 MiB in a build with 64-token hash tiles). */
msao_status msao_temporal_simhash(msao_ctx* ctx, const msao_segment* segs, int n, int n_requests,
                                  const msao_params* params, const msao_simhash* hashes, uint64_t* sig,
                                  uint32_t* d, const msao_frame_out* frm, float* temporal, void* ws,
                                  size_t ws_bytes, void* stream);

/* Sec. 4.1 with SimHash as Eq. 5's hash throughout: msao_run's outputs,
 * where the d of every temporal segment is SimHash's (the bits of its K-bit
 * signature that differ from the same patch in the previous frame, as in
 * msao_temporal_simhash) and every later step counts it in K bits per token
 * instead of C activity bits:
 *   frm: sim = 1 - D_t / (P K), gamma = 1 - sim;
 *   req: agg's Dsum is SimHash's, Qbits = sum over the clips of (T-1) P K,
 *     and the temporal term and MAS follow;
 *   tok->info of a clip's tokens: 1 - (lambda_s z / C + lambda_t (K - d) / K);
 *   selection: the key orders a clip's tokens by lambda_s z / C + lambda_t
 *     (K - d) / K with the Q24 weights, as an exact integer; ties by index.
 * z, l1, l2 and res (the squared difference of the rows) are as in msao_run.
 * hashes (host, [n]) as for msao_temporal_simhash. sig (device [total
 * tokens] u64, 8-byte aligned, required when there are tokens) receives
 * the signatures, 0 outside temporal segments. Every other argument,
 * the workspace size and the errors are those of msao_run, plus the hash
 * errors of msao_temporal_simhash. Precision: the projections are fp32 sums
 * on the matrix cores, so a signature bit whose projection is within
 * rounding of 0 may differ from an exact evaluation, and with it d, the
 * terms above and the choice among nearly tied tokens. */
msao_status msao_run_simhash(msao_ctx* ctx, const msao_segment* segs, int n, int n_requests,
                             const msao_params* params, const msao_simhash* hashes, const float* alpha,
                             const msao_token_out* tok, uint64_t* sig, const msao_frame_out* frm,
                             const msao_req_out* req, const msao_select_out* sel, void* out,
                             const int64_t* out_byte_off, int64_t out_bytes, void* workspace,
                             size_t workspace_bytes, void* stream);

/* ---- Sec. 4.2: the draft model's confidence ------------------------------- */

/* Outputs of msao_draft_entropy, each [rows] device memory or NULL (not
 * written). entropy: Eq. 9 in nats, H = -sum_v p_v ln p_v with p the softmax
 * of the row's logits. entropy_norm: H / ln(vocab), in [0, 1] (the scale of
 * the confidence threshold). draft_token: the greedy draft token, the index
 * of the largest logit (the first of equal maxima). speculate: Eq. 10,
 * 1 if entropy_norm <= theta else 0. */
typedef struct {
    float* entropy;
    float* entropy_norm;
    int32_t* draft_token;
    uint8_t* speculate;
} msao_entropy_out;

/* Eq. 9-10 for `rows` rows of draft-model logits (Sec. 4.2.1: confidence of
 * the draft model at each generation step). logits: device, row r starts at
 * element r * row_stride, `vocab` logits per row, dtype MSAO_F32 or
 * MSAO_BF16; 16-byte aligned, row_stride * element size a multiple of 16,
 * row_stride >= vocab, 2 <= vocab, vocab * element size < 2^31 - 2^20,
 * rows < 2^31. Logits may be -inf (probability 0); a row with a NaN or +inf
 * logit, or with no finite one, gets a NaN entropy. theta: the confidence
 * threshold on entropy_norm (finite). Errors: MSAO_ERR_INVALID_ARG,
 * MSAO_ERR_ALIGNMENT, MSAO_ERR_HIP; nothing is written on a validation error.
 * Enqueued on `stream`; outputs are valid after the caller synchronises. */
msao_status msao_draft_entropy(msao_ctx* ctx, const void* logits, int64_t rows, int64_t vocab, int64_t row_stride,
                               int dtype, float theta, const msao_entropy_out* out, void* stream);

/* ---- Sec. 4.2.2: Algorithm 1 on the host ----------------------------------- */

/* Parameters of Algorithm 1 (defaults from Sec. 5.1: P_target 0.8, N_max 5,
 * the 70th percentile of the calibration entropies as the initial threshold,
 * decay delta 0.95; theta_min and the EMA weight alpha are not given by the
 * paper: 0.05 and 0.1). */
typedef struct {
    double p_target;   /* target acceptance probability (line 3) */
    int32_t n_max;     /* longest draft (line 3) */
    double quantile;   /* quantile of the calibration entropies giving theta (line 2) */
    double delta;      /* threshold decay on an offload (line 11) */
    double theta_min;  /* floor of the decayed threshold (line 11) */
    double alpha;      /* EMA weight of a verified cache's mean entropy (line 8) */
} msao_sched_params;

/* Per-request state of the per-step loop. */
typedef struct {
    double theta;        /* confidence threshold on normalised entropy */
    double p_conf;       /* Eq. 12 of the calibration set at the initial threshold */
    int32_t n_draft;     /* draft length from line 3 */
    int32_t cache;       /* drafted tokens held on the edge, not yet sent */
    double cache_h;      /* sum of their normalised entropies */
    int64_t steps, held, sends, offloads, tokens_sent;
} msao_sched_state;

#define MSAO_DECIDE_HOLD 0     /* confident: the draft token joins the cache */
#define MSAO_DECIDE_SEND 1     /* confident and the cache reached n_draft: send it for verification */
#define MSAO_DECIDE_OFFLOAD 2  /* not confident: offload the intermediate state */

msao_sched_params msao_sched_default_params(void);
/* Lines 2-3: theta = lower empirical quantile sorted[ceil(q n) - 1] of the
 * host calibration entropies (normalised, [n], n >= 1, finite); p_conf = Eq.
 * 12 at that theta; n_draft = min(floor(log(1 - P_target) / log p_conf),
 * N_max), at least 1 (N_max when p_conf = 1). Resets the per-step state.
 * MSAO_ERR_INVALID_ARG on NULL pointers, n < 1, non-finite entropies or
 * parameters outside their ranges (0 < p_target < 1, n_max >= 1, 0 <= q <= 1,
 * 0 < delta <= 1, theta_min >= 0, 0 <= alpha <= 1). */
msao_status msao_sched_init(const float* calib_h_norm, int64_t n, const msao_sched_params* params,
                            msao_sched_state* state);
/* Lines 5-11 for one step with normalised entropy h_norm (from
 * msao_draft_entropy): h_norm <= theta adds the token to the cache, and once
 * the cache holds n_draft tokens they are sent (decision SEND) and theta
 * moves to (1 - alpha) theta + alpha * (their mean entropy); otherwise
 * (HOLD). h_norm > theta (or NaN) offloads: the cache travels with the
 * offloaded state and theta = max(theta * delta, theta_min). */
msao_status msao_sched_step(msao_sched_state* state, const msao_sched_params* params, float h_norm,
                            int32_t* decision);
/* msao_sched_step over `steps` host entropies; decisions and theta_after
 * ([steps], host) may be NULL. */
msao_status msao_sched_run(msao_sched_state* state, const msao_sched_params* params, const float* h_norm,
                           int64_t steps, int8_t* decisions, double* theta_after);
/* Line 1 at the floor of Eq. 11: beta_m = 1 - MAS_m (host arrays [n]). */
msao_status msao_retention_floor(const float* mas, int n, float* beta);
/* Eq. 8: data_bytes / bandwidth + rtt (seconds; bandwidth in bytes/s). */
double msao_comm_latency(double data_bytes, double bandwidth_bytes_per_s, double rtt_s);
/* Eq. 12: fraction of the n host entropies that are <= theta (0 if n < 1). */
double msao_p_conf(const float* h_norm, int64_t n, double theta);
/* Eq. 13: 1 / (1 - p_conf), +inf at p_conf >= 1. */
double msao_expected_spec_tokens(double p_conf);

/* Terms of Eq. 14 (seconds). comm_offloaded: sum of Eq. 8 over the
 * offloaded modalities. */
typedef struct {
    double prefill_edge, prefill_cloud, comm_offloaded;
    double p_conf;
    int32_t n_draft;
    double t_draft, t_verify, t_offload;  /* per draft token, per verified token, per offload */
} msao_latency_model;
/* Eq. 14: max(prefill_edge, prefill_cloud + comm_offloaded)
 *   + E[N_spec] (n_draft t_draft + p_conf n_draft t_verify) + (1 - p_conf) t_offload. */
double msao_expected_e2e_latency(const msao_latency_model* m);

/* ---- profiling ----------------------------------------------------------- */

/* Kernels of the library, for msao_kernel_times. */
#define MSAO_KERNEL_SCORE 0   /* per-token statistics and temporal term */
#define MSAO_KERNEL_POST 1    /* aggregation, MAS, per-frame terms, selection */
#define MSAO_KERNEL_GATHER 2  /* compaction */
#define MSAO_KERNEL_ENTROPY 3 /* draft confidence */
#define MSAO_KERNEL_HEAD 4    /* learned spatial head: pooling, sigmoid, Eq. 4 counts */
#define MSAO_KERNEL_SIMHASH 5 /* SimHash signatures */
#define MSAO_KERNEL_HASH_POST 6 /* SimHash d, per-frame terms, temporal term */
#define MSAO_KERNEL_CLIP 7    /* the SimHash run's clips: statistics and signatures in one pass */
#define MSAO_KERNEL_READ 8    /* msao_stream_read: the plain streaming read */
#define MSAO_NUM_KERNELS 9

/* When enabled, every launch is bracketed by a pair of HIP events recorded on
 * the caller's stream. */
msao_status msao_set_profiling(msao_ctx* ctx, int enable);
/* ms[MSAO_NUM_KERNELS]: mean milliseconds per launch of each kernel over the
 * launches recorded since the previous query (0 if none); blocks until they
 * have completed, then forgets them. */
msao_status msao_kernel_times(msao_ctx* ctx, float* ms);

/* ---- measurement ---------------------------------------------------------- */

/* A plain streaming read of `bytes` of device memory at `data`, the
 * ceiling the HBM-bound passes are measured against on the same machine (it
 * computes nothing of the analysis). Wavefront w reads bytes [w*chunk,
 * (w+1)*chunk) with chunk = chunk_kib KiB (8, 16, 32 or 64) as 128-bit
 * nontemporal loads, eight 1-KiB units in flight, and writes the XOR of the
 * 32-bit words it read to sink[w] (device, ceil(bytes / chunk) words,
 * sink_words at least that). data 16-byte aligned, bytes > 0. Errors:
 * MSAO_ERR_INVALID_ARG, MSAO_ERR_ALIGNMENT, MSAO_ERR_HIP. With profiling on,
 * its launch time is reported as MSAO_KERNEL_READ. */
msao_status msao_stream_read(msao_ctx* ctx, const void* data, int64_t bytes, int chunk_kib, uint32_t* sink,
                             int64_t sink_words, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* MSAO_H */
