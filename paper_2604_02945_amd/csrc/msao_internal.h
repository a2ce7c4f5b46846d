// msao_internal.h -- device-side tables shared by the host planner
// (msao_host.cpp) and the gfx950 kernels (msao_kernels.hip). Not part of the
// public ABI.
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace msao {

enum : int { kText = 0, kImage = 1, kVideo = 2, kAudio = 3, kNumMod = 4 };
enum : int { kF32 = 0, kBF16 = 1 };
constexpr uint32_t kFlagLiteral = 1u;  // Eq. 7 takes gamma_avg as printed (the public flag bit 1)
enum : int { kModeScore = 0, kModeTemporal = 1 };

// One segment as the kernels see it. Built on the host for every call and
// uploaded into the caller's workspace with the other tables.
struct DevSeg {
    const uint8_t* data;   // first row
    int64_t stride_bytes;  // bytes between consecutive rows
    int64_t out_off;       // compaction: byte offset of the segment's packed rows
    int32_t tok_off;       // global token id of row 0
    int32_t n_tok;         // N = T*P
    int32_t T, P, C;
    int32_t dtype;         // kF32 / kBF16
    int32_t modality, request;
    int32_t temporal;      // VIDEO with T >= 2 and P > 0
    int32_t frame_off;     // global frame id of frame 0 (temporal segments)
    int32_t wi_begin;      // first scoring work item (one wavefront each)
    int32_t per_item;      // rows per item, or frames per item for temporal segments
    int32_t nchunk;        // 16-byte chunks per row
    int32_t A_s;           // Eq. 4 as an integer test: sparse iff active < A_s = ceil(tau_s*C)
    uint32_t L_s, L_t;     // Q24 selection weights of the segment's modality
    float lam_s, lam_t;    // the same weights as floats (informativeness)
    int32_t k;             // fixed keep count, or -1 when MAS-guided
    int32_t cap;           // compaction capacity in rows
    int32_t g_begin;       // first gather work item
    int32_t copy_in_score; // every row is kept: the scoring pass writes the compacted rows itself
    // learned spatial head (Eq. 3), set only by learned calls
    const uint8_t* head_w; // [C] in the segment's dtype; NULL: no head
    float head_b;
    int32_t grid_w;        // patches per row of a frame's grid
    int32_t pool;          // odd AvgPool window
    int32_t hb_begin;      // first head block (one per frame)
    // per-frame selection scope
    int32_t kf;            // fixed keep count per frame, or -1 when MAS-guided
    // SimHash variant of Eq. 5, set only by SimHash calls
    const uint8_t* planes; // [hash_bits][C] hyperplanes in the segment's dtype
    int32_t hash_bits;     // K per token (16, 32, 48 or 64)
    int32_t hi_begin;      // first hash tile (kHashTokens tokens each)
    // Eq. 5's d counts E bits per token: C activity bits, or K SimHash bits
    // in a run with SimHash. The selection key Ms z + Mt (E - d) orders the
    // tokens as L_s z / C + L_t (E - d) / E: Ms = L_s E / g, Mt = L_t C / g
    // with g = gcd(C, E) (Ms = L_s, Mt = L_t for bit sampling).
    int32_t E;
    // a clip of a run with SimHash scored and hashed in one pass (k_clip):
    // work items of 15 frames x 1 position, cl_begin its first k_clip block
    int32_t fused;
    uint64_t key_ms, key_mt;
    int32_t cl_begin, ntiles;
    // a bf16 clip with rows of at most 2 KiB scored by k_pair: a wavefront
    // takes two adjacent positions over a range of per_item frames (tblk
    // ranges cover the clip; its items are rounded up to whole blocks)
    int32_t pair, tblk;
};

// Key kinds of a selection: Ms z + Mt (E - d) in general, z or E - d alone
// when the other weight is 0 (the same order, a narrower range); or, in a
// learned run, a segment with a head ranked by its Eq. 3 importance.
enum : int { kKeyZero = 0, kKeyZ = 1, kKeyE = 2, kKeyFull = 3, kKeyImp = 4 };

// One selection block: a whole segment (frame -1) or one frame of a clip
// (per-frame scope), or one of the nparts blocks of a large selection. Every
// block of a selection finds the same threshold from all of its keys; block
// `part` then writes the keep flags and kept indices of its own slice. It
// holds everything the block needs before its first load of z and d.
struct SelUnit {
    uint64_t Ms, Mt;        // key multipliers
    uint64_t kmax;          // largest key the selection can hold (z <= C, d <= E)
    int32_t seg, frame;     // segment; frame of a clip under the per-frame scope, else -1
    int32_t part, nparts;   // slice written by this block
    int32_t off, N;         // global token id of the selection's first token; its tokens
    int32_t kfix, kind;     // fixed keep count (-1: MAS-guided); key kind
    uint32_t E;             // bits d counts per token
    int32_t units;          // selections of the segment (T under the per-frame scope, else 1)
    int32_t seg_off;        // global token id of the segment's first token
    int32_t request, modality, pad_;
};
// Selections of the large-block launch (kPostBigSegment tokens or more,
// 1,024 threads) are split into parts of kSelBigPartTokens tokens for their
// counting and writing, one block each. Selections of kSelSplitMin tokens or
// more are split into parts of about kSelPartTokens tokens when the launch
// has fewer than kSelSplitMaxSelections selections: more parts would only
// queue behind each other on the CUs, since each part stages all of the keys
// again.
#ifndef MSAO_SEL_PART_TOKENS
#define MSAO_SEL_PART_TOKENS 768
#endif
constexpr int kSelPartTokens = MSAO_SEL_PART_TOKENS;
#ifndef MSAO_SEL_BIG_PART_TOKENS
#define MSAO_SEL_BIG_PART_TOKENS 2048
#endif
constexpr int kSelBigPartTokens = MSAO_SEL_BIG_PART_TOKENS;
#ifndef MSAO_SEL_SPLIT_MIN
#define MSAO_SEL_SPLIT_MIN 1024
#endif
constexpr int kSelSplitMin = MSAO_SEL_SPLIT_MIN;
#ifndef MSAO_SEL_SPLIT_MAX_SELECTIONS
#define MSAO_SEL_SPLIT_MAX_SELECTIONS 256
#endif
constexpr int kSelSplitMaxSelections = MSAO_SEL_SPLIT_MAX_SELECTIONS;

// Integer partial sums of one scoring work item (no atomics, no zeroing).
struct Partial {
    uint32_t nsparse;      // tokens with active < A_s
    uint32_t pad_;
    uint64_t dsum;         // sum of d over frames t >= 1
};

// One (request, modality): its sizes and its run of work-item ranges in rm_rng
// (one range per segment of that request and modality).
struct RmEntry {
    uint64_t ntok;         // tokens
    uint64_t qbits;        // activity bits compared by Eq. 5: sum over its video clips of (T-1)*P*C
    int32_t rng_begin, rng_end;
    int32_t pad_[2];
};

struct WiRange {
    int32_t begin, end;    // scoring work items of one segment
    int32_t seg, pad_;     // that segment
};

// More sums of one scoring work item, for the modality descriptor of Eq. 6
// (learned calls only).
struct PartialX {
    uint32_t asum;         // active channels over the item's tokens
    float l1, l2;          // sums of the tokens' L1 and L2
    uint32_t pad_;
};

// Device pointers into the workspace, plus scalars, passed by value.
struct Tables {
    const DevSeg* seg;
    const int32_t* wi_seg;   // [n_wi] segment of each scoring work item
    const int32_t* gi_seg;   // [n_gwi] segment of each gather work item
    const RmEntry* rm;       // [R*4]
    const WiRange* rm_rng;   // [n] work-item ranges grouped by (request, modality)
    const int32_t* tseg;     // [n_tseg] temporal segment ids in table order
    const int32_t* frame_seg;// [n_frames] segment of every temporal frame
    const float* alpha;      // [R*4] relevance logits
    Partial* partial;        // [n_wi]
    // learned calls only
    PartialX* partial_x;     // [n_wi]
    float* proj;             // [Ntot] w . x of tokens of segments with a head
    uint32_t* head_count;    // [n_hb] tokens with importance < tau_s, per head block
    const int32_t* hb_seg;   // [n_hb] segment of each head block
    int32_t n_hb;
    const SelUnit* sel_unit; // [n_sel] selections (one block each)
    const int32_t* hi_seg;   // [n_hi] segment of each hash tile (SimHash calls)
    const uint64_t* hdsum;   // [R*4] SimHash Dsum per (request, modality) in a run with SimHash, else NULL
    const int32_t* cl_seg;   // [n_cl] segment of each k_clip block (fused clips)
    int32_t n_cl;
    int32_t n_wi_score;      // work items of k_score: [0, n_wi_score); the fused clips' follow
    int32_t n_wi_pair;       // the first n_wi_pair of them (whole blocks) are k_pair's
    int32_t n_hi;
    int32_t n, R, n_wi, n_gwi, n_tseg, n_frames;
    float tau, tau_s;
    float lam_s[kNumMod], lam_t[kNumMod];
    uint32_t flags;
};

struct TokenOut {
    uint32_t* z; float* l1; float* l2; float* info; uint32_t* d; float* res;
    uint64_t* sig;  // a run with SimHash: signatures (k_score writes 0 for its tokens)
};
struct FrameOut {
    uint64_t* dframe; float* sim; float* gamma;
};
struct ReqOut {
    uint64_t* agg; float* rho; float* temporal; float* beta; float* mas; uint8_t* present;
};
struct SelOut {
    uint8_t* keep; int32_t* kept_idx; int32_t* kept_count;
};

// The relevance MLP of Eq. 6 (device pointers).
struct ModalMlp {
    const float* w1;       // [hidden][prompt_dim + kDesc]
    const float* b1;       // [hidden]
    const float* w2;       // [hidden]
    float b2;
    int32_t hidden, prompt_dim;
    const float* prompt;   // [R][prompt_dim]
};
constexpr int kDesc = 8;   // entries of the modality descriptor z_m

// Roles of the post-scoring launch.
struct PostArgs {
    Tables t;
    ReqOut req;           // request role outputs
    FrameOut frm;         // frame role outputs
    SelOut sel;           // selection role outputs
    const uint32_t* z;    // selection inputs
    const uint32_t* d;
    const float* mas_in;  // MAS from the caller (selection only); NULL: recompute
    int32_t n_sel_blocks; // blocks [0, n_sel_blocks): one per selection unit (SelUnit)
    int32_t n_req_blocks; // then one per request
    int32_t n_frame_blocks;// then one per temporal frame
    int32_t temporal_only;// request role writes only the temporal term
    int32_t keys_cap;     // selection keys staged in LDS per block (larger segments re-read z, d)
    int32_t big_block;    // 1: the launch's selections take 1024-thread blocks
    // learned calls: head counts and descriptors feed Eq. 4, Eq. 6 gives alpha
    int32_t learned;
    int32_t use_mlp;
    ModalMlp mlp;
    float* alpha_out;     // [R*4] (NULL: not written)
    float* desc_out;      // [R*4*kDesc]
    const float* mlp_u;   // [R][hidden] prompt half of the MLP's first layer plus b1
    float* mas_ws;        // learned request role: MAS per (request, modality) for a later selection (NULL: none)
};

struct ScoreArgs {
    Tables t;
    TokenOut tok;
    uint8_t* out;         // compaction output for copy_in_score segments (NULL: none)
    int32_t mode;
    int32_t xcd_order;    // 1: each XCD takes one contiguous range of workgroups
    int32_t learned;      // learned call: projections, importance of head-less tokens, PartialX
    float* importance;    // [Ntot] (learned calls; NULL: not written)
    int32_t wi_first;     // k_score's first work item (set by the launcher: the pair items precede it)
};

// Pooling, sigmoid and the Eq. 4 test of the learned spatial head: one
// block per frame of a segment with a head; then, when an MLP is given,
// n_mlp_blocks blocks computing u = W1[:, :prompt_dim] p + b1 per request
// (the part of Eq. 6's first layer that all modalities share).
struct HeadArgs {
    Tables t;
    float* importance;    // [Ntot] (NULL: not written)
    int32_t max_p;        // largest frame among segments with a head (LDS staging)
    int32_t n_mlp_blocks;
    ModalMlp mlp;
    float* u;             // [R][hidden]
};
constexpr int kHeadBlock = 256;
constexpr int kMaxHeadFrame = 16384;  // tokens per frame of a segment with a head (LDS)
constexpr int kMaxPool = 15;
constexpr int kMaxMlpHidden = 4096;

// The SimHash variant of Eq. 5: k_simhash computes each token's signature
// (one wavefront per tile of kHashTokens tokens, four tiles of one segment
// per block, MFMA over the channels);
// k_hash_post derives d, D_t, sim, gamma (one block per frame) and the
// temporal term (one block per request).
#ifndef MSAO_HASH_TOKENS
#define MSAO_HASH_TOKENS 32
#endif
constexpr int kHashTokens = MSAO_HASH_TOKENS;  // 16, 32 or 64
constexpr int kHashWaves = 4;                   // tiles (wavefronts) per block, one segment per block
constexpr int kHashBlockTokens = kHashWaves * kHashTokens;
struct HashArgs {
    Tables t;
    uint64_t* sig;        // [Ntot]
    uint32_t* d;          // [Ntot]
    FrameOut frm;
    float* temporal;      // [R*4] (NULL: not written)
    // a run with SimHash: the frame blocks also rewrite the informativeness
    // of the clip's tokens from z and the new d, and the request blocks write
    // Dsum per (request, modality) for the MAS of the following launch
    const uint32_t* z;    // [Ntot]
    float* info;          // [Ntot] (NULL: not written)
    uint64_t* hdsum;      // [R*4] (NULL: not written)
    int32_t n_frame_blocks, n_req_blocks;
};
constexpr int kMlpGroup = 8;          // requests per wavefront in the prompt product

// The run with SimHash reads each clip once: k_clip scores and hashes tiles
// of up to 16 consecutive frames of one patch position (one wavefront each,
// kClipWaves per block, all of one clip). Consecutive tiles overlap by one
// frame, so a tile holds the predecessor of each of its new frames (at most
// 15, the clip's frames split evenly; the first tile starts at the all-zero
// frame -1): z, l1, l2, res, the signature, d against the previous frame and
// the informativeness of those tokens, and the work item's integer partials.
#ifndef MSAO_CLIP_WAVES
#define MSAO_CLIP_WAVES 4
#endif
constexpr int kClipWaves = MSAO_CLIP_WAVES;      // tiles (wavefronts) per block: 4 or 8
constexpr int kClipFrames = 15;                 // most new frames per tile (16 rows with the predecessor)
struct ClipArgs {
    Tables t;
    TokenOut tok;         // z, l1, l2, info, d, res, sig of the clips' tokens
    int32_t clip_dtype;   // element type and signature width shared by every fused clip
    int32_t clip_bits;
};
int launch_clip(const ClipArgs& a, void* stream, void* ev0, void* ev1);

struct GatherArgs {
    Tables t;
    const int32_t* kept_idx;
    const int32_t* kept_count;
    uint8_t* out;
    int64_t out_bytes;
};

// Draft-model confidence (msao_entropy.hip): one row of logits per workgroup.
struct EntArgs {
    const uint8_t* logits;   // row r starts at logits + r * row_bytes
    int64_t row_bytes;
    int32_t rows, vocab, dtype;
    float theta;             // Eq. 10 threshold on the normalised entropy
    float inv_log_vocab;     // 1 / ln(vocab)
    float* entropy;          // [rows] nats (NULL: not written)
    float* entropy_norm;     // [rows] entropy / ln(vocab)
    int32_t* draft_token;    // [rows] arg max, first of equal maxima
    uint8_t* speculate;      // [rows] entropy_norm <= theta
};
#ifndef MSAO_ENT_BLOCK
#define MSAO_ENT_BLOCK 256
#endif
#ifndef MSAO_ENT_UNITS
#define MSAO_ENT_UNITS 4
#endif
constexpr int kEntBlock = MSAO_ENT_BLOCK;  // threads per row of logits
constexpr int kEntUnits = MSAO_ENT_UNITS;  // 16-byte chunks per thread per batch
int launch_entropy(const EntArgs& a, void* stream, void* ev0, void* ev1);

// Launchers (msao_kernels.hip). Return the HIP error code of the launch, or
// kNoLaunch when there is nothing to launch (then nothing is enqueued). ev0
// and ev1 (hipEvent_t, may be NULL) are recorded at the kernel's start and end.
constexpr int kNoLaunch = -1;
int launch_score(const ScoreArgs& a, void* stream, void* ev0, void* ev1);
int launch_post(const PostArgs& a, void* stream, void* ev0, void* ev1);
int launch_gather(const GatherArgs& a, void* stream, void* ev0, void* ev1);
int launch_head(const HeadArgs& a, void* stream, void* ev0, void* ev1);
int launch_simhash(const HashArgs& a, void* stream, void* ev0, void* ev1);
int launch_hash_post(const HashArgs& a, void* stream, void* ev0, void* ev1);

constexpr int kScoreBlock = 256;   // 4 wavefronts, one work item each
#ifndef MSAO_PAIR_WAVES
#define MSAO_PAIR_WAVES 4
#endif
// k_pair block: wavefronts on consecutive pairs of positions over the same
// frames (four: a clip batch of 1,024 wavefronts puts one on every SIMD)
constexpr int kPairWaves = MSAO_PAIR_WAVES;
// k_pair's register budget: a ring of four frames needs about 146 VGPRs
constexpr int kPairWavesPerEU = 2;
constexpr int kPairRing = 4;                  // frames in registers per k_pair wavefront (even)
constexpr int kPairMaxRowBytes = 2048;        // rows k_pair takes: four 512-byte units per half-wavefront
#ifndef MSAO_PAIR_MAX_FRAMES
#define MSAO_PAIR_MAX_FRAMES 32
#endif
constexpr int kPairMaxFrames = MSAO_PAIR_MAX_FRAMES;  // frames per k_pair wavefront (the token buffer holds 2 per frame)
static_assert(kPairMaxFrames >= 1 && kPairMaxFrames <= 32, "k_pair parks two tokens per frame in 64 lanes");
// k_pair range length: halved from kPairMaxFrames down to kPairMinFrames to
// spread a batch's frames evenly over kPairTargetWaves SIMDs
constexpr int kPairMinFrames = 8;
constexpr int kPairTargetWaves = 1024;
#ifndef MSAO_POST_BLOCK
#define MSAO_POST_BLOCK 256
#endif
constexpr int kPostBlock = MSAO_POST_BLOCK;  // threads per post-scoring block
#ifndef MSAO_POST_BIG_SEGMENT
#define MSAO_POST_BIG_SEGMENT 4096
#endif
constexpr int kPostBigSegment = MSAO_POST_BIG_SEGMENT;  // larger selections use 1024-thread blocks
// k_gather block size: one wavefront per block for launches of many kept
// rows, larger blocks for launches of at most kGatherFewItems work items
// (with other batches' scoring in flight, the few-row launches finish their
// share sooner in larger blocks; a long one of one-wavefront blocks
// interleaves better).
#ifndef MSAO_GATHER_BLOCK
#define MSAO_GATHER_BLOCK 64
#endif
constexpr int kGatherBlock = MSAO_GATHER_BLOCK;
#ifndef MSAO_GATHER_BLOCK_FEW
#define MSAO_GATHER_BLOCK_FEW 512
#endif
constexpr int kGatherBlockFew = MSAO_GATHER_BLOCK_FEW;
#ifndef MSAO_GATHER_FEW_ITEMS
#define MSAO_GATHER_FEW_ITEMS 98304
#endif
constexpr int kGatherFewItems = MSAO_GATHER_FEW_ITEMS;
#ifndef MSAO_GATHER_ROWS
#define MSAO_GATHER_ROWS 1
#endif
constexpr int kGatherRows = MSAO_GATHER_ROWS;  // kept rows per gather work item
constexpr int kMaxLdsKeys = 16384; // 128 KiB of LDS per selection block

// A plain streaming read (msao_calib.hip): wavefront w reads bytes
// [w * chunk_bytes, (w + 1) * chunk_bytes) of data and writes the XOR of
// the words it read to sink[w].
struct ReadArgs {
    const uint8_t* data;
    int64_t bytes;
    int64_t waves;
    int32_t chunk_bytes;  // a multiple of 8 KiB
    uint32_t* sink;       // [waves]
};
constexpr int kReadBlock = 256;
int launch_read(const ReadArgs& a, void* stream, void* ev0, void* ev1);

// msao_run_noalloc: the library's own scratch (msao_scratch.hip), one array
// per GPU in place of the caller's workspace. Its per-call tables are at most
// kNoAllocTableBytes (the pinned staging every context reserves at creation).
constexpr size_t kNoAllocScratchBytes = (size_t)16 << 20;
constexpr size_t kNoAllocTableBytes = (size_t)2 << 20;
constexpr int kMaxScratchDevices = 64;
int scratch_init(int device);   // with `device` current; returns a HIP error code
void* scratch_ptr(int device);  // NULL before scratch_init succeeded

}  // namespace msao
