// msao_host.cpp -- host side of the C ABI declared in include/msao.h:
// validation (before any device work), planning of the per-call tables
// (token/frame offsets, work items, Eq. 4 integer thresholds, Q24 selection
// weights, keep counts), upload into the caller's workspace from pinned
// staging, and the kernel launches on the caller's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <numeric>
#include <string>
#include <vector>

#include "../../include/msao.h"
#include "msao_internal.h"

using namespace msao;

struct msao_ctx {
    int device = 0;
    std::string err;
    // two pinned staging slots, each guarded by the event of its last upload
    void* stage[2] = {nullptr, nullptr};
    size_t stage_cap[2] = {0, 0};
    hipEvent_t stage_ev[2] = {nullptr, nullptr};
    bool stage_used[2] = {false, false};
    int next_slot = 0;
    // profiling: an event pair around every launch, averaged per kernel on query
    bool profiling = false;
    std::vector<hipEvent_t> pool;                       // free events
    std::vector<std::pair<hipEvent_t, hipEvent_t>> rec[MSAO_NUM_KERNELS];
    // tuning
    int row_item_bytes = 8192;
    int chain_frames = 0;       // frames per temporal work item; 0 = automatic
    int xcd_order = -1;         // scoring block order: -1 automatic, 0 dispatch order, 1 one range per XCD
    int clip_fuse = 1;          // the SimHash run scores and hashes its clips in one pass (k_clip)
    int pair_path = 1;          // bf16 clips with rows of at most 2 KiB are scored by k_pair
    int post_big_segment = kPostBigSegment;  // selections this large take 1024-thread blocks
};

namespace {

thread_local std::string g_err;

constexpr size_t kWsAlign = 256;

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

int elt_size(int dtype) { return dtype == MSAO_F32 ? 4 : 2; }

bool is_temporal(const msao_segment& s)
{
    return s.modality == MSAO_VIDEO && s.n_frames >= 2 && s.tokens_per_frame > 0;
}

msao_status fail(std::string* err, msao_status st, const std::string& msg)
{
    if (err) *err = msg;
    return st;
}

// Keep count: k = min(N, ceil(kappa * N)) in double.
int64_t keep_count(float kappa, int64_t N)
{
    double k = std::ceil((double)kappa * (double)N);
    if (k > (double)N) k = (double)N;
    if (k < 0.0) k = 0.0;
    return (int64_t)k;
}

// Q24 weight: round-to-nearest-even of lambda * 2^24.
uint32_t q24(float lambda) { return (uint32_t)std::nearbyint((double)lambda * 16777216.0); }

msao_status validate_impl(const msao_segment* segs, int n, int R, const msao_params* p, std::string* err)
{
    char buf[256];
    if (n < 0) return fail(err, MSAO_ERR_INVALID_ARG, "segment count is negative");
    if (n > 0 && !segs) return fail(err, MSAO_ERR_INVALID_ARG, "segment table is NULL");
    if (R < 0) return fail(err, MSAO_ERR_INVALID_ARG, "request count is negative");
    if (!p) return fail(err, MSAO_ERR_INVALID_ARG, "params is NULL");
    if (!(std::isfinite(p->tau) && p->tau >= 0.0f))
        return fail(err, MSAO_ERR_INVALID_ARG, "tau must be finite and >= 0");
    if (!(p->tau_s >= 0.0f && p->tau_s <= 1.0f))
        return fail(err, MSAO_ERR_INVALID_ARG, "tau_s must be in [0, 1]");
    for (int m = 0; m < MSAO_NUM_MODALITIES; ++m) {
        if (!(p->lambda_s[m] >= 0.0f && p->lambda_s[m] <= 1.0f) || !(p->lambda_t[m] >= 0.0f && p->lambda_t[m] <= 1.0f))
            return fail(err, MSAO_ERR_INVALID_ARG, "lambda_s and lambda_t must be in [0, 1]");
    }
    if (p->flags & ~(MSAO_FLAG_TEMPORAL_LITERAL | MSAO_FLAG_SELECT_PER_FRAME))
        return fail(err, MSAO_ERR_INVALID_ARG, "unknown flag bits");
    int64_t total = 0;
    for (int i = 0; i < n; ++i) {
        const msao_segment& s = segs[i];
        auto bad = [&](msao_status st, const char* what) {
            std::snprintf(buf, sizeof buf, "segment %d: %s", i, what);
            return fail(err, st, buf);
        };
        if (s.modality < 0 || s.modality >= MSAO_NUM_MODALITIES) return bad(MSAO_ERR_INVALID_ARG, "unknown modality");
        if (s.dtype != MSAO_F32 && s.dtype != MSAO_BF16) return bad(MSAO_ERR_INVALID_ARG, "unknown dtype");
        if (s.request < 0 || s.request >= R) return bad(MSAO_ERR_INVALID_ARG, "request id out of range");
        if (s.n_frames < 1) return bad(MSAO_ERR_INVALID_ARG, "n_frames must be >= 1");
        if (s.n_frames > 1 && s.modality != MSAO_VIDEO) return bad(MSAO_ERR_INVALID_ARG, "n_frames > 1 on a non-video segment");
        if (s.tokens_per_frame < 0) return bad(MSAO_ERR_INVALID_ARG, "tokens_per_frame is negative");
        if (s.hidden < 1 || s.hidden > MSAO_MAX_HIDDEN) return bad(MSAO_ERR_INVALID_ARG, "hidden out of range");
        if (s.hidden % (16 / elt_size(s.dtype)) != 0)
            return bad(MSAO_ERR_ALIGNMENT, "hidden must be a multiple of 8 (bf16) or 4 (fp32)");
        if (std::isnan(s.keep_ratio) || s.keep_ratio > 1.0f) return bad(MSAO_ERR_INVALID_ARG, "keep_ratio must be <= 1 (negative: MAS-guided)");
        const int64_t N = (int64_t)s.n_frames * s.tokens_per_frame;
        if (N > INT32_MAX) return bad(MSAO_ERR_UNSUPPORTED, "more than 2^31-1 tokens");
        total += N;
        if (total > INT32_MAX - 1) return bad(MSAO_ERR_UNSUPPORTED, "more than 2^31-2 tokens in total");
        if (N > 0) {
            if (!s.data) return bad(MSAO_ERR_INVALID_ARG, "data is NULL");
            if (s.row_stride < s.hidden) return bad(MSAO_ERR_INVALID_ARG, "row_stride < hidden");
            if (((uintptr_t)s.data) % 16 != 0) return bad(MSAO_ERR_ALIGNMENT, "data is not 16-byte aligned");
            if ((s.row_stride * elt_size(s.dtype)) % 16 != 0)
                return bad(MSAO_ERR_ALIGNMENT, "row pitch is not a multiple of 16 bytes");
        }
    }
    return MSAO_OK;
}

// Per-call tables, built on the host and uploaded into the workspace.
struct Plan {
    std::vector<DevSeg> seg;
    std::vector<int32_t> wi_b, wi_e;             // per segment: its scoring work items [wi_b, wi_e) (host only)
    std::vector<int32_t> seg_gi, tseg;           // seg_gi: per-segment prefix of gather items (host only)
    std::vector<int32_t> wi_seg, gi_seg;         // segment of every work item
    std::vector<RmEntry> rm;
    std::vector<WiRange> rm_rng;
    std::vector<float> alpha;
    int64_t ntok = 0, nframes = 0;
    int n_wi = 0, n_gwi = 0;
    int max_n = 0;                 // largest selection (LDS key staging)
    int big_seg = kPostBigSegment; // selections this large take 1024-thread blocks
    std::vector<SelUnit> sel_unit; // one selection block each: a segment, or a frame (per-frame scope)
    std::vector<int32_t> hi_seg;   // SimHash calls: segment of each hash tile
    bool any_temporal = false, any_guided = false;
    bool any_copy = false;         // some segment is compacted by the scoring pass
    // learned calls (Eq. 3 heads, Eq. 6 descriptors)
    bool learned = false;
    std::vector<int32_t> hb_seg;   // segment of each head block (one per frame of a segment with a head)
    int max_head_p = 0;            // largest frame among segments with a head
    int mlp_hidden = 0;            // > 0: the relevance MLP's u = W1[:, :P] p + b1 per request
    size_t off_hbseg = 0, off_partial_x = 0, off_proj = 0, off_head_count = 0, off_mlp_u = 0, off_mas = 0;
    size_t off_seg = 0, off_wi = 0, off_gi = 0, off_rmoff = 0, off_rmseg = 0, off_tseg = 0, off_alpha = 0;
    size_t off_selu = 0, off_hiseg = 0, off_clseg = 0, off_frseg = 0;
    std::vector<int32_t> frame_seg;  // segment of every temporal frame
    bool simhash_d = false;        // a run with SimHash: d of temporal segments in K-bit units
    size_t off_hdsum = 0;          // [R*4] SimHash Dsum (simhash_d without clip_fused)
    bool clip_fused = false;       // a run with SimHash whose clips k_clip scores and hashes in one pass
    int clip_dtype = -1, clip_bits = 0;
    std::vector<int32_t> cl_seg;   // segment of each k_clip block
    int n_wi_score = 0;            // k_score's work items [0, n_wi_score); the fused clips' follow
    int n_wi_pair = 0;             // k_pair's work items [0, n_wi_pair), whole blocks
    size_t table_bytes = 0, off_partial = 0, total_bytes = 0;
};

size_t table_layout(Plan& pl, int n, int R, int64_t n_wi, int64_t n_gwi, int64_t n_hb, int64_t n_sel, int64_t n_hi,
                    int64_t n_cl, int64_t n_fr)
{
    size_t o = 0;
    auto take = [&](size_t bytes) {
        const size_t at = o;
        o = align_up(o + bytes, 16);
        return at;
    };
    pl.off_seg = take(sizeof(DevSeg) * (size_t)std::max(n, 1));
    pl.off_wi = take(sizeof(int32_t) * (size_t)std::max<int64_t>(n_wi, 1));
    pl.off_gi = take(sizeof(int32_t) * (size_t)std::max<int64_t>(n_gwi, 1));
    pl.off_rmoff = take(sizeof(RmEntry) * (size_t)std::max(R * kNumMod, 1));
    pl.off_rmseg = take(sizeof(WiRange) * (size_t)std::max(n, 1));
    pl.off_tseg = take(sizeof(int32_t) * (size_t)std::max(n, 1));
    pl.off_alpha = take(sizeof(float) * (size_t)std::max(R * kNumMod, 1));
    pl.off_hbseg = take(sizeof(int32_t) * (size_t)std::max<int64_t>(n_hb, 1));
    pl.off_selu = take(sizeof(SelUnit) * (size_t)std::max<int64_t>(n_sel, 1));
    pl.off_hiseg = take(sizeof(int32_t) * (size_t)std::max<int64_t>(n_hi, 1));
    pl.off_clseg = take(sizeof(int32_t) * (size_t)std::max<int64_t>(n_cl, 1));
    pl.off_frseg = take(sizeof(int32_t) * (size_t)std::max<int64_t>(n_fr, 1));
    pl.table_bytes = o;
    return o;
}

// Workspace bound that does not depend on tuning: work items, gather items,
// head blocks and hash tiles never outnumber tokens plus segments, and
// selection blocks are bounded by segments, frames and one per
// kSelPartTokens tokens, so one Partial and table entries per token, plus
// what a learned call adds (a PartialX per work item, one
// projection and one head count per token, kMaxMlpHidden floats of the MLP's
// prompt product per request, and the MAS of every (request, modality) that
// a learned run's selection reads). A run with SimHash adds 4 Dsum counts
// per request, within the room of the prompt product.
size_t workspace_bytes_for(int n, int R, int64_t ntok, int64_t nframes)
{
    Plan pl;
    const int64_t items = ntok + n;
    // selection blocks: one per segment, or per frame of a clip, plus the
    // extra blocks of selections of kSelSplitMin tokens or more
    const int64_t sels = n + nframes + ntok / kSelPartTokens + 1;
    const size_t tb = table_layout(pl, n, R, items, items, items, sels, items, items, items);
    return align_up(tb, kWsAlign) + align_up(sizeof(Partial) * (size_t)std::max<int64_t>(items, 1), kWsAlign) +
           align_up(sizeof(PartialX) * (size_t)std::max<int64_t>(items, 1), kWsAlign) +
           align_up(sizeof(float) * (size_t)std::max<int64_t>(ntok, 1), kWsAlign) +
           align_up(sizeof(uint32_t) * (size_t)std::max<int64_t>(items, 1), kWsAlign) +
           align_up(sizeof(float) * (size_t)kMaxMlpHidden * (size_t)std::max(R, 1), kWsAlign) +
           align_up(sizeof(float) * (size_t)kNumMod * (size_t)std::max(R, 1), kWsAlign);
}

// fuse_copy: a full run with compaction, where segments that keep every row
// are copied by the scoring pass (they get no gather items).
void build_plan(const msao_ctx* ctx, const msao_segment* segs, int n, int R, const msao_params* p,
                const float* alpha, const int64_t* out_off, Plan& pl, bool fuse_copy = false,
                const msao_spatial_head* heads = nullptr, bool learned = false, int mlp_hidden = 0,
                const msao_simhash* hashes = nullptr, bool cap_any_scope = false, bool simhash_d = false,
                bool select_imp = false)
{
    const bool per_frame = (p->flags & MSAO_FLAG_SELECT_PER_FRAME) != 0;
    pl.big_seg = ctx ? ctx->post_big_segment : kPostBigSegment;
    pl.sel_unit.clear();
    pl.hi_seg.clear();
    pl.max_n = 0;
    pl.learned = learned;
    pl.mlp_hidden = learned ? mlp_hidden : 0;
    pl.hb_seg.clear();
    pl.max_head_p = 0;
    pl.seg.resize((size_t)n);
    pl.wi_b.assign((size_t)std::max(n, 1), 0);
    pl.wi_e.assign((size_t)std::max(n, 1), 0);
    pl.seg_gi.assign((size_t)n + 1, 0);
    pl.cl_seg.clear();
    pl.clip_fused = false;
    // a run with SimHash scores and hashes its clips in one pass when every
    // clip's tiles of 16 frames fit a 32-bit buffer resource
    // and all clips share one element type and signature width (one kernel instance)
    bool fuse = simhash_d && hashes != nullptr && (!ctx || ctx->clip_fuse);
    int clip_dtype = -1, clip_bits = 0;
    for (int i = 0; fuse && i < n; ++i) {
        if (!is_temporal(segs[i])) continue;
        if ((int64_t)segs[i].tokens_per_frame * segs[i].row_stride * elt_size(segs[i].dtype) * 16 > (int64_t)INT32_MAX)
            fuse = false;
        if (clip_dtype < 0) {
            clip_dtype = segs[i].dtype;
            clip_bits = hashes[i].bits;
        } else if (segs[i].dtype != clip_dtype || hashes[i].bits != clip_bits) {
            fuse = false;
        }
    }
    pl.clip_dtype = clip_dtype;
    pl.clip_bits = clip_bits;
    pl.tseg.clear();
    int64_t tok = 0, frame = 0;
    int wi = 0, gi = 0;
    int64_t chains_total = 0, pairs_total = 0;
    for (int i = 0; i < n; ++i)
        if (is_temporal(segs[i])) {
            chains_total += segs[i].tokens_per_frame;
            pairs_total += (segs[i].tokens_per_frame + 1) / 2;
        }
    // selections before any split: mid-size ones are split only while the
    // launch would otherwise leave CUs without a selection block
    int64_t whole_sels = 0;
    for (int i = 0; i < n; ++i)
        whole_sels += per_frame && segs[i].n_frames >= 2 && segs[i].tokens_per_frame > 0 ? segs[i].n_frames : 1;
    const bool split_mid = whole_sels < kSelSplitMaxSelections;
    for (int i = 0; i < n; ++i) {
        const msao_segment& s = segs[i];
        DevSeg& d = pl.seg[(size_t)i];
        std::memset(&d, 0, sizeof d);
        const int64_t N = (int64_t)s.n_frames * s.tokens_per_frame;
        const int es = elt_size(s.dtype);
        d.data = (const uint8_t*)s.data;
        d.stride_bytes = s.row_stride * es;
        d.out_off = out_off ? out_off[i] : 0;
        d.tok_off = (int32_t)tok;
        d.n_tok = (int32_t)N;
        d.T = s.n_frames;
        d.P = s.tokens_per_frame;
        d.C = s.hidden;
        d.dtype = s.dtype;
        d.modality = s.modality;
        d.request = s.request;
        d.temporal = is_temporal(s) ? 1 : 0;
        d.frame_off = d.temporal ? (int32_t)frame : -1;
        d.nchunk = s.hidden * es / 16;
        d.A_s = (int32_t)std::ceil((double)p->tau_s * (double)s.hidden);
        d.L_s = q24(p->lambda_s[s.modality]);
        d.L_t = q24(p->lambda_t[s.modality]);
        d.lam_s = p->lambda_s[s.modality];
        d.lam_t = p->lambda_t[s.modality];
        d.E = s.hidden;
        d.key_ms = d.L_s;
        d.key_mt = d.L_t;
        if (simhash_d && hashes && d.temporal) {
            // d counts K SimHash bits: keys in units of C K / g
            const int64_t K = hashes[i].bits, g = std::gcd((int64_t)s.hidden, K);
            d.E = (int32_t)K;
            d.key_ms = (uint64_t)d.L_s * (uint64_t)(K / g);
            d.key_mt = (uint64_t)d.L_t * (uint64_t)(s.hidden / g);
        }
        // selections: the segment, or each of its frames (per-frame scope);
        // a large one is written by several blocks, each of a slice
        const bool framed = per_frame && s.n_frames >= 2 && s.tokens_per_frame > 0;
        // a learned run ranks a segment with a head by its Eq. 3 importance
        const bool by_imp = select_imp && learned && heads && heads[i].weight && N > 0;
        const int kind = by_imp ? kKeyImp
                         : d.temporal && d.L_t > 0 ? (d.L_s > 0 ? kKeyFull : kKeyE) : (d.L_s > 0 ? kKeyZ : kKeyZero);
        auto push_selection = [&](int frame, int n_u, int kfix) {
            const int parts = n_u >= pl.big_seg                 ? (n_u + kSelBigPartTokens - 1) / kSelBigPartTokens
                              : n_u >= kSelSplitMin && split_mid ? (n_u + kSelPartTokens - 1) / kSelPartTokens
                                                                 : 1;
            for (int q = 0; q < parts; ++q) {
                SelUnit u;
                std::memset(&u, 0, sizeof u);
                u.Ms = d.key_ms;
                u.Mt = d.key_mt;
                u.kmax = kind == kKeyZ ? (uint64_t)d.C
                         : kind == kKeyE ? (uint64_t)d.E
                         : kind == kKeyFull ? d.key_ms * (uint64_t)d.C + d.key_mt * (uint64_t)d.E
                         : kind == kKeyImp ? 0xFFFFFFFFull : 0ull;
                u.seg = i;
                u.frame = frame;
                u.part = q;
                u.nparts = parts;
                u.off = d.tok_off + (frame >= 0 ? frame * s.tokens_per_frame : 0);
                u.N = n_u;
                u.kfix = kfix;
                u.kind = kind;
                u.E = (uint32_t)d.E;
                u.units = frame >= 0 ? s.n_frames : 1;
                u.seg_off = d.tok_off;
                u.request = s.request;
                u.modality = s.modality;
                pl.sel_unit.push_back(u);
            }
        };
        if (framed) {
            d.kf = s.keep_ratio < 0.0f ? -1 : (int32_t)keep_count(s.keep_ratio, s.tokens_per_frame);
            d.k = d.kf < 0 ? -1 : d.kf * s.n_frames;
            for (int f = 0; f < s.n_frames; ++f) push_selection(f, s.tokens_per_frame, d.kf);
            pl.max_n = std::max(pl.max_n, s.tokens_per_frame);
        } else {
            d.kf = -1;
            d.k = s.keep_ratio < 0.0f ? -1 : (int32_t)keep_count(s.keep_ratio, N);
            push_selection(-1, (int)N, d.k);
            pl.max_n = std::max(pl.max_n, (int)N);
        }
        d.cap = d.k < 0 ? (int32_t)N : d.k;
        // a compaction that does not know the selection's scope (msao_compact)
        // takes room for either: T ceil(kappa P) may exceed ceil(kappa N)
        if (cap_any_scope && d.k >= 0 && s.n_frames >= 2)
            d.cap = std::max<int32_t>(d.cap, s.n_frames * (int32_t)keep_count(s.keep_ratio, s.tokens_per_frame));
        if (hashes) {
            // SimHash blocks of kHashBlockTokens tokens (segments without a hash get zeros)
            d.hi_begin = (int32_t)pl.hi_seg.size();
            if (d.temporal) {
                d.planes = (const uint8_t*)hashes[i].planes;
                d.hash_bits = hashes[i].bits;
            }
            for (int64_t r = 0; r < N; r += kHashBlockTokens) pl.hi_seg.push_back(i);
        }
        d.fused = (fuse && d.temporal) ? 1 : 0;
        // (a fused clip's kept rows are always left to the gather)
        d.copy_in_score = (fuse_copy && out_off && N > 0 && d.k == (int32_t)N && !d.fused) ? 1 : 0;
        if (learned && heads && heads[i].weight && N > 0) {
            d.head_w = (const uint8_t*)heads[i].weight;
            d.head_b = heads[i].bias;
            d.grid_w = heads[i].grid_w > 0 ? heads[i].grid_w : s.tokens_per_frame;
            d.pool = heads[i].pool;
            d.hb_begin = (int32_t)pl.hb_seg.size();
            for (int f = 0; f < s.n_frames; ++f) pl.hb_seg.push_back(i);
            pl.max_head_p = std::max(pl.max_head_p, s.tokens_per_frame);
        }
        // scoring work items, one wavefront each
        int items = 0;
        const int64_t row_bytes = (int64_t)s.hidden * es;
        if (d.temporal && !d.fused && !learned && !d.copy_in_score && (!ctx || ctx->pair_path) && s.dtype == MSAO_BF16 &&
            row_bytes <= kPairMaxRowBytes && row_bytes % 512 == 0 && s.tokens_per_frame >= 2 &&
            d.stride_bytes + row_bytes <= (1 << 30)) {
            // k_pair: one wavefront per pair of positions and range of at most
            // kPairMaxFrames frames (a range after the first reads the frame
            // before it as a halo), the items rounded up to whole blocks (the
            // extra ones have no frames)
            // the range length (halved from the longest, down to
            // kPairMinFrames) with the fewest frames read per SIMD: wavefronts
            // beyond one per SIMD queue behind the first, and a range after a
            // clip's first re-reads one frame; ties keep the longer range
            int F = std::min(s.n_frames, kPairMaxFrames);
            {
                int best = F;
                int64_t best_cost = INT64_MAX;
                for (int f = F;; f = (f + 1) / 2) {
                    const int64_t tb = (s.n_frames + f - 1) / f;
                    const int64_t rounds = (pairs_total * tb + kPairTargetWaves - 1) / kPairTargetWaves;
                    const int64_t cost = rounds * (f + (tb > 1 ? 1 : 0));
                    if (cost < best_cost) {
                        best_cost = cost;
                        best = f;
                    }
                    if (f <= kPairMinFrames) break;
                }
                F = best;
            }
            const int tblk = (s.n_frames + F - 1) / F;
            const int64_t pitems =
                ((int64_t)((s.tokens_per_frame + 1) / 2) * tblk + kPairWaves - 1) / kPairWaves * kPairWaves;
            if (pitems <= N) {
                d.pair = 1;
                d.tblk = tblk;
                d.per_item = F;
                items = (int)pitems;
                pl.tseg.push_back(i);
                pl.any_temporal = true;
            }
        }
        if (d.pair) {
        } else if (d.fused) {
            // tiles of at most 15 new frames of one position, the frames split
            // evenly; their work items follow all others
            d.ntiles = (s.n_frames + kClipFrames - 1) / kClipFrames;
            d.per_item = (s.n_frames + d.ntiles - 1) / d.ntiles;
            pl.tseg.push_back(i);
            pl.any_temporal = true;
            pl.clip_fused = true;
        } else if (d.temporal) {
            int fpi = ctx && ctx->chain_frames > 0 ? ctx->chain_frames : s.n_frames;
            if (!(ctx && ctx->chain_frames > 0)) {
                // split long chains until there are enough wavefronts to cover the chip
                while (fpi > 8 && chains_total * ((s.n_frames + fpi - 1) / fpi) < 4096) fpi = (fpi + 1) / 2;
            }
            fpi = std::min(fpi, s.n_frames);
            d.per_item = fpi;
            items = s.tokens_per_frame * ((s.n_frames + fpi - 1) / fpi);
            pl.tseg.push_back(i);
            pl.any_temporal = true;
        } else if (N > 0) {
            // the fewest rows that reach the target bytes, unless they pass it
            // by more than a quarter (then one row less, at least one)
            const int64_t target = ctx ? ctx->row_item_bytes : 8192, row = (int64_t)s.hidden * es;
            int64_t rb = (target + row - 1) / row;
            if (rb > 1 && rb * row * 4 > target * 5) --rb;
            d.per_item = (int32_t)rb;
            items = (int)((N + rb - 1) / rb);
        } else {
            d.per_item = 1;
        }
        pl.wi_e[(size_t)i] = items;  // the item count until the ranges are laid out below
        d.g_begin = gi;
        if (!d.copy_in_score) gi += (d.cap + kGatherRows - 1) / kGatherRows;
        pl.seg_gi[(size_t)i + 1] = gi;
        if (d.k < 0) pl.any_guided = true;
        if (d.copy_in_score) pl.any_copy = true;
        tok += N;
        if (d.temporal) frame += s.n_frames;
    }
    // work items: k_pair's clips first (whole blocks from item 0), then the
    // other segments in table order, then the fused clips
    for (int pass = 0; pass < 2; ++pass) {
        for (int i = 0; i < n; ++i) {
            DevSeg& d = pl.seg[(size_t)i];
            if (d.fused || (d.pair != 0) != (pass == 0)) continue;
            const int items = pl.wi_e[(size_t)i];
            d.wi_begin = wi;
            pl.wi_b[(size_t)i] = wi;
            wi += items;
            pl.wi_e[(size_t)i] = wi;
        }
        if (pass == 0) pl.n_wi_pair = wi;
    }
    pl.n_wi_score = wi;
    for (int i = 0; i < n; ++i) {
        DevSeg& d = pl.seg[(size_t)i];
        if (!d.fused) continue;
        const int items = d.P * d.ntiles;
        d.wi_begin = wi;
        pl.wi_b[(size_t)i] = wi;
        wi += items;
        pl.wi_e[(size_t)i] = wi;
        d.cl_begin = (int32_t)pl.cl_seg.size();
        for (int b = 0; b < (items + kClipWaves - 1) / kClipWaves; ++b) pl.cl_seg.push_back(i);
    }
    pl.ntok = tok;
    pl.nframes = frame;
    pl.n_wi = wi;
    pl.n_gwi = gi;
    // segments grouped by (request, modality), table order inside a group
    pl.rm.assign((size_t)std::max(R * kNumMod, 1), RmEntry{});
    std::vector<int32_t> count((size_t)R * kNumMod + 1, 0);
    for (int i = 0; i < n; ++i) count[(size_t)(segs[i].request * kNumMod + segs[i].modality) + 1]++;
    for (size_t x = 1; x < count.size(); ++x) count[x] += count[x - 1];
    for (int x = 0; x < R * kNumMod; ++x) {
        pl.rm[(size_t)x].rng_begin = count[(size_t)x];
        pl.rm[(size_t)x].rng_end = count[(size_t)x + 1];
    }
    pl.rm_rng.assign((size_t)std::max(n, 1), WiRange{0, 0, 0, 0});
    for (int i = 0; i < n; ++i) {
        const msao_segment& s = segs[i];
        const DevSeg& d = pl.seg[(size_t)i];
        RmEntry& e = pl.rm[(size_t)(s.request * kNumMod + s.modality)];
        e.ntok += (uint64_t)d.n_tok;
        if (d.temporal) e.qbits += (uint64_t)(d.T - 1) * (uint64_t)d.P * (uint64_t)d.E;
        pl.rm_rng[(size_t)count[(size_t)(s.request * kNumMod + s.modality)]++] =
            WiRange{pl.wi_b[(size_t)i], pl.wi_e[(size_t)i], i, 0};
    }
    pl.wi_seg.resize((size_t)pl.n_wi);
    pl.gi_seg.resize((size_t)pl.n_gwi);
    for (int i = 0; i < n; ++i) {
        std::fill(pl.wi_seg.begin() + pl.wi_b[(size_t)i], pl.wi_seg.begin() + pl.wi_e[(size_t)i], i);
        std::fill(pl.gi_seg.begin() + pl.seg_gi[(size_t)i], pl.gi_seg.begin() + pl.seg_gi[(size_t)i + 1], i);
    }
    pl.alpha.assign((size_t)std::max(R * kNumMod, 1), 0.0f);
    if (alpha)
        for (int x = 0; x < R * kNumMod; ++x) pl.alpha[(size_t)x] = alpha[x];
    pl.frame_seg.clear();
    for (int i = 0; i < n; ++i)
        if (pl.seg[(size_t)i].temporal) pl.frame_seg.insert(pl.frame_seg.end(), (size_t)pl.seg[(size_t)i].T, i);
    table_layout(pl, n, R, pl.n_wi, pl.n_gwi, (int64_t)pl.hb_seg.size(), (int64_t)pl.sel_unit.size(),
                 (int64_t)pl.hi_seg.size(), (int64_t)pl.cl_seg.size(), (int64_t)pl.frame_seg.size());
    pl.off_partial = align_up(pl.table_bytes, kWsAlign);
    pl.total_bytes = pl.off_partial + sizeof(Partial) * (size_t)std::max(pl.n_wi, 1);
    pl.simhash_d = simhash_d && pl.any_temporal;
    if (pl.simhash_d && !pl.clip_fused) {
        pl.off_hdsum = align_up(pl.total_bytes, kWsAlign);
        pl.total_bytes = pl.off_hdsum + sizeof(uint64_t) * (size_t)std::max(R * kNumMod, 1);
    }
    if (learned) {
        pl.off_partial_x = align_up(pl.total_bytes, kWsAlign);
        pl.off_proj = align_up(pl.off_partial_x + sizeof(PartialX) * (size_t)std::max(pl.n_wi, 1), kWsAlign);
        pl.off_head_count = align_up(pl.off_proj + sizeof(float) * (size_t)std::max<int64_t>(pl.ntok, 1), kWsAlign);
        pl.total_bytes = pl.off_head_count + sizeof(uint32_t) * std::max<size_t>(pl.hb_seg.size(), 1);
        if (pl.mlp_hidden > 0) {
            pl.off_mlp_u = align_up(pl.total_bytes, kWsAlign);
            pl.total_bytes = pl.off_mlp_u + sizeof(float) * (size_t)pl.mlp_hidden * (size_t)std::max(R, 1);
        }
        if (select_imp) {  // the learned MAS, read by the selection launch
            pl.off_mas = align_up(pl.total_bytes, kWsAlign);
            pl.total_bytes = pl.off_mas + sizeof(float) * (size_t)std::max(R * kNumMod, 1);
        }
    }
}

#define MSAO_TRY(x)                                                                                                   \
    do {                                                                                                              \
        msao_status st_ = (x);                                                                                        \
        if (st_ != MSAO_OK) return st_;                                                                               \
    } while (0)

msao_status hip_fail(msao_ctx* ctx, hipError_t e, const char* what)
{
    ctx->err = std::string(what) + ": " + hipGetErrorString(e);
    return MSAO_ERR_HIP;
}

struct DeviceGuard {
    int prev = -1;
    bool changed = false;
    explicit DeviceGuard(int dev)
    {
        if (hipGetDevice(&prev) == hipSuccess && prev != dev) changed = hipSetDevice(dev) == hipSuccess;
    }
    ~DeviceGuard()
    {
        if (changed) (void)hipSetDevice(prev);
    }
};

// Pinned staging slot `slot` of at least `bytes` (grown when smaller).
msao_status reserve_stage(msao_ctx* ctx, int slot, size_t bytes)
{
    if (ctx->stage_cap[slot] >= bytes) return MSAO_OK;
    if (ctx->stage[slot]) (void)hipHostFree(ctx->stage[slot]);
    ctx->stage[slot] = nullptr;
    ctx->stage_cap[slot] = 0;
    const size_t cap = align_up(std::max<size_t>(bytes, 65536), 65536);
    const hipError_t e = hipHostMalloc(&ctx->stage[slot], cap, hipHostMallocDefault);
    if (e != hipSuccess) return hip_fail(ctx, e, "hipHostMalloc");
    ctx->stage_cap[slot] = cap;
    return MSAO_OK;
}

// Copy the tables into a pinned slot and enqueue its upload into the
// workspace. With grow false a slot smaller than the tables is an error
// instead of a new pinned allocation (msao_run_noalloc allocates nothing).
msao_status upload(msao_ctx* ctx, const Plan& pl, void* ws, hipStream_t stream, bool grow = true)
{
    const int slot = ctx->next_slot;
    hipError_t e;
    if (!grow && ctx->stage_cap[slot] < pl.table_bytes)
        return fail(&ctx->err, MSAO_ERR_UNSUPPORTED, "per-call tables larger than the context's reserved staging");
    ctx->next_slot ^= 1;
    if (ctx->stage_used[slot]) {
        if ((e = hipEventSynchronize(ctx->stage_ev[slot])) != hipSuccess) return hip_fail(ctx, e, "hipEventSynchronize");
    }
    if (ctx->stage_cap[slot] < pl.table_bytes) MSAO_TRY(reserve_stage(ctx, slot, pl.table_bytes));
    uint8_t* h = (uint8_t*)ctx->stage[slot];
    std::memset(h, 0, pl.table_bytes);
    auto put = [&](size_t off, const void* src, size_t bytes) {
        if (bytes) std::memcpy(h + off, src, bytes);
    };
    put(pl.off_seg, pl.seg.data(), sizeof(DevSeg) * pl.seg.size());
    put(pl.off_wi, pl.wi_seg.data(), sizeof(int32_t) * pl.wi_seg.size());
    put(pl.off_gi, pl.gi_seg.data(), sizeof(int32_t) * pl.gi_seg.size());
    put(pl.off_rmoff, pl.rm.data(), sizeof(RmEntry) * pl.rm.size());
    put(pl.off_rmseg, pl.rm_rng.data(), sizeof(WiRange) * pl.rm_rng.size());
    put(pl.off_tseg, pl.tseg.data(), sizeof(int32_t) * pl.tseg.size());
    put(pl.off_alpha, pl.alpha.data(), sizeof(float) * pl.alpha.size());
    put(pl.off_hbseg, pl.hb_seg.data(), sizeof(int32_t) * pl.hb_seg.size());
    put(pl.off_selu, pl.sel_unit.data(), sizeof(SelUnit) * pl.sel_unit.size());
    put(pl.off_hiseg, pl.hi_seg.data(), sizeof(int32_t) * pl.hi_seg.size());
    put(pl.off_clseg, pl.cl_seg.data(), sizeof(int32_t) * pl.cl_seg.size());
    put(pl.off_frseg, pl.frame_seg.data(), sizeof(int32_t) * pl.frame_seg.size());
    if ((e = hipMemcpyAsync(ws, h, pl.table_bytes, hipMemcpyHostToDevice, stream)) != hipSuccess)
        return hip_fail(ctx, e, "hipMemcpyAsync");
    if ((e = hipEventRecord(ctx->stage_ev[slot], stream)) != hipSuccess) return hip_fail(ctx, e, "hipEventRecord");
    ctx->stage_used[slot] = true;
    return MSAO_OK;
}

Tables device_tables(const Plan& pl, void* ws, int n, int R, const msao_params* p)
{
    uint8_t* b = (uint8_t*)ws;
    Tables t;
    std::memset(&t, 0, sizeof t);
    t.seg = (const DevSeg*)(b + pl.off_seg);
    t.wi_seg = (const int32_t*)(b + pl.off_wi);
    t.gi_seg = (const int32_t*)(b + pl.off_gi);
    t.rm = (const RmEntry*)(b + pl.off_rmoff);
    t.rm_rng = (const WiRange*)(b + pl.off_rmseg);
    t.tseg = (const int32_t*)(b + pl.off_tseg);
    t.alpha = (const float*)(b + pl.off_alpha);
    t.partial = (Partial*)(b + pl.off_partial);
    t.partial_x = pl.learned ? (PartialX*)(b + pl.off_partial_x) : nullptr;
    t.proj = pl.learned ? (float*)(b + pl.off_proj) : nullptr;
    t.head_count = pl.learned ? (uint32_t*)(b + pl.off_head_count) : nullptr;
    t.hb_seg = (const int32_t*)(b + pl.off_hbseg);
    t.n_hb = (int32_t)pl.hb_seg.size();
    t.sel_unit = (const SelUnit*)(b + pl.off_selu);
    t.hi_seg = (const int32_t*)(b + pl.off_hiseg);
    t.hdsum = pl.simhash_d && !pl.clip_fused ? (const uint64_t*)(b + pl.off_hdsum) : nullptr;
    t.cl_seg = (const int32_t*)(b + pl.off_clseg);
    t.frame_seg = (const int32_t*)(b + pl.off_frseg);
    t.n_cl = (int32_t)pl.cl_seg.size();
    t.n_wi_score = pl.n_wi_score;
    t.n_wi_pair = pl.n_wi_pair;
    t.n_hi = (int32_t)pl.hi_seg.size();
    t.n = n;
    t.R = R;
    t.n_wi = pl.n_wi;
    t.n_gwi = pl.n_gwi;
    t.n_tseg = (int)pl.tseg.size();
    t.n_frames = (int)pl.nframes;
    // -0 passes the tau >= 0 check; the bf16 kernels take their threshold
    // from the float's bits, where -0 would read as 0x8000 (above every
    // magnitude), so it goes down as +0, the same threshold.
    t.tau = p->tau == 0.0f ? 0.0f : p->tau;
    t.tau_s = p->tau_s;
    for (int m = 0; m < kNumMod; ++m) {
        t.lam_s[m] = p->lambda_s[m];
        t.lam_t[m] = p->lambda_t[m];
    }
    t.flags = p->flags;
    return t;
}

msao_status check_ws(msao_ctx* ctx, const Plan& pl, void* ws, size_t ws_bytes)
{
    if (!ws) return fail(&ctx->err, MSAO_ERR_WORKSPACE, "workspace is NULL");
    if (((uintptr_t)ws) % kWsAlign != 0) return fail(&ctx->err, MSAO_ERR_WORKSPACE, "workspace is not 256-byte aligned");
    if (ws_bytes < pl.total_bytes) {
        char buf[160];
        std::snprintf(buf, sizeof buf, "workspace too small: %zu bytes given, %zu needed", ws_bytes, pl.total_bytes);
        return fail(&ctx->err, MSAO_ERR_WORKSPACE, buf);
    }
    return MSAO_OK;
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p) % a == 0; }

// Output arrays of 4 or 8 bytes must be naturally aligned.
msao_status check_out_alignment(msao_ctx* ctx, std::initializer_list<std::pair<const void*, size_t>> ptrs)
{
    for (const auto& pr : ptrs)
        if (pr.first && !aligned(pr.first, pr.second))
            return fail(&ctx->err, MSAO_ERR_ALIGNMENT, "an output array is not naturally aligned");
    return MSAO_OK;
}

hipEvent_t pooled_event(msao_ctx* ctx)
{
    if (!ctx->pool.empty()) {
        hipEvent_t e = ctx->pool.back();
        ctx->pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    return hipEventCreate(&e) == hipSuccess ? e : nullptr;
}

// Launch, with profiling events recorded at the kernel's start and end.
msao_status launched(msao_ctx* ctx, int kernel, hipStream_t stream, int (*fn)(const void*, void*, void*, void*),
                     const void* args)
{
    hipEvent_t e0 = nullptr, e1 = nullptr;
    if (ctx->profiling) {
        e0 = pooled_event(ctx);
        e1 = pooled_event(ctx);
        if (!e0 || !e1) return fail(&ctx->err, MSAO_ERR_HIP, "hipEventCreate failed");
    }
    const int rc = fn(args, stream, e0, e1);
    if (rc == kNoLaunch) {  // nothing to launch: the events were not recorded
        if (e0) ctx->pool.push_back(e0);
        if (e1) ctx->pool.push_back(e1);
        return MSAO_OK;
    }
    if (rc != 0) return hip_fail(ctx, (hipError_t)rc, "kernel launch");
    if (ctx->profiling) ctx->rec[kernel].push_back({e0, e1});
    return MSAO_OK;
}

int run_score(const void* a, void* s, void* e0, void* e1) { return launch_score(*(const ScoreArgs*)a, s, e0, e1); }
int run_post(const void* a, void* s, void* e0, void* e1) { return launch_post(*(const PostArgs*)a, s, e0, e1); }
int run_gather(const void* a, void* s, void* e0, void* e1) { return launch_gather(*(const GatherArgs*)a, s, e0, e1); }
int run_entropy(const void* a, void* s, void* e0, void* e1) { return launch_entropy(*(const EntArgs*)a, s, e0, e1); }
int run_head(const void* a, void* s, void* e0, void* e1) { return launch_head(*(const HeadArgs*)a, s, e0, e1); }
int run_simhash(const void* a, void* s, void* e0, void* e1) { return launch_simhash(*(const HashArgs*)a, s, e0, e1); }
int run_clip(const void* a, void* s, void* e0, void* e1) { return launch_clip(*(const ClipArgs*)a, s, e0, e1); }
int run_read(const void* a, void* s, void* e0, void* e1) { return launch_read(*(const ReadArgs*)a, s, e0, e1); }
int run_hash_post(const void* a, void* s, void* e0, void* e1)
{
    return launch_hash_post(*(const HashArgs*)a, s, e0, e1);
}

// Scoring block order. The order with one contiguous range of work items per
// XCD makes the per-token statistic stores cheaper, but was measured slower
// when the scoring pass also writes compacted rows, so it is used only for
// launches that copy no rows (unless MSAO_XCD_ORDER forces either order).
int32_t xcd_order_for(const msao_ctx* ctx, bool copies_rows)
{
    if (ctx->xcd_order >= 0) return ctx->xcd_order ? 1 : 0;
    return copies_rows ? 0 : 1;
}

TokenOut token_out(const msao_token_out* t)
{
    TokenOut o{};
    if (t) o = TokenOut{t->z, t->l1, t->l2, t->info, t->d, t->res};
    return o;
}

msao_status check_compact_out(msao_ctx* ctx, const Plan& pl, const msao_segment* segs, int n, void* out,
                              const int64_t* off, int64_t out_bytes)
{
    if (!out) return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "compaction output is NULL");
    if (!off) return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "out_byte_off is NULL");
    if (!aligned(out, 16)) return fail(&ctx->err, MSAO_ERR_ALIGNMENT, "out is not 16-byte aligned");
    for (int i = 0; i < n; ++i) {
        const DevSeg& d = pl.seg[(size_t)i];
        const int64_t need = (int64_t)d.cap * segs[i].hidden * elt_size(segs[i].dtype);
        if (off[i] < 0 || off[i] % 16 != 0) return fail(&ctx->err, MSAO_ERR_ALIGNMENT, "out_byte_off entry negative or not 16-byte aligned");
        if (off[i] + need > out_bytes) return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "compaction output too small for a segment's rows");
    }
    return MSAO_OK;
}

// The hash of every temporal segment (SimHash calls).
msao_status check_hashes(msao_ctx* ctx, const msao_segment* segs, int n, const msao_simhash* hashes)
{
    if (n > 0 && !hashes) return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "hashes is NULL");
    char buf[160];
    for (int i = 0; i < n; ++i) {
        const msao_segment& s = segs[i];
        if (!is_temporal(s)) continue;
        auto bad = [&](msao_status st, const char* what) {
            std::snprintf(buf, sizeof buf, "hash of segment %d: %s", i, what);
            return fail(&ctx->err, st, buf);
        };
        const msao_simhash& h = hashes[i];
        if (!h.planes) return bad(MSAO_ERR_INVALID_ARG, "planes is NULL");
        if (h.bits != 16 && h.bits != 32 && h.bits != 48 && h.bits != 64)
            return bad(MSAO_ERR_INVALID_ARG, "bits must be 16, 32, 48 or 64");
        if (!aligned(h.planes, 16)) return bad(MSAO_ERR_ALIGNMENT, "planes is not 16-byte aligned");
        // a hash tile's rows are one buffer resource of kHashTokens pitches (32-bit size)
        if (s.row_stride * elt_size(s.dtype) * kHashTokens > (int64_t)INT32_MAX)
            return bad(MSAO_ERR_UNSUPPORTED, "row pitch too large for a hash tile (64 MiB or more)");
    }
    return MSAO_OK;
}

}  // namespace

// ---------------------------------------------------------------- C ABI

extern "C" {

const char* msao_status_string(msao_status s)
{
    switch (s) {
    case MSAO_OK: return "MSAO_OK";
    case MSAO_ERR_INVALID_ARG: return "MSAO_ERR_INVALID_ARG";
    case MSAO_ERR_ALIGNMENT: return "MSAO_ERR_ALIGNMENT";
    case MSAO_ERR_WORKSPACE: return "MSAO_ERR_WORKSPACE";
    case MSAO_ERR_UNSUPPORTED: return "MSAO_ERR_UNSUPPORTED";
    case MSAO_ERR_HIP: return "MSAO_ERR_HIP";
    }
    return "unknown status";
}

msao_params msao_default_params(void)
{
    msao_params p;
    std::memset(&p, 0, sizeof p);
    p.tau = 0.1f;
    p.tau_s = 0.3f;
    p.lambda_s[MSAO_TEXT] = 0.0f;
    p.lambda_s[MSAO_IMAGE] = 0.6f;
    p.lambda_s[MSAO_VIDEO] = 0.6f;
    p.lambda_s[MSAO_AUDIO] = 0.6f;
    p.lambda_t[MSAO_VIDEO] = 0.4f;
    p.flags = 0;
    return p;
}

const char* msao_last_error(const msao_ctx* ctx) { return ctx ? ctx->err.c_str() : "context is NULL"; }

const char* msao_last_error_global(void) { return g_err.c_str(); }

msao_status msao_validate(const msao_segment* segs, int n, int n_requests, const msao_params* params)
{
    return validate_impl(segs, n, n_requests, params, &g_err);
}

msao_status msao_count(const msao_segment* segs, int n, int64_t* n_tokens, int64_t* n_frames)
{
    if (n < 0 || (n > 0 && !segs) || !n_tokens || !n_frames)
        return fail(&g_err, MSAO_ERR_INVALID_ARG, "msao_count: bad arguments");
    int64_t t = 0, f = 0;
    for (int i = 0; i < n; ++i) {
        if (segs[i].n_frames < 1 || segs[i].tokens_per_frame < 0)
            return fail(&g_err, MSAO_ERR_INVALID_ARG, "msao_count: bad segment shape");
        t += (int64_t)segs[i].n_frames * segs[i].tokens_per_frame;
        if (is_temporal(segs[i])) f += segs[i].n_frames;
    }
    *n_tokens = t;
    *n_frames = f;
    return MSAO_OK;
}

msao_status msao_workspace_size(const msao_segment* segs, int n, int n_requests, size_t* bytes)
{
    if (!bytes) return fail(&g_err, MSAO_ERR_INVALID_ARG, "bytes is NULL");
    msao_params p = msao_default_params();
    MSAO_TRY(validate_impl(segs, n, n_requests, &p, &g_err));
    int64_t t = 0, f = 0;
    MSAO_TRY(msao_count(segs, n, &t, &f));
    int64_t frames_all = 0;  // frames of every segment of two or more (per-frame scope)
    for (int i = 0; i < n; ++i)
        if (segs[i].n_frames >= 2) frames_all += segs[i].n_frames;
    *bytes = workspace_bytes_for(n, n_requests, t, frames_all);
    return MSAO_OK;
}

msao_status msao_compact_layout(const msao_segment* segs, int n, int64_t* out_byte_off, int64_t* total_bytes)
{
    if (n < 0 || (n > 0 && (!segs || !out_byte_off)) || !total_bytes)
        return fail(&g_err, MSAO_ERR_INVALID_ARG, "msao_compact_layout: bad arguments");
    int64_t o = 0;
    for (int i = 0; i < n; ++i) {
        const msao_segment& s = segs[i];
        const int64_t N = (int64_t)s.n_frames * s.tokens_per_frame;
        if (s.n_frames < 1 || s.tokens_per_frame < 0 || std::isnan(s.keep_ratio))
            return fail(&g_err, MSAO_ERR_INVALID_ARG, "msao_compact_layout: bad segment");
        int64_t cap = s.keep_ratio < 0.0f ? N : keep_count(s.keep_ratio, N);
        if (s.keep_ratio >= 0.0f && s.n_frames >= 2)  // room for the per-frame scope's count too
            cap = std::max<int64_t>(cap, s.n_frames * keep_count(s.keep_ratio, s.tokens_per_frame));
        out_byte_off[i] = o;
        o = (int64_t)align_up((size_t)(o + cap * (int64_t)s.hidden * elt_size(s.dtype)), kWsAlign);
    }
    *total_bytes = o;
    return MSAO_OK;
}

msao_status msao_create(msao_ctx** out, int device)
{
    if (!out) return fail(&g_err, MSAO_ERR_INVALID_ARG, "ctx pointer is NULL");
    *out = nullptr;
    int count = 0;
    hipError_t e = hipGetDeviceCount(&count);
    if (e != hipSuccess || count <= 0) return fail(&g_err, MSAO_ERR_HIP, "no HIP device available");
    if (device < 0 || device >= count) return fail(&g_err, MSAO_ERR_INVALID_ARG, "device id out of range");
    msao_ctx* c = new msao_ctx();
    c->device = device;
    DeviceGuard guard(device);
    for (int i = 0; i < 2; ++i) {
        if ((e = hipEventCreateWithFlags(&c->stage_ev[i], hipEventDisableTiming)) != hipSuccess) {
            g_err = std::string("hipEventCreate: ") + hipGetErrorString(e);
            msao_destroy(c);
            return MSAO_ERR_HIP;
        }
    }
    // set-up of msao_run_noalloc, which allocates nothing: both staging slots
    // hold its largest tables, and this device's copy of the library's
    // scratch array has its device address looked up
    for (int i = 0; i < 2; ++i) {
        if (reserve_stage(c, i, kNoAllocTableBytes) != MSAO_OK) {
            g_err = c->err;
            msao_destroy(c);
            return MSAO_ERR_HIP;
        }
    }
    if ((e = (hipError_t)scratch_init(device)) != hipSuccess) {
        g_err = std::string("hipGetSymbolAddress of the scratch array: ") + hipGetErrorString(e);
        msao_destroy(c);
        return MSAO_ERR_HIP;
    }
    if (const char* v = std::getenv("MSAO_ROW_ITEM_BYTES")) c->row_item_bytes = std::max(1, std::atoi(v));
    if (const char* v = std::getenv("MSAO_CHAIN_FRAMES")) c->chain_frames = std::max(0, std::atoi(v));
    if (const char* v = std::getenv("MSAO_XCD_ORDER")) c->xcd_order = std::atoi(v) < 0 ? -1 : (std::atoi(v) ? 1 : 0);
    if (const char* v = std::getenv("MSAO_CLIP_FUSE")) c->clip_fuse = std::atoi(v) ? 1 : 0;
    if (const char* v = std::getenv("MSAO_PAIR")) c->pair_path = std::atoi(v) ? 1 : 0;
    if (const char* v = std::getenv("MSAO_POST_BIG_SEGMENT")) c->post_big_segment = std::max(1, std::atoi(v));
    *out = c;
    return MSAO_OK;
}

void msao_destroy(msao_ctx* ctx)
{
    if (!ctx) return;
    DeviceGuard guard(ctx->device);
    for (int i = 0; i < 2; ++i) {
        if (ctx->stage_ev[i]) {
            if (ctx->stage_used[i]) (void)hipEventSynchronize(ctx->stage_ev[i]);
            (void)hipEventDestroy(ctx->stage_ev[i]);
        }
        if (ctx->stage[i]) (void)hipHostFree(ctx->stage[i]);
    }
    for (int k = 0; k < MSAO_NUM_KERNELS; ++k)
        for (auto& pr : ctx->rec[k]) {
            (void)hipEventSynchronize(pr.second);
            ctx->pool.push_back(pr.first);
            ctx->pool.push_back(pr.second);
        }
    for (hipEvent_t e : ctx->pool) (void)hipEventDestroy(e);
    delete ctx;
}

static_assert(kClipWaves == 4 || kClipWaves == 8, "k_clip is built and tested with 4 or 8 tiles per block");

msao_status msao_set_profiling(msao_ctx* ctx, int enable)
{
    if (!ctx) return MSAO_ERR_INVALID_ARG;
    ctx->profiling = enable != 0;
    return MSAO_OK;
}

msao_status msao_kernel_times(msao_ctx* ctx, float* ms)
{
    if (!ctx || !ms) return MSAO_ERR_INVALID_ARG;
    DeviceGuard guard(ctx->device);
    msao_status st = MSAO_OK;
    for (int k = 0; k < MSAO_NUM_KERNELS; ++k) {
        double sum = 0.0;
        for (auto& pr : ctx->rec[k]) {
            float t = 0.0f;
            hipError_t e = hipEventSynchronize(pr.second);
            if (e == hipSuccess) e = hipEventElapsedTime(&t, pr.first, pr.second);
            if (e != hipSuccess && st == MSAO_OK) st = hip_fail(ctx, e, "msao_kernel_times");
            sum += t;
            ctx->pool.push_back(pr.first);
            ctx->pool.push_back(pr.second);
        }
        ms[k] = ctx->rec[k].empty() ? 0.0f : (float)(sum / (double)ctx->rec[k].size());
        ctx->rec[k].clear();
    }
    return st;
}

msao_status msao_mas_score(msao_ctx* ctx, const msao_segment* segs, int n, int R, const msao_params* params,
                           const float* alpha, const msao_token_out* tok, const msao_frame_out* frm,
                           const msao_req_out* req, void* ws, size_t ws_bytes, void* stream)
{
    if (!ctx) return fail(&g_err, MSAO_ERR_INVALID_ARG, "ctx is NULL");
    MSAO_TRY(validate_impl(segs, n, R, params, &ctx->err));
    Plan pl;
    build_plan(ctx, segs, n, R, params, alpha, nullptr, pl);
    MSAO_TRY(check_ws(ctx, pl, ws, ws_bytes));
    const bool want_frames = frm && (frm->dframe || frm->sim || frm->gamma) && pl.nframes > 0;
    if (want_frames && !(tok && tok->d))
        return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "per-frame outputs need tok->d");
    if (tok) MSAO_TRY(check_out_alignment(ctx, {{tok->z, 4}, {tok->l1, 4}, {tok->l2, 4}, {tok->info, 4}, {tok->d, 4}, {tok->res, 4}}));
    if (frm) MSAO_TRY(check_out_alignment(ctx, {{frm->dframe, 8}, {frm->sim, 4}, {frm->gamma, 4}}));
    if (req) MSAO_TRY(check_out_alignment(ctx, {{req->agg, 8}, {req->rho, 4}, {req->temporal, 4}, {req->beta, 4}, {req->mas, 4}}));
    DeviceGuard guard(ctx->device);
    hipStream_t st = (hipStream_t)stream;
    MSAO_TRY(upload(ctx, pl, ws, st));
    ScoreArgs sa;
    std::memset(&sa, 0, sizeof sa);
    sa.t = device_tables(pl, ws, n, R, params);
    sa.tok = token_out(tok);
    sa.out = nullptr;
    sa.mode = kModeScore;
    sa.xcd_order = xcd_order_for(ctx, false);
    MSAO_TRY(launched(ctx, MSAO_KERNEL_SCORE, st, run_score, &sa));
    PostArgs pa;
    std::memset(&pa, 0, sizeof pa);
    pa.t = sa.t;
    if (req) pa.req = ReqOut{req->agg, req->rho, req->temporal, req->beta, req->mas, req->present};
    if (frm) pa.frm = FrameOut{frm->dframe, frm->sim, frm->gamma};
    pa.d = tok ? tok->d : nullptr;
    const bool want_req = req && (req->agg || req->rho || req->temporal || req->beta || req->mas || req->present);
    pa.n_req_blocks = want_req ? R : 0;
    pa.n_frame_blocks = want_frames ? (int)pl.nframes : 0;
    pa.n_sel_blocks = 0;
    return launched(ctx, MSAO_KERNEL_POST, st, run_post, &pa);
}

msao_status msao_temporal_redundancy(msao_ctx* ctx, const msao_segment* segs, int n, int R,
                                     const msao_params* params, uint32_t* d, float* res,
                                     const msao_frame_out* frm, float* temporal, void* ws, size_t ws_bytes,
                                     void* stream)
{
    if (!ctx) return fail(&g_err, MSAO_ERR_INVALID_ARG, "ctx is NULL");
    MSAO_TRY(validate_impl(segs, n, R, params, &ctx->err));
    Plan pl;
    build_plan(ctx, segs, n, R, params, nullptr, nullptr, pl);
    MSAO_TRY(check_ws(ctx, pl, ws, ws_bytes));
    const bool want_frames = frm && (frm->dframe || frm->sim || frm->gamma) && pl.nframes > 0;
    if (want_frames && !d) return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "per-frame outputs need d");
    MSAO_TRY(check_out_alignment(ctx, {{d, 4}, {res, 4}, {temporal, 4}}));
    if (frm) MSAO_TRY(check_out_alignment(ctx, {{frm->dframe, 8}, {frm->sim, 4}, {frm->gamma, 4}}));
    DeviceGuard guard(ctx->device);
    hipStream_t st = (hipStream_t)stream;
    MSAO_TRY(upload(ctx, pl, ws, st));
    ScoreArgs sa;
    std::memset(&sa, 0, sizeof sa);
    sa.t = device_tables(pl, ws, n, R, params);
    sa.tok.d = d;
    sa.tok.res = res;
    sa.mode = kModeTemporal;
    sa.xcd_order = xcd_order_for(ctx, false);
    MSAO_TRY(launched(ctx, MSAO_KERNEL_SCORE, st, run_score, &sa));
    PostArgs pa;
    std::memset(&pa, 0, sizeof pa);
    pa.t = sa.t;
    if (frm) pa.frm = FrameOut{frm->dframe, frm->sim, frm->gamma};
    pa.req.temporal = temporal;
    pa.d = d;
    pa.temporal_only = 1;
    pa.n_req_blocks = temporal ? R : 0;
    pa.n_frame_blocks = want_frames ? (int)pl.nframes : 0;
    return launched(ctx, MSAO_KERNEL_POST, st, run_post, &pa);
}

msao_status msao_temporal_simhash(msao_ctx* ctx, const msao_segment* segs, int n, int R, const msao_params* params,
                                  const msao_simhash* hashes, uint64_t* sig, uint32_t* d, const msao_frame_out* frm,
                                  float* temporal, void* ws, size_t ws_bytes, void* stream)
{
    if (!ctx) return fail(&g_err, MSAO_ERR_INVALID_ARG, "ctx is NULL");
    MSAO_TRY(validate_impl(segs, n, R, params, &ctx->err));
    MSAO_TRY(check_hashes(ctx, segs, n, hashes));
    Plan pl;
    build_plan(ctx, segs, n, R, params, nullptr, nullptr, pl, false, nullptr, false, 0, hashes);
    MSAO_TRY(check_ws(ctx, pl, ws, ws_bytes));
    if (pl.ntok > 0 && (!sig || !d)) return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "sig and d are required");
    MSAO_TRY(check_out_alignment(ctx, {{sig, 8}, {d, 4}, {temporal, 4}}));
    if (frm) MSAO_TRY(check_out_alignment(ctx, {{frm->dframe, 8}, {frm->sim, 4}, {frm->gamma, 4}}));
    DeviceGuard guard(ctx->device);
    hipStream_t st = (hipStream_t)stream;
    MSAO_TRY(upload(ctx, pl, ws, st));
    HashArgs ha;
    std::memset(&ha, 0, sizeof ha);
    ha.t = device_tables(pl, ws, n, R, params);
    ha.sig = sig;
    ha.d = d;
    if (frm) ha.frm = FrameOut{frm->dframe, frm->sim, frm->gamma};
    ha.temporal = temporal;
    MSAO_TRY(launched(ctx, MSAO_KERNEL_SIMHASH, st, run_simhash, &ha));
    // frame blocks write d for every temporal token, so they always run
    ha.n_frame_blocks = (int)pl.nframes;
    ha.n_req_blocks = temporal ? R : 0;
    return launched(ctx, MSAO_KERNEL_HASH_POST, st, run_hash_post, &ha);
}

msao_status msao_select_tokens(msao_ctx* ctx, const msao_segment* segs, int n, int R, const msao_params* params,
                               const uint32_t* z, const uint32_t* d, const float* mas, const msao_select_out* sel,
                               void* ws, size_t ws_bytes, void* stream)
{
    if (!ctx) return fail(&g_err, MSAO_ERR_INVALID_ARG, "ctx is NULL");
    MSAO_TRY(validate_impl(segs, n, R, params, &ctx->err));
    Plan pl;
    build_plan(ctx, segs, n, R, params, nullptr, nullptr, pl);
    MSAO_TRY(check_ws(ctx, pl, ws, ws_bytes));
    if (!sel || !sel->kept_idx || !sel->kept_count)
        return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "selection needs kept_idx and kept_count");
    if (pl.ntok > 0 && !z) return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "z is NULL");
    if (pl.any_temporal && !d) return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "d is NULL but a segment is temporal");
    if (pl.any_guided && !mas) return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "mas is NULL but a keep ratio is negative");
    MSAO_TRY(check_out_alignment(ctx, {{z, 4}, {d, 4}, {mas, 4}, {sel->kept_idx, 4}, {sel->kept_count, 4}}));
    DeviceGuard guard(ctx->device);
    hipStream_t st = (hipStream_t)stream;
    MSAO_TRY(upload(ctx, pl, ws, st));
    PostArgs pa;
    std::memset(&pa, 0, sizeof pa);
    pa.t = device_tables(pl, ws, n, R, params);
    pa.sel = SelOut{sel->keep, sel->kept_idx, sel->kept_count};
    pa.z = z;
    pa.d = d;
    pa.mas_in = mas;
    pa.n_sel_blocks = (int)pl.sel_unit.size();
    pa.keys_cap = std::min(pl.max_n, kMaxLdsKeys);
    pa.big_block = pl.max_n >= pl.big_seg ? 1 : 0;
    return launched(ctx, MSAO_KERNEL_POST, st, run_post, &pa);
}

msao_status msao_compact(msao_ctx* ctx, const msao_segment* segs, int n, const int32_t* kept_idx,
                         const int32_t* kept_count, void* out, const int64_t* out_byte_off, int64_t out_bytes,
                         void* ws, size_t ws_bytes, void* stream)
{
    if (!ctx) return fail(&g_err, MSAO_ERR_INVALID_ARG, "ctx is NULL");
    int R = 0;
    for (int i = 0; i < n && segs; ++i) R = std::max(R, segs[i].request + 1);
    msao_params p = msao_default_params();
    MSAO_TRY(validate_impl(segs, n, R, &p, &ctx->err));
    Plan pl;
    build_plan(ctx, segs, n, R, &p, nullptr, out_byte_off, pl, false, nullptr, false, 0, nullptr, true);
    MSAO_TRY(check_ws(ctx, pl, ws, ws_bytes));
    if (pl.ntok > 0 && (!kept_idx || !kept_count))
        return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "kept_idx and kept_count are required");
    MSAO_TRY(check_out_alignment(ctx, {{kept_idx, 4}, {kept_count, 4}}));
    MSAO_TRY(check_compact_out(ctx, pl, segs, n, out, out_byte_off, out_bytes));
    DeviceGuard guard(ctx->device);
    hipStream_t st = (hipStream_t)stream;
    MSAO_TRY(upload(ctx, pl, ws, st));
    GatherArgs ga;
    std::memset(&ga, 0, sizeof ga);
    ga.t = device_tables(pl, ws, n, R, &p);
    ga.kept_idx = kept_idx;
    ga.kept_count = kept_count;
    ga.out = (uint8_t*)out;
    ga.out_bytes = out_bytes;
    return launched(ctx, MSAO_KERNEL_GATHER, st, run_gather, &ga);
}

}  // extern "C"

namespace {

// The heads (Eq. 3) and MLP (Eq. 6) of a learned call.
msao_status check_learned(msao_ctx* ctx, const msao_segment* segs, int n, const msao_spatial_head* heads,
                          const msao_modal_mlp* mlp)
{
    char buf[160];
    for (int i = 0; heads && i < n; ++i) {
        const msao_spatial_head& h = heads[i];
        if (!h.weight) continue;
        auto bad = [&](msao_status st, const char* what) {
            std::snprintf(buf, sizeof buf, "head of segment %d: %s", i, what);
            return fail(&ctx->err, st, buf);
        };
        if (((uintptr_t)h.weight) % 16 != 0) return bad(MSAO_ERR_ALIGNMENT, "weight is not 16-byte aligned");
        if (!std::isfinite(h.bias)) return bad(MSAO_ERR_INVALID_ARG, "bias is not finite");
        if (h.pool < 1 || h.pool > kMaxPool || h.pool % 2 == 0) return bad(MSAO_ERR_INVALID_ARG, "pool must be odd, 1..15");
        const int P = segs[i].tokens_per_frame;
        if (P > kMaxHeadFrame) return bad(MSAO_ERR_UNSUPPORTED, "more than 16384 tokens per frame");
        if (h.grid_w < 0 || (h.grid_w > 0 && P % h.grid_w != 0))
            return bad(MSAO_ERR_INVALID_ARG, "grid_w must be 0 or divide tokens_per_frame");
    }
    if (mlp) {
        if (!mlp->w1 || !mlp->b1 || !mlp->w2) return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "MLP weights are NULL");
        if (mlp->hidden < 1 || mlp->hidden > kMaxMlpHidden)
            return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "MLP hidden out of range");
        if (mlp->prompt_dim < 0 || mlp->prompt_dim > 16384)
            return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "MLP prompt_dim out of range");
        if (mlp->prompt_dim > 0 && !mlp->prompt) return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "prompt is NULL");
        if (!std::isfinite(mlp->b2)) return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "b2 is not finite");
        MSAO_TRY(check_out_alignment(ctx, {{mlp->w1, 4}, {mlp->b1, 4}, {mlp->w2, 4}, {mlp->prompt, 4}}));
    }
    return MSAO_OK;
}

}  // namespace

extern "C" {

msao_status msao_mas_score_learned(msao_ctx* ctx, const msao_segment* segs, int n, int R, const msao_params* params,
                                   const msao_spatial_head* heads, const msao_modal_mlp* mlp, const float* alpha,
                                   const msao_token_out* tok, float* importance, const msao_frame_out* frm,
                                   const msao_req_out* req, float* alpha_out, float* desc, void* ws, size_t ws_bytes,
                                   void* stream)
{
    if (!ctx) return fail(&g_err, MSAO_ERR_INVALID_ARG, "ctx is NULL");
    MSAO_TRY(validate_impl(segs, n, R, params, &ctx->err));
    MSAO_TRY(check_learned(ctx, segs, n, heads, mlp));
    Plan pl;
    build_plan(ctx, segs, n, R, params, alpha, nullptr, pl, false, heads, true, mlp ? mlp->hidden : 0);
    MSAO_TRY(check_ws(ctx, pl, ws, ws_bytes));
    const bool want_frames = frm && (frm->dframe || frm->sim || frm->gamma) && pl.nframes > 0;
    if (want_frames && !(tok && tok->d))
        return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "per-frame outputs need tok->d");
    if (tok) MSAO_TRY(check_out_alignment(ctx, {{tok->z, 4}, {tok->l1, 4}, {tok->l2, 4}, {tok->info, 4}, {tok->d, 4}, {tok->res, 4}}));
    if (frm) MSAO_TRY(check_out_alignment(ctx, {{frm->dframe, 8}, {frm->sim, 4}, {frm->gamma, 4}}));
    if (req) MSAO_TRY(check_out_alignment(ctx, {{req->agg, 8}, {req->rho, 4}, {req->temporal, 4}, {req->beta, 4}, {req->mas, 4}}));
    MSAO_TRY(check_out_alignment(ctx, {{importance, 4}, {alpha_out, 4}, {desc, 4}}));
    DeviceGuard guard(ctx->device);
    hipStream_t st = (hipStream_t)stream;
    MSAO_TRY(upload(ctx, pl, ws, st));
    ScoreArgs sa;
    std::memset(&sa, 0, sizeof sa);
    sa.t = device_tables(pl, ws, n, R, params);
    sa.tok = token_out(tok);
    sa.mode = kModeScore;
    sa.xcd_order = xcd_order_for(ctx, false);
    sa.learned = 1;
    sa.importance = importance;
    MSAO_TRY(launched(ctx, MSAO_KERNEL_SCORE, st, run_score, &sa));
    float* mlp_u = mlp ? (float*)((uint8_t*)ws + pl.off_mlp_u) : nullptr;
    if (!pl.hb_seg.empty() || mlp) {
        HeadArgs ha;
        std::memset(&ha, 0, sizeof ha);
        ha.t = sa.t;
        ha.importance = importance;
        ha.max_p = pl.max_head_p;
        if (mlp) {
            ha.mlp = ModalMlp{mlp->w1, mlp->b1, mlp->w2, mlp->b2, mlp->hidden, mlp->prompt_dim, mlp->prompt};
            ha.u = mlp_u;
            const int64_t waves = (int64_t)mlp->hidden * ((R + kMlpGroup - 1) / kMlpGroup);
            ha.n_mlp_blocks = (int32_t)((waves + kHeadBlock / 64 - 1) / (kHeadBlock / 64));
        }
        MSAO_TRY(launched(ctx, MSAO_KERNEL_HEAD, st, run_head, &ha));
    }
    PostArgs pa;
    std::memset(&pa, 0, sizeof pa);
    pa.t = sa.t;
    if (req) pa.req = ReqOut{req->agg, req->rho, req->temporal, req->beta, req->mas, req->present};
    if (frm) pa.frm = FrameOut{frm->dframe, frm->sim, frm->gamma};
    pa.d = tok ? tok->d : nullptr;
    pa.learned = 1;
    if (mlp) {
        pa.use_mlp = 1;
        pa.mlp = ModalMlp{mlp->w1, mlp->b1, mlp->w2, mlp->b2, mlp->hidden, mlp->prompt_dim, mlp->prompt};
        pa.mlp_u = mlp_u;
    }
    pa.alpha_out = alpha_out;
    pa.desc_out = desc;
    pa.n_req_blocks = R;
    pa.n_frame_blocks = want_frames ? (int)pl.nframes : 0;
    return launched(ctx, MSAO_KERNEL_POST, st, run_post, &pa);
}

msao_status msao_stream_read(msao_ctx* ctx, const void* data, int64_t bytes, int chunk_kib, uint32_t* sink,
                             int64_t sink_words, void* stream)
{
    if (!ctx) return fail(&g_err, MSAO_ERR_INVALID_ARG, "ctx is NULL");
    if (!data || bytes <= 0) return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "data is NULL or bytes <= 0");
    if (chunk_kib != 8 && chunk_kib != 16 && chunk_kib != 32 && chunk_kib != 64)
        return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "chunk_kib must be 8, 16, 32 or 64");
    const int64_t chunk = (int64_t)chunk_kib * 1024, waves = (bytes + chunk - 1) / chunk;
    if (!sink || sink_words < waves) return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "sink is NULL or too small");
    if (!aligned(data, 16) || !aligned(sink, 4)) return fail(&ctx->err, MSAO_ERR_ALIGNMENT, "data or sink misaligned");
    if (waves > ((int64_t)1 << 31) * (kReadBlock / 64)) return fail(&ctx->err, MSAO_ERR_UNSUPPORTED, "buffer too large");
    DeviceGuard guard(ctx->device);
    ReadArgs a;
    a.data = (const uint8_t*)data;
    a.bytes = bytes;
    a.waves = waves;
    a.chunk_bytes = (int32_t)chunk;
    a.sink = sink;
    return launched(ctx, MSAO_KERNEL_READ, (hipStream_t)stream, run_read, &a);
}

msao_status msao_draft_entropy(msao_ctx* ctx, const void* logits, int64_t rows, int64_t vocab, int64_t row_stride,
                               int dtype, float theta, const msao_entropy_out* out, void* stream)
{
    if (!ctx) return fail(&g_err, MSAO_ERR_INVALID_ARG, "ctx is NULL");
    if (!out) return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "out is NULL");
    if (dtype != MSAO_F32 && dtype != MSAO_BF16) return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "unknown dtype");
    const int64_t es = elt_size(dtype);
    if (rows < 0 || rows > INT32_MAX) return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "rows out of range");
    if (vocab < 2 || vocab * es >= ((int64_t)1 << 31) - ((int64_t)1 << 20))
        return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "vocab out of range");
    if (row_stride < vocab) return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "row_stride < vocab");
    if (std::isnan(theta) || std::isinf(theta)) return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "theta is not finite");
    if (rows > 0 && !logits) return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "logits is NULL");
    if (((uintptr_t)logits) % 16 != 0) return fail(&ctx->err, MSAO_ERR_ALIGNMENT, "logits are not 16-byte aligned");
    if ((row_stride * es) % 16 != 0) return fail(&ctx->err, MSAO_ERR_ALIGNMENT, "row pitch is not a multiple of 16 bytes");
    MSAO_TRY(check_out_alignment(ctx, {{out->entropy, 4}, {out->entropy_norm, 4}, {out->draft_token, 4}}));
    if (rows == 0) return MSAO_OK;
    DeviceGuard guard(ctx->device);
    EntArgs a;
    std::memset(&a, 0, sizeof a);
    a.logits = (const uint8_t*)logits;
    a.row_bytes = row_stride * es;
    a.rows = (int32_t)rows;
    a.vocab = (int32_t)vocab;
    a.dtype = dtype;
    a.theta = theta;
    a.inv_log_vocab = (float)(1.0 / std::log((double)vocab));
    a.entropy = out->entropy;
    a.entropy_norm = out->entropy_norm;
    a.draft_token = out->draft_token;
    a.speculate = out->speculate;
    return launched(ctx, MSAO_KERNEL_ENTROPY, (hipStream_t)stream, run_entropy, &a);
}

}  // extern "C"

namespace {

// Output checks of a full run (scoring, MAS, selection, optional compaction).
msao_status check_run_outputs(msao_ctx* ctx, const Plan& pl, const std::vector<msao_segment>& segs,
                              const msao_token_out* tok, const msao_frame_out* frm, const msao_req_out* req,
                              const msao_select_out* sel, void* out, const int64_t* out_byte_off, int64_t out_bytes)
{
    if (pl.ntok > 0 && !(tok && tok->z)) return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "a full run needs tok->z");
    if (pl.any_temporal && !(tok && tok->d))
        return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "a full run needs tok->d for temporal segments");
    if (!sel || !sel->kept_idx || !sel->kept_count)
        return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "selection needs kept_idx and kept_count");
    if (tok) MSAO_TRY(check_out_alignment(ctx, {{tok->z, 4}, {tok->l1, 4}, {tok->l2, 4}, {tok->info, 4}, {tok->d, 4}, {tok->res, 4}}));
    if (frm) MSAO_TRY(check_out_alignment(ctx, {{frm->dframe, 8}, {frm->sim, 4}, {frm->gamma, 4}}));
    if (req) MSAO_TRY(check_out_alignment(ctx, {{req->agg, 8}, {req->rho, 4}, {req->temporal, 4}, {req->beta, 4}, {req->mas, 4}}));
    MSAO_TRY(check_out_alignment(ctx, {{sel->kept_idx, 4}, {sel->kept_count, 4}}));
    if (out) MSAO_TRY(check_compact_out(ctx, pl, segs.data(), (int)segs.size(), out, out_byte_off, out_bytes));
    return MSAO_OK;
}

// The three launches of a full run, on tables already in the workspace. A
// run with SimHash (pl.simhash_d) puts two between scoring and the post
// launch: the signatures (into sig), then d, the clips' informativeness and
// Dsum per (request, modality) from them (t.hdsum), which replace bit
// sampling's before MAS, the per-frame terms and selection read them.
msao_status enqueue_run(msao_ctx* ctx, const Plan& pl, const Tables& t, const msao_token_out* tok,
                        const msao_frame_out* frm, const msao_req_out* req, const msao_select_out* sel, void* out,
                        int64_t out_bytes, hipStream_t st, uint64_t* sig = nullptr)
{
    ScoreArgs sa;
    std::memset(&sa, 0, sizeof sa);
    sa.t = t;
    sa.tok = token_out(tok);
    if (pl.clip_fused) sa.tok.sig = sig;
    sa.out = (uint8_t*)out;
    sa.mode = kModeScore;
    sa.xcd_order = xcd_order_for(ctx, out && pl.any_copy);
    MSAO_TRY(launched(ctx, MSAO_KERNEL_SCORE, st, run_score, &sa));
    if (pl.clip_fused) {
        // the clips: statistics, signatures, d and partials in one pass
        ClipArgs ca;
        std::memset(&ca, 0, sizeof ca);
        ca.t = t;
        ca.tok = token_out(tok);
        ca.tok.sig = sig;
        ca.clip_dtype = pl.clip_dtype;
        ca.clip_bits = pl.clip_bits;
        MSAO_TRY(launched(ctx, MSAO_KERNEL_CLIP, st, run_clip, &ca));
    } else if (sig && t.n_hi > 0) {
        // signatures of every token (zeros outside temporal segments)
        HashArgs ha;
        std::memset(&ha, 0, sizeof ha);
        ha.t = t;
        ha.sig = sig;
        ha.d = tok->d;
        ha.z = tok->z;
        ha.info = tok->info;
        ha.hdsum = const_cast<uint64_t*>(t.hdsum);
        MSAO_TRY(launched(ctx, MSAO_KERNEL_SIMHASH, st, run_simhash, &ha));
        if (pl.simhash_d) {
            ha.n_frame_blocks = (int)pl.nframes;
            ha.n_req_blocks = t.R;
            MSAO_TRY(launched(ctx, MSAO_KERNEL_HASH_POST, st, run_hash_post, &ha));
        }
    }
    PostArgs pa;
    std::memset(&pa, 0, sizeof pa);
    pa.t = t;
    if (req) pa.req = ReqOut{req->agg, req->rho, req->temporal, req->beta, req->mas, req->present};
    if (frm) pa.frm = FrameOut{frm->dframe, frm->sim, frm->gamma};
    pa.sel = SelOut{sel->keep, sel->kept_idx, sel->kept_count};
    pa.z = tok ? tok->z : nullptr;
    pa.d = tok ? tok->d : nullptr;
    pa.mas_in = nullptr;
    const bool want_req = req && (req->agg || req->rho || req->temporal || req->beta || req->mas || req->present);
    const bool want_frames = frm && (frm->dframe || frm->sim || frm->gamma) && pl.nframes > 0;
    pa.n_req_blocks = want_req ? t.R : 0;
    pa.n_frame_blocks = want_frames ? (int)pl.nframes : 0;
    pa.n_sel_blocks = (int)pl.sel_unit.size();
    pa.keys_cap = std::min(pl.max_n, kMaxLdsKeys);
    pa.big_block = pl.max_n >= pl.big_seg ? 1 : 0;
    MSAO_TRY(launched(ctx, MSAO_KERNEL_POST, st, run_post, &pa));
    if (!out || t.n_gwi == 0) return MSAO_OK;
    GatherArgs ga;
    std::memset(&ga, 0, sizeof ga);
    ga.t = t;
    ga.kept_idx = sel->kept_idx;
    ga.kept_count = sel->kept_count;
    ga.out = (uint8_t*)out;
    ga.out_bytes = out_bytes;
    return launched(ctx, MSAO_KERNEL_GATHER, st, run_gather, &ga);
}

}  // namespace

struct msao_plan {
    msao_ctx* ctx = nullptr;
    Plan pl;
    Tables t{};
    std::vector<msao_segment> segs;
    std::vector<int64_t> out_off;
    msao_params params{};
};

extern "C" {

msao_status msao_run(msao_ctx* ctx, const msao_segment* segs, int n, int R, const msao_params* params,
                     const float* alpha, const msao_token_out* tok, const msao_frame_out* frm,
                     const msao_req_out* req, const msao_select_out* sel, void* out, const int64_t* out_byte_off,
                     int64_t out_bytes, void* ws, size_t ws_bytes, void* stream)
{
    if (!ctx) return fail(&g_err, MSAO_ERR_INVALID_ARG, "ctx is NULL");
    MSAO_TRY(validate_impl(segs, n, R, params, &ctx->err));
    Plan pl;
    build_plan(ctx, segs, n, R, params, alpha, out_byte_off, pl, out != nullptr);
    MSAO_TRY(check_ws(ctx, pl, ws, ws_bytes));
    const std::vector<msao_segment> sv(segs, segs + n);
    MSAO_TRY(check_run_outputs(ctx, pl, sv, tok, frm, req, sel, out, out_byte_off, out_bytes));
    DeviceGuard guard(ctx->device);
    hipStream_t st = (hipStream_t)stream;
    MSAO_TRY(upload(ctx, pl, ws, st));
    return enqueue_run(ctx, pl, device_tables(pl, ws, n, R, params), tok, frm, req, sel, out, out_bytes, st);
}

static_assert(kNoAllocScratchBytes == MSAO_NOALLOC_SCRATCH_BYTES && kNoAllocTableBytes == MSAO_NOALLOC_TABLE_BYTES,
              "the header states the scratch limits");

msao_status msao_run_noalloc(msao_ctx* ctx, const msao_segment* segs, int n, int R, const msao_params* params,
                             const float* alpha, const msao_token_out* tok, const msao_frame_out* frm,
                             const msao_req_out* req, const msao_select_out* sel, void* out,
                             const int64_t* out_byte_off, int64_t out_bytes, void* stream)
{
    if (!ctx) return fail(&g_err, MSAO_ERR_INVALID_ARG, "ctx is NULL");
    MSAO_TRY(validate_impl(segs, n, R, params, &ctx->err));
    Plan pl;
    build_plan(ctx, segs, n, R, params, alpha, out_byte_off, pl, out != nullptr);
    char buf[200];
    if (pl.table_bytes > kNoAllocTableBytes || pl.total_bytes > kNoAllocScratchBytes) {
        std::snprintf(buf, sizeof buf,
                      "msao_run_noalloc: the call needs %zu bytes of tables and %zu of scratch; the limits are "
                      "%zu and %zu (use msao_run with a workspace)",
                      pl.table_bytes, pl.total_bytes, kNoAllocTableBytes, kNoAllocScratchBytes);
        return fail(&ctx->err, MSAO_ERR_UNSUPPORTED, buf);
    }
    const std::vector<msao_segment> sv(segs, segs + n);
    MSAO_TRY(check_run_outputs(ctx, pl, sv, tok, frm, req, sel, out, out_byte_off, out_bytes));
    // the device address of this GPU's scratch array, looked up by msao_create
    void* ws = scratch_ptr(ctx->device);
    if (!ws) return fail(&ctx->err, MSAO_ERR_HIP, "the scratch array of this device was not set up");
    DeviceGuard guard(ctx->device);
    hipStream_t st = (hipStream_t)stream;
    MSAO_TRY(upload(ctx, pl, ws, st, false));
    return enqueue_run(ctx, pl, device_tables(pl, ws, n, R, params), tok, frm, req, sel, out, out_bytes, st);
}

msao_status msao_run_simhash(msao_ctx* ctx, const msao_segment* segs, int n, int R, const msao_params* params,
                             const msao_simhash* hashes, const float* alpha, const msao_token_out* tok,
                             uint64_t* sig, const msao_frame_out* frm, const msao_req_out* req,
                             const msao_select_out* sel, void* out, const int64_t* out_byte_off, int64_t out_bytes,
                             void* ws, size_t ws_bytes, void* stream)
{
    if (!ctx) return fail(&g_err, MSAO_ERR_INVALID_ARG, "ctx is NULL");
    MSAO_TRY(validate_impl(segs, n, R, params, &ctx->err));
    MSAO_TRY(check_hashes(ctx, segs, n, hashes));
    Plan pl;
    build_plan(ctx, segs, n, R, params, alpha, out_byte_off, pl, out != nullptr, nullptr, false, 0, hashes, false,
               true);
    MSAO_TRY(check_ws(ctx, pl, ws, ws_bytes));
    const std::vector<msao_segment> sv(segs, segs + n);
    MSAO_TRY(check_run_outputs(ctx, pl, sv, tok, frm, req, sel, out, out_byte_off, out_bytes));
    if (pl.ntok > 0 && !sig) return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "sig is required");
    MSAO_TRY(check_out_alignment(ctx, {{sig, 8}}));
    DeviceGuard guard(ctx->device);
    hipStream_t st = (hipStream_t)stream;
    MSAO_TRY(upload(ctx, pl, ws, st));
    return enqueue_run(ctx, pl, device_tables(pl, ws, n, R, params), tok, frm, req, sel, out, out_bytes, st, sig);
}

msao_status msao_run_learned(msao_ctx* ctx, const msao_segment* segs, int n, int R, const msao_params* params,
                             const msao_spatial_head* heads, const msao_modal_mlp* mlp, const float* alpha,
                             const msao_token_out* tok, float* importance, const msao_frame_out* frm,
                             const msao_req_out* req, float* alpha_out, float* desc, const msao_select_out* sel,
                             void* out, const int64_t* out_byte_off, int64_t out_bytes, void* ws, size_t ws_bytes,
                             void* stream)
{
    if (!ctx) return fail(&g_err, MSAO_ERR_INVALID_ARG, "ctx is NULL");
    MSAO_TRY(validate_impl(segs, n, R, params, &ctx->err));
    MSAO_TRY(check_learned(ctx, segs, n, heads, mlp));
    Plan pl;
    build_plan(ctx, segs, n, R, params, alpha, out_byte_off, pl, out != nullptr, heads, true, mlp ? mlp->hidden : 0,
               nullptr, false, false, true);
    MSAO_TRY(check_ws(ctx, pl, ws, ws_bytes));
    const std::vector<msao_segment> sv(segs, segs + n);
    MSAO_TRY(check_run_outputs(ctx, pl, sv, tok, frm, req, sel, out, out_byte_off, out_bytes));
    MSAO_TRY(check_out_alignment(ctx, {{importance, 4}, {alpha_out, 4}, {desc, 4}}));
    DeviceGuard guard(ctx->device);
    hipStream_t st = (hipStream_t)stream;
    MSAO_TRY(upload(ctx, pl, ws, st));
    const Tables t = device_tables(pl, ws, n, R, params);
    // statistics, head projections (and the rows of segments kept whole)
    ScoreArgs sa;
    std::memset(&sa, 0, sizeof sa);
    sa.t = t;
    sa.tok = token_out(tok);
    sa.out = (uint8_t*)out;
    sa.mode = kModeScore;
    sa.xcd_order = xcd_order_for(ctx, out && pl.any_copy);
    sa.learned = 1;
    sa.importance = importance;
    MSAO_TRY(launched(ctx, MSAO_KERNEL_SCORE, st, run_score, &sa));
    // Eq. 3 importance of the head segments, kept in the workspace for the selection
    float* mlp_u = mlp ? (float*)((uint8_t*)ws + pl.off_mlp_u) : nullptr;
    if (!pl.hb_seg.empty() || mlp) {
        HeadArgs ha;
        std::memset(&ha, 0, sizeof ha);
        ha.t = t;
        ha.importance = importance;
        ha.max_p = pl.max_head_p;
        if (mlp) {
            ha.mlp = ModalMlp{mlp->w1, mlp->b1, mlp->w2, mlp->b2, mlp->hidden, mlp->prompt_dim, mlp->prompt};
            ha.u = mlp_u;
            const int64_t waves = (int64_t)mlp->hidden * ((R + kMlpGroup - 1) / kMlpGroup);
            ha.n_mlp_blocks = (int32_t)((waves + kHeadBlock / 64 - 1) / (kHeadBlock / 64));
        }
        MSAO_TRY(launched(ctx, MSAO_KERNEL_HEAD, st, run_head, &ha));
    }
    // Eq. 4 on the heads, the descriptor, Eq. 6, softmax and Eq. 7; the MAS
    // also into the workspace for MAS-guided keep counts
    float* mas_ws = (float*)((uint8_t*)ws + pl.off_mas);
    PostArgs pa;
    std::memset(&pa, 0, sizeof pa);
    pa.t = t;
    if (req) pa.req = ReqOut{req->agg, req->rho, req->temporal, req->beta, req->mas, req->present};
    if (frm) pa.frm = FrameOut{frm->dframe, frm->sim, frm->gamma};
    pa.d = tok ? tok->d : nullptr;
    pa.learned = 1;
    if (mlp) {
        pa.use_mlp = 1;
        pa.mlp = ModalMlp{mlp->w1, mlp->b1, mlp->w2, mlp->b2, mlp->hidden, mlp->prompt_dim, mlp->prompt};
        pa.mlp_u = mlp_u;
    }
    pa.alpha_out = alpha_out;
    pa.desc_out = desc;
    pa.mas_ws = mas_ws;
    const bool want_frames = frm && (frm->dframe || frm->sim || frm->gamma) && pl.nframes > 0;
    pa.n_req_blocks = R;
    pa.n_frame_blocks = want_frames ? (int)pl.nframes : 0;
    MSAO_TRY(launched(ctx, MSAO_KERNEL_POST, st, run_post, &pa));
    // Sec. 4.1.1 pruning: head segments by importance, the others by the redundancy key
    PostArgs ps;
    std::memset(&ps, 0, sizeof ps);
    ps.t = t;
    ps.sel = SelOut{sel->keep, sel->kept_idx, sel->kept_count};
    ps.z = tok ? tok->z : nullptr;
    ps.d = tok ? tok->d : nullptr;
    ps.mas_in = mas_ws;
    ps.n_sel_blocks = (int)pl.sel_unit.size();
    ps.keys_cap = std::min(pl.max_n, kMaxLdsKeys);
    ps.big_block = pl.max_n >= pl.big_seg ? 1 : 0;
    MSAO_TRY(launched(ctx, MSAO_KERNEL_POST, st, run_post, &ps));
    if (!out || t.n_gwi == 0) return MSAO_OK;
    GatherArgs ga;
    std::memset(&ga, 0, sizeof ga);
    ga.t = t;
    ga.kept_idx = sel->kept_idx;
    ga.kept_count = sel->kept_count;
    ga.out = (uint8_t*)out;
    ga.out_bytes = out_bytes;
    return launched(ctx, MSAO_KERNEL_GATHER, st, run_gather, &ga);
}

msao_status msao_plan_create(msao_ctx* ctx, const msao_segment* segs, int n, int R, const msao_params* params,
                             const float* alpha, const int64_t* out_byte_off, void* ws, size_t ws_bytes,
                             void* stream, msao_plan** plan)
{
    if (!ctx) return fail(&g_err, MSAO_ERR_INVALID_ARG, "ctx is NULL");
    if (!plan) return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "plan pointer is NULL");
    *plan = nullptr;
    MSAO_TRY(validate_impl(segs, n, R, params, &ctx->err));
    msao_plan* p = new msao_plan();
    p->ctx = ctx;
    p->segs.assign(segs, segs + n);
    if (out_byte_off) p->out_off.assign(out_byte_off, out_byte_off + n);
    p->params = *params;
    build_plan(ctx, segs, n, R, params, alpha, out_byte_off, p->pl, out_byte_off != nullptr);
    msao_status st = check_ws(ctx, p->pl, ws, ws_bytes);
    if (st == MSAO_OK) {
        DeviceGuard guard(ctx->device);
        st = upload(ctx, p->pl, ws, (hipStream_t)stream);
    }
    if (st != MSAO_OK) {
        delete p;
        return st;
    }
    p->t = device_tables(p->pl, ws, n, R, params);
    *plan = p;
    return MSAO_OK;
}

msao_status msao_plan_run(msao_plan* plan, const msao_token_out* tok, const msao_frame_out* frm,
                          const msao_req_out* req, const msao_select_out* sel, void* out, int64_t out_bytes,
                          void* stream)
{
    if (!plan) return fail(&g_err, MSAO_ERR_INVALID_ARG, "plan is NULL");
    msao_ctx* ctx = plan->ctx;
    if (out && plan->out_off.size() != plan->segs.size())
        return fail(&ctx->err, MSAO_ERR_INVALID_ARG, "the plan was created without out_byte_off");
    MSAO_TRY(check_run_outputs(ctx, plan->pl, plan->segs, tok, frm, req, sel, out, plan->out_off.data(), out_bytes));
    DeviceGuard guard(ctx->device);
    return enqueue_run(ctx, plan->pl, plan->t, tok, frm, req, sel, out, out_bytes, (hipStream_t)stream);
}

void msao_plan_destroy(msao_plan* plan) { delete plan; }

}  // extern "C"
