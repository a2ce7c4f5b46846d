// msao_kernels.hip -- gfx950 (CDNA4) kernels of MSAO's fine-grained sparsity
// analysis (Sec. 4.1) and of the MAS-guided token selection it drives.
//
// The path is HBM-bandwidth bound: every input byte is read once with 128-bit
// loads, no step is a dense contraction (no MFMA). Three launch slots:
//   scoring  k_pair for bf16 clips with rows of 512-2,048 bytes (a wavefront
//            streams two neighbouring patch positions through a range of
//            frames, a ring of frames in registers), k_score for the rest
//            (one wavefront per work item: a run of rows, or one patch's run
//            of frames). Per token: active count, L1/L2 and, for video, the
//            temporal terms of Eq. 5 against the previous frame, whose values
//            and activity bits stay in registers (no extra HBM traffic). Per
//            work item they write integer partials (sparse-token count, sum
//            of d), so no atomics and no zeroing are needed and results are
//            bit-stable. (A call with learned heads launches k_head between
//            the scoring pass and k_post: the heads' pooling and MLP.)
//   k_post   block roles: one block per request (integer aggregation, modal
//            softmax, Eq. 4 ratio, Eq. 7 MAS), one per video frame (Eq. 5
//            per frame), one or more per selection (top-k by LDS radix
//            select over exact integer keys, ties by index, block-scan
//            compaction).
//   k_gather one wavefront per kept row: packed bitwise copy.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "msao_device.h"
#include "msao_internal.h"

namespace msao {
namespace {

constexpr int kWave = 64;

template <int CTRL>
__device__ __forceinline__ float dpp_f(float v)
{
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_rows(float v)
{
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, ROW_MASK, 0xF, false));
}

// Sum over the 64 lanes, returned as a wave-uniform value. Fixed order, so it
// is bit-reproducible: quad_perm [1,0,3,2], quad_perm [2,3,0,1],
// row_half_mirror and row_mirror give every 16-lane row its sum; row_bcast:15
// and row_bcast:31 then fold the rows into lane 63.
__device__ __forceinline__ float wave_sum(float v)
{
    v += dpp_f<0xB1>(v);
    v += dpp_f<0x4E>(v);
    v += dpp_f<0x141>(v);
    v += dpp_f<0x140>(v);
    v += dpp_rows<0x142, 0xA>(v);
    v += dpp_rows<0x143, 0xC>(v);
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

typedef unsigned int vec4 __attribute__((ext_vector_type(4)));
typedef __amdgpu_buffer_rsrc_t rsrc_t;

// Raw buffer resources (GFX9 word 3): a load whose offset lies past
// num_records returns 0 and a store there is dropped, so ragged row tails
// and absent rows need no lane predicates.
constexpr int kRsrcWord3 = 0x00020000;
#ifndef MSAO_LOAD_AUX
#define MSAO_LOAD_AUX 2  // nontemporal: every input row is read once
#endif
#ifndef MSAO_STORE_AUX
#define MSAO_STORE_AUX 2  // nontemporal: compacted rows are written once and not re-read here
#endif
#ifndef MSAO_GATHER_LOAD_AUX
#define MSAO_GATHER_LOAD_AUX 0  // kept rows may still be cached from the scoring pass
#endif

__device__ __forceinline__ rsrc_t make_rsrc(const void* base, int bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, bytes, kRsrcWord3);
}

__device__ __forceinline__ vec4 bload(rsrc_t r, int off)
{
    return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, MSAO_LOAD_AUX);
}

__device__ __forceinline__ vec4 bload_gather(rsrc_t r, int off)
{
    return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, MSAO_GATHER_LOAD_AUX);
}

__device__ __forceinline__ void bstore(vec4 v, rsrc_t r, int off)
{
    __builtin_amdgcn_raw_buffer_store_b128(v, r, off, 0, MSAO_STORE_AUX);
}

__device__ __forceinline__ uint32_t lanes_below(uint64_t m)
{
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int o)
{
    const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)v, o);
    const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(v >> 32), o);
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += shfl_xor_u64(v, o);
    return v;
}

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const uint64_t w = shfl_xor_u64(v, o);
        v = w < v ? w : v;
    }
    return v;
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const uint64_t w = shfl_xor_u64(v, o);
        v = w > v ? w : v;
    }
    return v;
}

// Widening of one 16-byte chunk to floats (exact).
template <int DT> struct Lane;
template <> struct Lane<kBF16> {
    static constexpr int EPC = 8;
    __device__ static __forceinline__ void widen(const vec4& v, float* x)
    {
        x[0] = __uint_as_float(v.x << 16); x[1] = __uint_as_float(v.x & 0xFFFF0000u);
        x[2] = __uint_as_float(v.y << 16); x[3] = __uint_as_float(v.y & 0xFFFF0000u);
        x[4] = __uint_as_float(v.z << 16); x[5] = __uint_as_float(v.z & 0xFFFF0000u);
        x[6] = __uint_as_float(v.w << 16); x[7] = __uint_as_float(v.w & 0xFFFF0000u);
    }
};
template <> struct Lane<kF32> {
    static constexpr int EPC = 4;
    __device__ static __forceinline__ void widen(const vec4& v, float* x)
    {
        x[0] = __uint_as_float(v.x); x[1] = __uint_as_float(v.y);
        x[2] = __uint_as_float(v.z); x[3] = __uint_as_float(v.w);
    }
};

// Ballot of (low 16 bits of ax) > lo: one 16-bit compare, no masking step.
__device__ __forceinline__ uint64_t ballot_lo16_gt(uint32_t ax, uint32_t lo)
{
    uint64_t m;
    asm("v_cmp_gt_u16_e64 %0, %1, %2" : "=s"(m) : "v"(ax), "s"(lo));
    return m;
}

// Statistics of one 16-byte chunk: active count (ballot + scalar popcount),
// L1 and L2 partial sums of this lane.
template <int DT>
__device__ __forceinline__ void chunk_stats(const vec4& v, float tau, const Thr& th, uint32_t& act, float& l1,
                                            float& l2)
{
    if constexpr (DT == kBF16) {
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            const uint32_t x = v[w];
            const uint32_t ax = x & 0x7FFF7FFFu;
            act += (uint32_t)__popcll(__ballot(ax > th.hi));
            act += (uint32_t)__popcll(ballot_lo16_gt(ax, th.lo));
            l1 = dot2(ax, kBf16OnePair, l1);
            l2 = dot2(x, x, l2);
        }
    } else {
        float x[4];
        Lane<kF32>::widen(v, x);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            act += (uint32_t)__popcll(__ballot(active(x[e], tau)));
            l1 += fabsf(x[e]);
            l2 = fmaf(x[e], x[e], l2);
        }
    }
}

// The same plus the temporal term against the previous frame: prev holds the
// previous frame's channel values of this lane, pmask its activity ballots
// (one per channel slot); both are updated to the current frame.
template <int DT>
__device__ __forceinline__ void chunk_chain(const vec4& v, float tau, const Thr& th, float* prev, uint64_t* pmask,
                                            uint32_t& act, uint32_t& d, float& l1, float& l2, float& res)
{
    if constexpr (DT == kBF16) {
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            const uint32_t x = v[w];
            const uint32_t ax = x & 0x7FFF7FFFu;
            const uint64_t mlo = ballot_lo16_gt(ax, th.lo);
            const uint64_t mhi = __ballot(ax > th.hi);
            act += (uint32_t)(__popcll(mlo) + __popcll(mhi));
            d += (uint32_t)(__popcll(mlo ^ pmask[2 * w]) + __popcll(mhi ^ pmask[2 * w + 1]));
            pmask[2 * w] = mlo;
            pmask[2 * w + 1] = mhi;
            l1 = dot2(ax, kBf16OnePair, l1);
            l2 = dot2(x, x, l2);
            const float flo = __uint_as_float(x << 16), fhi = __uint_as_float(x & 0xFFFF0000u);
            const float dlo = flo - prev[2 * w], dhi = fhi - prev[2 * w + 1];
            res = fmaf(dlo, dlo, res);
            res = fmaf(dhi, dhi, res);
            prev[2 * w] = flo;
            prev[2 * w + 1] = fhi;
        }
    } else {
        float x[4];
        Lane<kF32>::widen(v, x);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const uint64_t m = __ballot(active(x[e], tau));
            act += (uint32_t)__popcll(m);
            d += (uint32_t)__popcll(m ^ pmask[e]);
            pmask[e] = m;
            l1 += fabsf(x[e]);
            l2 = fmaf(x[e], x[e], l2);
            const float df = x[e] - prev[e];
            res = fmaf(df, df, res);
            prev[e] = x[e];
        }
    }
}

// ---------------------------------------------------------------- k_score

struct TokStat {
    uint32_t act;   // active channels
    uint32_t d;     // Hamming distance to the previous frame's activity bits
    float l1, l2, res;
};

// Statistics of up to 64 tokens of one wavefront: lane j holds the j-th token
// of the current run, so that each output array is written with one store
// instruction per run instead of one per token.
struct TokBuf {
    uint32_t act, d;
    float l1, l2, res;
    float y;        // learned calls: the head's projection w . x
};

__device__ __forceinline__ void tokbuf_put(TokBuf& b, int slot, int lane, const TokStat& s, float y = 0.0f)
{
    if (lane == slot) {
        b.act = s.act;
        b.d = s.d;
        b.l1 = s.l1;
        b.l2 = s.l2;
        b.res = s.res;
        b.y = y;
    }
}

// Per-lane state of a learned call's work item: sums of the item's tokens for
// the modality descriptor of Eq. 6 (wave-uniform values).
struct Lrn {
    uint32_t asum;
    float l1, l2;
};

__device__ __forceinline__ void lrn_add(Lrn& l, const TokStat& s)
{
    l.asum += s.act;
    l.l1 += s.l1;
    l.l2 += s.l2;
}

// Partial dot product of a 16-byte chunk of a row with the same chunk of the
// head's weights (Eq. 3's 1x1 convolution), products exact in fp32 for bf16.
template <int DT>
__device__ __forceinline__ float dot_chunk(const vec4& x, const vec4& w, float acc)
{
    if constexpr (DT == kBF16) {
#pragma unroll
        for (int k = 0; k < 4; ++k) acc = dot2(x[k], w[k], acc);
    } else {
#pragma unroll
        for (int k = 0; k < 4; ++k) acc = fmaf(__uint_as_float(x[k]), __uint_as_float(w[k]), acc);
    }
    return acc;
}

// The head's weights as NU 1-KiB units of this lane (zero without a head;
// the resource cuts the ragged last unit).
template <int NU>
__device__ __forceinline__ void load_head(vec4 (&wv)[NU], const DevSeg& sg, int voff)
{
    const rsrc_t rw = make_rsrc(sg.head_w, sg.head_w ? sg.nchunk * 16 : 0);
#pragma unroll
    for (int u = 0; u < NU; ++u) wv[u] = bload_gather(rw, voff + u * 1024);
}

// Writes tokens first_row + j * row_step (j < count) of the segment from
// lanes j: z = C - active count, L1, L2, info = 1 - (lambda_s z + lambda_t e)/C
// with e = C - d for temporal tokens, and d, res (zero outside temporal segments).
// Learned calls also write the projection of tokens of segments with a head,
// and the density importance a / C of the other tokens.
template <bool LR>
__device__ __forceinline__ void tokbuf_flush(const ScoreArgs& a, const DevSeg& sg, const TokBuf& b, int first_row,
                                             int row_step, int count, int lane, bool temporal, int mode)
{
    if (lane >= count) return;
    const TokenOut& o = a.tok;
    const int g = sg.tok_off + first_row + lane * row_step;
    if constexpr (LR) {
        if (sg.head_w) a.t.proj[g] = b.y;
        else if (a.importance) a.importance[g] = (float)b.act / (float)sg.C;
    }
    const uint32_t z = (uint32_t)sg.C - b.act;
    if (mode == kModeScore) {
        if (o.z) o.z[g] = z;
        if (o.l1) o.l1[g] = b.l1;
        if (o.l2) o.l2[g] = b.l2;
        if (o.info) {
            float red = sg.lam_s * (float)z;
            if (temporal) red += sg.lam_t * (float)((uint32_t)sg.C - b.d);
            o.info[g] = 1.0f - red * __builtin_amdgcn_rcpf((float)sg.C);
        }
    }
    if (o.d) o.d[g] = temporal ? b.d : 0u;
    if (o.res) o.res[g] = temporal ? b.res : 0.0f;
    // a run with SimHash (never learned): this pass scores no clip; the
    // learned instance leaves the store out, which keeps it from spilling
    if constexpr (!LR) {
        if (o.sig) o.sig[g] = 0ull;
    }
}

// A segment that keeps every row is compacted by the scoring pass itself: the
// row just read is written to its packed slot (row i of the segment goes to
// out + out_off + i * row bytes), so the gather never re-reads it.
template <int NU>
__device__ __forceinline__ void copy_row_out(const ScoreArgs& a, const DevSeg& sg, int row, const vec4 (&v)[NU],
                                             int voff)
{
    const int rb = sg.nchunk * 16;
    const rsrc_t rd = make_rsrc(a.out + sg.out_off + (int64_t)row * rb, rb);
#pragma unroll
    for (int u = 0; u < NU; ++u) bstore(v[u], rd, voff + u * 1024);
}

// Statistics of one row held as NU 1-KiB units (64 lanes x 16 B each).
template <int DT, int NU>
__device__ __forceinline__ TokStat row_stats(const vec4 (&v)[NU], float tau, const Thr& th)
{
    TokStat s{0u, 0u, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int u = 0; u < NU; ++u) chunk_stats<DT>(v[u], tau, th, s.act, s.l1, s.l2);
    s.l1 = wave_sum(s.l1);
    s.l2 = wave_sum(s.l2);
    return s;
}

// RPI rows starting at r into v; rows at or past r1 read as zero (empty resource).
template <int NU, int RPI>
__device__ __forceinline__ void load_rows(vec4 (&v)[RPI][NU], const DevSeg& sg, int r, int r1, int voff)
{
    const int rb = sg.nchunk * 16;
#pragma unroll
    for (int i = 0; i < RPI; ++i) {
        const bool ok = r + i < r1;
        const rsrc_t rs = make_rsrc(sg.data + (int64_t)(ok ? r + i : 0) * sg.stride_bytes, ok ? rb : 0);
#pragma unroll
        for (int u = 0; u < NU; ++u) v[i][u] = bload(rs, voff + u * 1024);
    }
}

// Rows [r, r + RPI) clipped to r1 of the item that starts at row r0. Row
// statistics go to slot (row - r0) & 63 of the token buffer, which is written
// out when it holds 64 rows or the item ends (RPI divides 64, so a batch
// never straddles a flush).
template <int DT, int NU, int RPI, bool LR>
__device__ __forceinline__ void rows_batch(const ScoreArgs& a, const DevSeg& sg, const vec4 (&v)[RPI][NU],
                                           int r0, int r, int r1, int lane, uint32_t& nsp, TokBuf& tb,
                                           const vec4 (&wv)[NU], Lrn& lr)
{
    static_assert(64 % RPI == 0, "a row batch must divide the token buffer");
    const bool copy = a.out && sg.copy_in_score;
#pragma unroll
    for (int i = 0; i < RPI; ++i) {
        if (r + i >= r1) break;
        if (copy) copy_row_out<NU>(a, sg, r + i, v[i], lane * 16);
        const TokStat s = row_stats<DT, NU>(v[i], a.t.tau, bf16_thresholds(a.t.tau));
        float y = 0.0f;
        if constexpr (LR) {
            if (sg.head_w) {
                float acc = 0.0f;
#pragma unroll
                for (int u = 0; u < NU; ++u) {
                    // rows over 3 KiB re-read the weights (L1 hits) instead of holding
                    // them: the registers go to the double-buffered rows
                    const vec4 w = NU > 3 ? bload_gather(make_rsrc(sg.head_w, sg.nchunk * 16), lane * 16 + u * 1024)
                                          : wv[u];
                    acc = dot_chunk<DT>(v[i][u], w, acc);
                }
                y = wave_sum(acc);
            }
            lrn_add(lr, s);
        }
        tokbuf_put(tb, (r + i - r0) & 63, lane, s, y);
        nsp += s.act < (uint32_t)sg.A_s;
    }
    const int done = min(r + RPI, r1);
    if (((done - r0) & 63) == 0 || done == r1) {
        const int first = (done - 1) - ((done - 1 - r0) & 63);
        tokbuf_flush<LR>(a, sg, tb, first, 1, done - first, lane, false, kModeScore);
    }
}

#ifndef MSAO_ROW_BATCH_UNITS
#define MSAO_ROW_BATCH_UNITS 8  // 1-KiB units per row batch (double-buffered)
#endif

// Rows [r0, r1) of a non-temporal segment whose rows span NU units. For
// rows up to 4 KiB, batches of RPI rows (about 4 KiB) are double-buffered:
// the next batch is in flight while the current one is reduced. Wider rows
// already keep NU KiB in flight per wavefront and are single-buffered, which
// holds the data registers at 32 per lane.
template <int DT, int NU, bool LR>
__device__ __forceinline__ void score_rows(const ScoreArgs& a, const DevSeg& sg, int r0, int r1,
                                           int lane, uint32_t& nsp, Lrn& lr)
{
    constexpr int RPI = NU >= MSAO_ROW_BATCH_UNITS ? 1 : MSAO_ROW_BATCH_UNITS / NU;
    const int voff = lane * 16;
    TokBuf tb{};
    vec4 wv[NU];
    if constexpr (LR && NU <= 3) load_head<NU>(wv, sg, voff);
    if constexpr (NU > 4) {
        for (int r = r0; r < r1; ++r) {
            vec4 A[1][NU];
            load_rows<NU, 1>(A, sg, r, r1, voff);
            rows_batch<DT, NU, 1, LR>(a, sg, A, r0, r, r1, lane, nsp, tb, wv, lr);
        }
    } else {
        vec4 A[RPI][NU], B[RPI][NU];
        load_rows<NU, RPI>(A, sg, r0, r1, voff);
        int r = r0;
        while (true) {
            if (r + RPI < r1) load_rows<NU, RPI>(B, sg, r + RPI, r1, voff);
            rows_batch<DT, NU, RPI, LR>(a, sg, A, r0, r, r1, lane, nsp, tb, wv, lr);
            r += RPI;
            if (r >= r1) break;
            if (r + RPI < r1) load_rows<NU, RPI>(A, sg, r + RPI, r1, voff);
            rows_batch<DT, NU, RPI, LR>(a, sg, B, r0, r, r1, lane, nsp, tb, wv, lr);
            r += RPI;
            if (r >= r1) break;
        }
    }
}

// Any row width: units processed in blocks of 4.
template <int DT, bool LR>
__device__ void score_rows_generic(const ScoreArgs& a, const DevSeg& sg, int r0, int r1, int lane,
                                   uint32_t& nsp, Lrn& lr)
{
    const float tau = a.t.tau;
    const Thr th = bf16_thresholds(tau);
    const int nu = (sg.nchunk + kWave - 1) / kWave;
    const int rb = sg.nchunk * 16;
    const bool copy = a.out && sg.copy_in_score;
    const rsrc_t rw = make_rsrc(sg.head_w, LR && sg.head_w ? rb : 0);
    TokBuf tb{};
    for (int r = r0; r < r1; ++r) {
        const rsrc_t rs = make_rsrc(sg.data + (int64_t)r * sg.stride_bytes, rb);
        const rsrc_t rd = make_rsrc(a.out + sg.out_off + (int64_t)r * rb, copy ? rb : 0);
        TokStat s{0u, 0u, 0.0f, 0.0f, 0.0f};
        float yacc = 0.0f;
        for (int u0 = 0; u0 < nu; u0 += 4) {
            vec4 v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) v[u] = bload(rs, ((u0 + u) * kWave + lane) * 16);
            if (copy) {
#pragma unroll
                for (int u = 0; u < 4; ++u) bstore(v[u], rd, ((u0 + u) * kWave + lane) * 16);
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) chunk_stats<DT>(v[u], tau, th, s.act, s.l1, s.l2);
            if constexpr (LR) {
                if (sg.head_w) {
#pragma unroll
                    for (int u = 0; u < 4; ++u)
                        yacc = dot_chunk<DT>(v[u], bload_gather(rw, ((u0 + u) * kWave + lane) * 16), yacc);
                }
            }
        }
        s.l1 = wave_sum(s.l1);
        s.l2 = wave_sum(s.l2);
        float y = 0.0f;
        if constexpr (LR) {
            if (sg.head_w) y = wave_sum(yacc);
            lrn_add(lr, s);
        }
        const int slot = (r - r0) & 63;
        tokbuf_put(tb, slot, lane, s, y);
        if (slot == 63 || r == r1 - 1) tokbuf_flush<LR>(a, sg, tb, r - slot, 1, slot + 1, lane, false, kModeScore);
        nsp += s.act < (uint32_t)sg.A_s;
    }
}

// Frames [t0, t1) of patch p of a temporal segment (rows t*P + p). The
// previous frame's values and activity ballots stay in registers; frame t+1
// is loaded before frame t is reduced. A run that starts after frame 0 first
// loads frame t0-1 (its halo).
template <int DT, int NU, bool LR>
__device__ __forceinline__ void score_chain(const ScoreArgs& a, const DevSeg& sg, int p, int t0, int t1,
                                            int lane, uint32_t& nsp, uint64_t& dsum, Lrn& lr)
{
    using L = Lane<DT>;
    constexpr int EPC = L::EPC;
    constexpr int NE = NU * EPC;
    const float tau = a.t.tau;
    const Thr th = bf16_thresholds(tau);
    const int64_t fstride = (int64_t)sg.P * sg.stride_bytes;
    const uint8_t* base = sg.data + (int64_t)p * sg.stride_bytes;
    const int rb = sg.nchunk * 16;
    const int voff = lane * 16;
    auto load = [&](vec4 (&v)[NU], int t, bool ok) {
        const rsrc_t rs = make_rsrc(base + (ok ? (int64_t)t * fstride : 0), ok ? rb : 0);
#pragma unroll
        for (int u = 0; u < NU; ++u) v[u] = bload(rs, voff + u * 1024);
    };
    float prev[NE];
    uint64_t pmask[NE];
    {
        vec4 v[NU];
        load(v, t0 - 1, t0 > 0);
#pragma unroll
        for (int u = 0; u < NU; ++u) {
            L::widen(v[u], &prev[u * EPC]);
#pragma unroll
            for (int e = 0; e < EPC; ++e) pmask[u * EPC + e] = __ballot(active(prev[u * EPC + e], tau));
        }
    }
    vec4 cur[NU];
    load(cur, t0, true);
    vec4 wv[NU];
    if constexpr (LR && NU <= 2) load_head<NU>(wv, sg, voff);
    TokBuf tb{};
    for (int t = t0; t < t1; ++t) {
        vec4 nxt[NU];
        load(nxt, t + 1, t + 1 < t1);
        if (a.out && sg.copy_in_score) copy_row_out<NU>(a, sg, t * sg.P + p, cur, voff);
        TokStat s{0u, 0u, 0.0f, 0.0f, 0.0f};
        float yacc = 0.0f;
        if constexpr (LR) {
            if (sg.head_w) {
#pragma unroll
                for (int u = 0; u < NU; ++u) {
                    // the chain already holds the previous frame: re-read (L1 hits) beyond 2 units
                    const vec4 w = NU > 2 ? bload_gather(make_rsrc(sg.head_w, sg.nchunk * 16), voff + u * 1024) : wv[u];
                    yacc = dot_chunk<DT>(cur[u], w, yacc);
                }
            }
        }
#pragma unroll
        for (int u = 0; u < NU; ++u)
            chunk_chain<DT>(cur[u], tau, th, &prev[u * EPC], &pmask[u * EPC], s.act, s.d, s.l1, s.l2, s.res);
        s.l1 = wave_sum(s.l1);
        s.l2 = wave_sum(s.l2);
        s.res = wave_sum(s.res);
        float y = 0.0f;
        if constexpr (LR) {
            if (sg.head_w) y = wave_sum(yacc);
            lrn_add(lr, s);
        }
        const int slot = (t - t0) & 63;
        tokbuf_put(tb, slot, lane, s, y);
        if (slot == 63 || t == t1 - 1)
            tokbuf_flush<LR>(a, sg, tb, (t - slot) * sg.P + p, sg.P, slot + 1, lane, true, a.mode);
        nsp += s.act < (uint32_t)sg.A_s;
        if (t >= 1) dsum += s.d;
#pragma unroll
        for (int u = 0; u < NU; ++u) cur[u] = nxt[u];
    }
}

// Any row width: the previous frame's row is re-read (it was just read by
// this wavefront, so it is normally served by the L2).
template <int DT, bool LR>
__device__ void score_chain_generic(const ScoreArgs& a, const DevSeg& sg, int p, int t0, int t1, int lane,
                                    uint32_t& nsp, uint64_t& dsum, Lrn& lr)
{
    using L = Lane<DT>;
    constexpr int EPC = L::EPC;
    const float tau = a.t.tau;
    const int64_t fstride = (int64_t)sg.P * sg.stride_bytes;
    const uint8_t* base = sg.data + (int64_t)p * sg.stride_bytes;
    const int nu = (sg.nchunk + kWave - 1) / kWave;
    const int rb = sg.nchunk * 16;
    const bool copy = a.out && sg.copy_in_score;
    const rsrc_t rw = make_rsrc(sg.head_w, LR && sg.head_w ? rb : 0);
    TokBuf tb{};
    for (int t = t0; t < t1; ++t) {
        const rsrc_t rc = make_rsrc(base + (int64_t)t * fstride, rb);
        const rsrc_t rp = make_rsrc(base + (t > 0 ? (int64_t)(t - 1) * fstride : 0), t > 0 ? rb : 0);
        const rsrc_t rd = make_rsrc(a.out + sg.out_off + (int64_t)(t * sg.P + p) * rb, copy ? rb : 0);
        TokStat s{0u, 0u, 0.0f, 0.0f, 0.0f};
        float yacc = 0.0f;
        for (int u0 = 0; u0 < nu; u0 += 2) {
            vec4 v[2], w[2];
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const int off = ((u0 + u) * kWave + lane) * 16;
                v[u] = bload(rc, off);
                w[u] = bload(rp, off);
            }
            if (copy) {
#pragma unroll
                for (int u = 0; u < 2; ++u) bstore(v[u], rd, ((u0 + u) * kWave + lane) * 16);
            }
            if constexpr (LR) {
                if (sg.head_w) {
#pragma unroll
                    for (int u = 0; u < 2; ++u)
                        yacc = dot_chunk<DT>(v[u], bload_gather(rw, ((u0 + u) * kWave + lane) * 16), yacc);
                }
            }
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                float x[EPC], y[EPC];
                L::widen(v[u], x);
                L::widen(w[u], y);
#pragma unroll
                for (int e = 0; e < EPC; ++e) {
                    const uint64_t m = __ballot(active(x[e], tau));
                    const uint64_t q = __ballot(active(y[e], tau));
                    s.act += (uint32_t)__popcll(m);
                    s.d += (uint32_t)__popcll(m ^ q);
                    s.l1 += fabsf(x[e]);
                    s.l2 = fmaf(x[e], x[e], s.l2);
                    const float df = x[e] - y[e];
                    s.res = fmaf(df, df, s.res);
                }
            }
        }
        s.l1 = wave_sum(s.l1);
        s.l2 = wave_sum(s.l2);
        s.res = wave_sum(s.res);
        float yv = 0.0f;
        if constexpr (LR) {
            if (sg.head_w) yv = wave_sum(yacc);
            lrn_add(lr, s);
        }
        const int slot = (t - t0) & 63;
        tokbuf_put(tb, slot, lane, s, yv);
        if (slot == 63 || t == t1 - 1)
            tokbuf_flush<LR>(a, sg, tb, (t - slot) * sg.P + p, sg.P, slot + 1, lane, true, a.mode);
        nsp += s.act < (uint32_t)sg.A_s;
        if (t >= 1) dsum += s.d;
    }
}

template <int DT, bool LR>
__device__ __forceinline__ void dispatch_rows(const ScoreArgs& a, const DevSeg& sg, int r0, int r1, int lane,
                                              uint32_t& nsp, Lrn& lr)
{
    const int nu = (sg.nchunk + kWave - 1) / kWave;
    switch (nu) {
    case 1: score_rows<DT, 1, LR>(a, sg, r0, r1, lane, nsp, lr); break;
    case 2: score_rows<DT, 2, LR>(a, sg, r0, r1, lane, nsp, lr); break;
    case 3: score_rows<DT, 3, LR>(a, sg, r0, r1, lane, nsp, lr); break;
    case 4: score_rows<DT, 4, LR>(a, sg, r0, r1, lane, nsp, lr); break;
    case 5: score_rows<DT, 5, LR>(a, sg, r0, r1, lane, nsp, lr); break;
    case 6: score_rows<DT, 6, LR>(a, sg, r0, r1, lane, nsp, lr); break;
    case 7: score_rows<DT, 7, LR>(a, sg, r0, r1, lane, nsp, lr); break;
    case 8: score_rows<DT, 8, LR>(a, sg, r0, r1, lane, nsp, lr); break;
    default: score_rows_generic<DT, LR>(a, sg, r0, r1, lane, nsp, lr); break;
    }
}

// Register-resident chains are used while a lane holds at most 16 channels
// (their activity ballots live in 32 scalar registers); wider rows take the
// generic path.
template <int DT, bool LR>
__device__ __forceinline__ void dispatch_chain(const ScoreArgs& a, const DevSeg& sg, int p, int t0, int t1,
                                               int lane, uint32_t& nsp, uint64_t& dsum, Lrn& lr)
{
    const int nu = (sg.nchunk + kWave - 1) / kWave;
    if constexpr (DT == kBF16) {
        switch (nu) {
        case 1: score_chain<DT, 1, LR>(a, sg, p, t0, t1, lane, nsp, dsum, lr); break;
        case 2: score_chain<DT, 2, LR>(a, sg, p, t0, t1, lane, nsp, dsum, lr); break;
        default: score_chain_generic<DT, LR>(a, sg, p, t0, t1, lane, nsp, dsum, lr); break;
        }
    } else {
        switch (nu) {
        case 1: score_chain<DT, 1, LR>(a, sg, p, t0, t1, lane, nsp, dsum, lr); break;
        case 2: score_chain<DT, 2, LR>(a, sg, p, t0, t1, lane, nsp, dsum, lr); break;
        case 3: score_chain<DT, 3, LR>(a, sg, p, t0, t1, lane, nsp, dsum, lr); break;
        case 4: score_chain<DT, 4, LR>(a, sg, p, t0, t1, lane, nsp, dsum, lr); break;
        default: score_chain_generic<DT, LR>(a, sg, p, t0, t1, lane, nsp, dsum, lr); break;
        }
    }
}

// Workgroups are dispatched to the eight XCDs in turn (block b to XCD b % 8).
// With xcd_order set, blocks are renumbered so that each XCD takes one
// contiguous range of work items: the per-token statistics its wavefronts
// write then share cache lines only within that XCD's L2.
__device__ __forceinline__ int score_block(const ScoreArgs& a)
{
    const int b = blockIdx.x;
    if (!a.xcd_order) return b;
    const int nb = gridDim.x, x = b & 7, per = nb >> 3, rem = nb & 7;
    return x * per + min(x, rem) + (b >> 3);
}

// LR: a learned call (Eq. 3 head projections, density importance of tokens
// without a head, and the descriptor sums of Eq. 6); a separate instance, so
// that the plain kernel keeps its registers. Both are held to 96 VGPRs (five
// wavefronts per SIMD, the loads in flight this HBM-bound pass needs): the
// plain instance needs 83; the learned one, which also holds the head's
// weights of rows up to 3 KiB, takes 96 without spilling.
template <bool LR>
__global__ __launch_bounds__(kScoreBlock) __attribute__((amdgpu_waves_per_eu(5, 8))) void k_score(ScoreArgs a)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int w = uniform(a.wi_first + score_block(a) * (kScoreBlock / kWave) + (threadIdx.x >> 6));
    if (w >= a.t.n_wi_score) return;
    const int s = uniform(a.t.wi_seg[w]);
    const DevSeg sg = a.t.seg[s];
    const int q = w - sg.wi_begin;
    uint32_t nsp = 0;
    uint64_t dsum = 0;
    Lrn lr{0u, 0.0f, 0.0f};
    if (sg.temporal) {
        const int p = q % sg.P;
        const int t0 = (q / sg.P) * sg.per_item;
        const int t1 = min(sg.T, t0 + sg.per_item);
        if (sg.dtype == kBF16) dispatch_chain<kBF16, LR>(a, sg, p, t0, t1, lane, nsp, dsum, lr);
        else dispatch_chain<kF32, LR>(a, sg, p, t0, t1, lane, nsp, dsum, lr);
    } else {
        const int r0 = q * sg.per_item;
        const int r1 = min(sg.n_tok, r0 + sg.per_item);
        if (a.mode == kModeTemporal) {
            // temporal term only: tokens outside temporal segments get d = res = 0
            for (int r = r0 + lane; r < r1; r += kWave) {
                if (a.tok.d) a.tok.d[sg.tok_off + r] = 0u;
                if (a.tok.res) a.tok.res[sg.tok_off + r] = 0.0f;
            }
        } else if (sg.dtype == kBF16) {
            dispatch_rows<kBF16, LR>(a, sg, r0, r1, lane, nsp, lr);
        } else {
            dispatch_rows<kF32, LR>(a, sg, r0, r1, lane, nsp, lr);
        }
    }
    if (lane == 0) {
        Partial pr;
        pr.nsparse = nsp;
        pr.pad_ = 0u;
        pr.dsum = dsum;
        a.t.partial[w] = pr;
        if constexpr (LR) a.t.partial_x[w] = PartialX{lr.asum, lr.l1, lr.l2, 0u};
    }
}

// ---------------------------------------------------------------- k_pair

// bf16 clips whose rows are 512, 1024, 1536 or 2048 bytes (and that are not
// kept whole, whose rows the chain pass copies out). A wavefront takes two
// adjacent patch positions p0, p0 + 1 over a range of up to 32 frames: lanes
// 0-31 hold the first position's row of a frame, lanes 32-63 the second's, so
// each frame is one run of consecutive rows (4 KiB for 1024 channels), and a
// block's kPairWaves wavefronts take consecutive pairs of positions over the
// same frames. The frames of a range follow one another in a ring of
// kPairRing register sets: frame t is scored against its predecessor in the
// set before it, and once a unit of that predecessor has been used the same
// unit of frame t + kPairRing - 1 is loaded into its registers, so two frames
// beyond the next are in flight while one is scored. A range after a clip's
// first reads the frame before it (halo). Per channel the arithmetic is
// vector-only: the activity sign of tau - |x| as packed 16-bit differences,
// four of them gathered into one word of 0x00/0xFF bytes whose popcount (/8)
// gives the active count and, XOR the previous frame's word, the changed
// count d; L1 and L2 as bf16 pair dot products; res from the widened values
// of this and the previous frame. Half-wavefront sums end in lanes 31 and 63
// and are parked in a token buffer (lane 2i + h: frame t0 + i, position
// p0 + h), written out once per wavefront, so the frame loop issues no stores
// and every wait in it is for one known load.

typedef short s16x2 __attribute__((ext_vector_type(2)));

// Sum over each 16-lane row (every lane of the row gets it), then rows 1 and
// 3 add the sums of rows 0 and 2: lanes 16-31 hold the sum of lanes 0-31,
// lanes 48-63 the sum of lanes 32-63.
__device__ __forceinline__ float half_sum(float v)
{
    v += dpp_f<0xB1>(v);
    v += dpp_f<0x4E>(v);
    v += dpp_f<0x141>(v);
    v += dpp_f<0x140>(v);
    v += dpp_f<0x142>(v);
    return v;
}

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_all_u(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}

__device__ __forceinline__ uint32_t half_sum_u(uint32_t v)
{
    v += dpp_all_u<0xB1>(v);
    v += dpp_all_u<0x4E>(v);
    v += dpp_all_u<0x141>(v);
    v += dpp_all_u<0x140>(v);
    v += dpp_all_u<0x142>(v);
    return v;
}

struct PairSums {
    float l1, l2, res;
    uint32_t act, chg;  // 8 per active channel, 8 per changed channel
};

// tau - |x| per 16-bit half: negative (sign bit set) iff the channel is active.
__device__ __forceinline__ uint32_t act_sign(uint32_t th2, uint32_t x)
{
    return __builtin_bit_cast(uint32_t, __builtin_bit_cast(s16x2, th2) - __builtin_bit_cast(s16x2, x & 0x7FFF7FFFu));
}

// One frame of this lane's position (4 NU dwords, 8 NU channels) against the
// previous frame's raw words y and activity words pq; nq gets this frame's.
// after(u) runs once unit u of y has been used.
template <int NU, typename Hook>
__device__ __forceinline__ PairSums pair_frame(const vec4 (&v)[NU], const vec4 (&y)[NU], uint32_t th2,
                                               const uint32_t (&pq)[NU * 2], uint32_t (&nq)[NU * 2], Hook&& after)
{
    PairSums c{0.0f, 0.0f, 0.0f, 0u, 0u};
#pragma unroll
    for (int u = 0; u < NU; ++u) {
        uint32_t sg[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const uint32_t x = v[u][e], yp = y[u][e];
            sg[e] = act_sign(th2, x);
            c.l1 = dot2(x & 0x7FFF7FFFu, kBf16OnePair, c.l1);
            c.l2 = dot2(x, x, c.l2);
            const float dlo = __uint_as_float(x << 16) - __uint_as_float(yp << 16);
            const float dhi = __uint_as_float(x & 0xFFFF0000u) - __uint_as_float(yp & 0xFFFF0000u);
            c.res = fmaf(dlo, dlo, c.res);
            c.res = fmaf(dhi, dhi, c.res);
        }
#pragma unroll
        for (int e = 0; e < 2; ++e) {
            // bytes 0xFF / 0x00 from the sign bits 15 and 31 of two words
            const uint32_t m = __builtin_amdgcn_perm(sg[2 * e + 1], sg[2 * e], 0x0B0A0908u);
            c.act += (uint32_t)__builtin_popcount(m);
            c.chg += (uint32_t)__builtin_popcount(m ^ pq[u * 2 + e]);
            nq[u * 2 + e] = m;
        }
        after(u);
    }
    return c;
}

// Activity words of a frame (the halo frame before a block's range).
template <int NU>
__device__ __forceinline__ void pair_words(const vec4 (&v)[NU], uint32_t th2, uint32_t (&nq)[NU * 2])
{
#pragma unroll
    for (int u = 0; u < NU; ++u)
#pragma unroll
        for (int e = 0; e < 2; ++e)
            nq[u * 2 + e] = __builtin_amdgcn_perm(act_sign(th2, v[u][2 * e + 1]), act_sign(th2, v[u][2 * e]),
                                                  0x0B0A0908u);
}

// The two positions' statistics of one frame (half sums in lanes 31 and 63).
struct PairTok {
    float l1, l2, res;
    uint32_t cnt;  // active count | d << 16
};

__device__ __forceinline__ PairTok pair_reduce(const PairSums& c)
{
    return PairTok{half_sum(c.l1), half_sum(c.l2), half_sum(c.res), half_sum_u((c.act >> 3) | ((c.chg >> 3) << 16))};
}

// Lane slot of the buffer takes lane 31's value of v, lane slot + 1 lane 63's.
template <typename T>
__device__ __forceinline__ T park(T buf, T v, bool at0, bool at1)
{
    const T a = __builtin_bit_cast(T, __builtin_amdgcn_readlane((int)__builtin_bit_cast(uint32_t, v), 31));
    const T b = __builtin_bit_cast(T, __builtin_amdgcn_readlane((int)__builtin_bit_cast(uint32_t, v), 63));
    return at0 ? a : (at1 ? b : buf);
}

template <int NU>
__device__ __forceinline__ void vcopy(vec4 (&d)[NU], const vec4 (&s)[NU])
{
#pragma unroll
    for (int u = 0; u < NU; ++u) d[u] = s[u];
}

// Writes token (frame t, position p) with its statistics: main z, l1, l2 (and
// the signature placeholder); temporal d, res, info.
__device__ __forceinline__ void pair_write(const ScoreArgs& a, const DevSeg& sg, int g, const PairTok& s, bool main,
                                           bool temporal)
{
    const TokenOut& o = a.tok;
    const uint32_t act = s.cnt & 0xFFFFu, dd = s.cnt >> 16;
    const uint32_t z = (uint32_t)sg.C - act;
    if (main) {
        if (a.mode == kModeScore) {
            if (o.z) o.z[g] = z;
            if (o.l1) o.l1[g] = s.l1;
            if (o.l2) o.l2[g] = s.l2;
        }
        if (o.sig) o.sig[g] = 0ull;
    }
    if (temporal) {
        if (a.mode == kModeScore && o.info) {
            float red = sg.lam_s * (float)z;
            red += sg.lam_t * (float)((uint32_t)sg.C - dd);
            o.info[g] = 1.0f - red * __builtin_amdgcn_rcpf((float)sg.C);
        }
        if (o.d) o.d[g] = dd;
        if (o.res) o.res[g] = s.res;
    }
}

// Work item q of a k_pair segment: pair j = q mod the pair count, range
// q / the pair count (none past the clip's end: the items of a segment are
// rounded up to whole blocks).
template <int NU>
__device__ __forceinline__ void score_pair(const ScoreArgs& a, const DevSeg& sg, int q, int lane, uint32_t& nsp,
                                           uint32_t& dsum)
{
    constexpr int RING = kPairRing;
    static_assert(RING % 2 == 0 && RING >= 2, "activity words alternate between two sets with the frame's parity");
    const int npairs = (sg.P + 1) >> 1;
    const int tbi = uniform(q / npairs), j = uniform(q - (q / npairs) * npairs);
    const int F = uniform(sg.per_item);
    const int t0 = uniform(min(sg.T, tbi * F)), t1 = uniform(min(sg.T, t0 + F));
    if (t0 >= t1) return;
    const int p0 = uniform(2 * j);
    const int h = lane >> 5, l = lane & 31;
    const bool two = uniform(p0 + 1 < sg.P ? 1 : 0) != 0;
    const bool present = h == 0 || two;
    const int rb = uniform(sg.nchunk * 16);
    const int64_t fstride = (int64_t)sg.P * sg.stride_bytes;
    const uint8_t* base = sg.data + (int64_t)p0 * sg.stride_bytes;
    const int nrec = uniform(two ? (int)sg.stride_bytes + rb : rb);
    // unit u of this lane's row at voff + 512 u; a missing second position
    // reads as zeros (an offset past the resource)
    const int voff = present ? h * (int)sg.stride_bytes + l * 16 : 0x7FFFFFF0;
    // a frame outside the range reads as zeros from an empty resource: every
    // load is issued, so the waits count them exactly
    auto frame_rsrc = [&](int t, bool ok) {
        return make_rsrc(base + (ok ? (int64_t)t * fstride : 0), ok ? nrec : 0);
    };
    auto load = [&](vec4 (&v)[NU], int t, bool ok) {
        const rsrc_t rs = frame_rsrc(t, ok);
#pragma unroll
        for (int u = 0; u < NU; ++u) v[u] = bload(rs, voff + u * 512);
    };
    const uint32_t lo = bf16_thresholds(a.t.tau).lo;
    const uint32_t th2 = lo | (lo << 16);
    PairTok tok{0.0f, 0.0f, 0.0f, 0u};
    // frame t0 + i in R[i mod RING] with its activity words in Q[i mod 2];
    // the frame before t0 (the zero frame before the clip's first) in
    // R[RING - 1], its words in Q[1]
    vec4 R[RING][NU];
    uint32_t Q[2][NU * 2];
    load(R[RING - 1], t0 - 1, t0 > 0);
#pragma unroll
    for (int i = 0; i < RING - 1; ++i) load(R[i], t0 + i, t0 + i < t1);
    pair_words<NU>(R[RING - 1], th2, Q[1]);
    int t = t0;
    while (t < t1) {
#pragma unroll
        for (int i = 0; i < RING; ++i) {
            if (t >= t1) break;
            const int pi = (i + RING - 1) % RING;
            const rsrc_t rs = frame_rsrc(t + RING - 1, t + RING - 1 < t1);
            const PairSums c = pair_frame<NU>(R[i], R[pi], th2, Q[(i + 1) & 1], Q[i & 1], [&](int u) {
                R[pi][u] = bload(rs, voff + u * 512);
                // keep the load here, where its registers have just been freed
                __builtin_amdgcn_sched_barrier(0);
            });
            const PairTok r = pair_reduce(c);
            const int slot = 2 * (t - t0);
            const bool at0 = lane == slot, at1 = lane == slot + 1;
            tok.l1 = park(tok.l1, r.l1, at0, at1);
            tok.l2 = park(tok.l2, r.l2, at0, at1);
            tok.res = park(tok.res, r.res, at0, at1);
            tok.cnt = park(tok.cnt, r.cnt, at0, at1);
            ++t;
        }
    }
    // the range's tokens: lane 2i + h holds frame t0 + i, position p0 + h
    const int nslot = 2 * (t1 - t0);
    const int fi = lane >> 1, hh = lane & 1;
    const bool mine = lane < nslot && (hh == 0 || two);
    const uint32_t act = tok.cnt & 0xFFFFu, dd = tok.cnt >> 16;
    if (mine) pair_write(a, sg, sg.tok_off + (t0 + fi) * sg.P + p0 + hh, tok, true, true);
    nsp += (uint32_t)__popcll(__ballot(mine && act < (uint32_t)sg.A_s));
    uint32_t dpart = mine && t0 + fi >= 1 ? dd : 0u;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) dpart += (uint32_t)__shfl_xor((int)dpart, o);
    dsum += dpart;
}

// One wavefront per k_pair work item; consecutive blocks (neighbouring pairs
// of positions, whose statistics share cache lines) run on one XCD.
__global__ __launch_bounds__(kPairWaves * 64) __attribute__((amdgpu_waves_per_eu(1, kPairWavesPerEU)))
void k_pair(ScoreArgs a)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = uniform(threadIdx.x >> 6);
    const int nb = gridDim.x, b = blockIdx.x, x = b & 7, per = nb >> 3, rem = nb & 7;
    const int vb = uniform(x * per + min(x, rem) + (b >> 3));
    const int w = vb * kPairWaves + wv;
    const int s = uniform(a.t.wi_seg[w]);
    const DevSeg sg = a.t.seg[s];
    const int q = w - sg.wi_begin;
    uint32_t nsp = 0, dsum = 0;  // wave-uniform
    switch (sg.nchunk >> 5) {  // rows of 512-byte units
    case 1: score_pair<1>(a, sg, q, lane, nsp, dsum); break;
    case 2: score_pair<2>(a, sg, q, lane, nsp, dsum); break;
    case 3: score_pair<3>(a, sg, q, lane, nsp, dsum); break;
    default: score_pair<4>(a, sg, q, lane, nsp, dsum); break;
    }
    if (lane == 0) {
        Partial pr;
        pr.nsparse = nsp;
        pr.pad_ = 0u;
        pr.dsum = dsum;
        a.t.partial[w] = pr;
    }
}

// ---------------------------------------------------------------- k_post


constexpr int kRadixBits = 11;
constexpr int kRadixBins = 1 << kRadixBits;

// Shared state of a post-scoring block of NT threads.
typedef unsigned int post_u32x4 __attribute__((ext_vector_type(4)));

template <int NT>
struct PostShared {
    static constexpr int kWaves = NT / kWave;
    static_assert(kWaves % kNumMod == 0, "the request role splits the wavefronts evenly over the modalities");
    static_assert(kRadixBins % NT == 0, "every thread owns the same number of radix bins");
    alignas(16) uint32_t hist[kRadixBins];  // read 16 bytes at a time by the digit scan
    uint32_t scan[kWaves];
    uint32_t wcnt[kWaves][4];
    unsigned long long lo, hi, red;
    uint64_t vsel;            // selection: key of the wanted rank among few candidates
    uint64_t nsp[kWaves], dsum[kWaves], ntok[kNumMod], qbits[kNumMod];
    uint32_t digit, below, in_bin, ncand;
    uint32_t ncopy;           // selection: candidates copied for a direct rank
    // learned calls
    uint64_t asum[kWaves], csum[kWaves];
    double l1[kWaves], l2[kWaves];
    float fred[kWaves];
    float fred4[kWaves][kNumMod];
    float alpha[kNumMod];
};

// Radix candidates copied out of the staged keys once few remain (LDS entries
// after the keys).
constexpr int kMaxCand = 2048;
constexpr int kSmallCand = 256;  // candidates ranked directly instead of by further digit passes
__device__ __host__ __forceinline__ int cand_cap_for(int keys_cap) { return keys_cap < kMaxCand ? keys_cap : kMaxCand; }

// Block-wide sum of a 64-bit integer (exact, so the order does not matter).
template <int NT>
__device__ __forceinline__ uint64_t block_sum_u64(uint64_t v, PostShared<NT>& sh)
{
    v = wave_sum_u64(v);
    __syncthreads();
    if (threadIdx.x == 0) sh.red = 0ull;
    __syncthreads();
    if ((threadIdx.x & (kWave - 1)) == 0 && v) atomicAdd(&sh.red, (unsigned long long)v);
    __syncthreads();
    return (uint64_t)sh.red;
}

// Block-wide exclusive scan of 32-bit counts in thread order; *total gets the sum.
template <int NT>
__device__ __forceinline__ uint32_t block_exscan(uint32_t v, PostShared<NT>& sh, uint32_t* total)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int wid = threadIdx.x >> 6;
    uint32_t x = v;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const uint32_t y = __shfl_up(x, o);
        if (lane >= o) x += y;
    }
    __syncthreads();
    if (lane == kWave - 1) sh.scan[wid] = x;
    __syncthreads();
    uint32_t before = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < (NT / kWave); ++i) {
        const uint32_t t = sh.scan[i];
        if (i < wid) before += t;
        tot += t;
    }
    *total = tot;
    return before + x - v;
}

struct RMAgg {
    uint64_t ntok, nsparse, dsum, qbits;
};

// Eq. 4 and Eq. 5 integer aggregates of request r, all four modalities:
// wavefront w sums every kParts-th 64-item stripe of the scoring partials of
// modality w % 4. Every thread of the block calls this and receives the same
// values.
template <int NT>
__device__ void rm_aggregate_all(const Tables& t, int r, PostShared<NT>& sh, RMAgg g[kNumMod])
{
    constexpr int kParts = (NT / kWave) / kNumMod;
    const int wid = threadIdx.x >> 6;
    const int m = wid % kNumMod, part = wid / kNumMod;
    const int lane = threadIdx.x & (kWave - 1);
    const RmEntry e = t.rm[r * kNumMod + m];
    uint64_t nsp = 0, ds = 0;
    constexpr int U = 8;  // partials in flight per lane (an audio track has ~500)
    for (int j = e.rng_begin; j < e.rng_end; ++j) {
        const WiRange wr = t.rm_rng[j];
        for (int w0 = wr.begin + part * kWave + lane; w0 < wr.end; w0 += U * kParts * kWave) {
            Partial pr[U];
#pragma unroll
            for (int u = 0; u < U; ++u) pr[u] = t.partial[min(w0 + u * kParts * kWave, wr.end - 1)];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (w0 + u * kParts * kWave < wr.end) {
                    nsp += pr[u].nsparse;
                    ds += pr[u].dsum;
                }
            }
        }
    }
    nsp = wave_sum_u64(nsp);
    ds = wave_sum_u64(ds);
    __syncthreads();
    if (lane == 0) {
        sh.nsp[wid] = nsp;
        sh.dsum[wid] = ds;
        if (part == 0) {
            sh.ntok[m] = e.ntok;
            sh.qbits[m] = e.qbits;
        }
    }
    __syncthreads();
#pragma unroll
    for (int mm = 0; mm < kNumMod; ++mm) {
        g[mm].ntok = sh.ntok[mm];
        g[mm].qbits = sh.qbits[mm];
        uint64_t a = 0, b = 0;
#pragma unroll
        for (int q = 0; q < kParts; ++q) {
            a += sh.nsp[q * kNumMod + mm];
            b += sh.dsum[q * kNumMod + mm];
        }
        g[mm].nsparse = a;
        g[mm].dsum = t.hdsum ? t.hdsum[r * kNumMod + mm] : b;
    }
}

// Sec. 4.1.3: softmax of the logits over the modalities present.
__device__ void modal_softmax(const double al[kNumMod], const bool pres[kNumMod], double beta[kNumMod])
{
#pragma clang fp contract(off)
    double mx = -INFINITY;
#pragma unroll
    for (int m = 0; m < kNumMod; ++m)
        if (pres[m] && al[m] > mx) mx = al[m];
    // each exponential once; exp(0) is exactly 1 (the logits of equal
    // relevance, e.g. none given), so it is not evaluated
    double ex[kNumMod], den = 0.0;
#pragma unroll
    for (int m = 0; m < kNumMod; ++m) {
        const double x = al[m] - mx;
        ex[m] = pres[m] ? (x == 0.0 ? 1.0 : exp(x)) : 0.0;
        if (pres[m]) den += ex[m];
    }
#pragma unroll
    for (int m = 0; m < kNumMod; ++m) beta[m] = pres[m] ? ex[m] / den : 0.0;
}

struct MasTerms {
    double rho, tterm, beta, mas;
    bool has_t;
};

// Eq. 4 ratio, temporal term and Eq. 7 for one (request, modality), in double.
__device__ MasTerms mas_terms(const Tables& t, const RMAgg& g, double beta, int m)
{
#pragma clang fp contract(off)
    MasTerms o;
    o.beta = beta;
    o.rho = (double)g.nsparse / (double)g.ntok;
    o.has_t = g.qbits > 0;
    o.tterm = 0.0;
    if (o.has_t) {
        const double gamma_avg = (double)g.dsum / (double)g.qbits;
        o.tterm = (t.flags & kFlagLiteral) ? gamma_avg : 1.0 - gamma_avg;
    }
    double inner = 1.0 - (double)t.lam_s[m] * o.rho;
    if (o.has_t) inner = inner - (double)t.lam_t[m] * o.tterm;
    inner = inner < 0.0 ? 0.0 : inner;
    inner = inner > 1.0 ? 1.0 : inner;
    o.mas = 1.0 - beta * inner;
    return o;
}

// MAS of every modality of request r (terms[m] is zero where absent).
__device__ void request_terms(const Tables& t, int r, const RMAgg g[kNumMod], MasTerms terms[kNumMod],
                              bool pres[kNumMod])
{
    double al[kNumMod], beta[kNumMod];
#pragma unroll
    for (int m = 0; m < kNumMod; ++m) {
        pres[m] = g[m].ntok > 0;
        al[m] = (double)t.alpha[r * kNumMod + m];
    }
    modal_softmax(al, pres, beta);
#pragma unroll
    for (int m = 0; m < kNumMod; ++m) {
        terms[m] = MasTerms{0.0, 0.0, 0.0, 0.0, false};
        if (pres[m]) terms[m] = mas_terms(t, g[m], beta[m], m);
    }
}

template <int NT>
__device__ void role_request(const PostArgs& a, int r, PostShared<NT>& sh)
{
    const Tables& t = a.t;
    RMAgg g[kNumMod];
    rm_aggregate_all(t, r, sh, g);
    if (threadIdx.x != 0) return;
    MasTerms o[kNumMod];
    bool pres[kNumMod];
    request_terms(t, r, g, o, pres);
#pragma unroll
    for (int m = 0; m < kNumMod; ++m) {
        const int x = r * kNumMod + m;
        if (a.temporal_only) {
            if (a.req.temporal) a.req.temporal[x] = (float)o[m].tterm;
            continue;
        }
        if (a.req.agg) {
            a.req.agg[x * 4 + 0] = g[m].ntok;
            a.req.agg[x * 4 + 1] = g[m].nsparse;
            a.req.agg[x * 4 + 2] = g[m].dsum;
            a.req.agg[x * 4 + 3] = g[m].qbits;
        }
        if (a.req.rho) a.req.rho[x] = (float)o[m].rho;
        if (a.req.temporal) a.req.temporal[x] = (float)o[m].tterm;
        if (a.req.beta) a.req.beta[x] = (float)o[m].beta;
        if (a.req.mas) a.req.mas[x] = (float)o[m].mas;
        if (a.req.present) a.req.present[x] = pres[m] ? 1 : 0;
    }
}

// The modality descriptor z_m of Eq. 6 (zero for an absent modality).
__device__ __forceinline__ void modality_descriptor(bool pres, const MasTerms& pre, uint64_t asum, uint64_t csum,
                                                    double l1, double l2, uint64_t ntok, double* z)
{
#pragma clang fp contract(off)
    z[0] = pres ? 1.0 : 0.0;
    z[1] = pre.rho;
    z[2] = pres ? (double)asum / (double)csum : 0.0;
    z[3] = pres ? l1 / (double)csum : 0.0;
    z[4] = pres ? sqrt(l2 / (double)csum) : 0.0;
    z[5] = pre.tterm;
    z[6] = pre.has_t ? 1.0 : 0.0;
    z[7] = pres ? log(1.0 + (double)ntok) / 16.0 : 0.0;
}

__device__ __forceinline__ double wave_sum_f64(double v)
{
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) v += __shfl_xor(v, o);
    return v;
}

// Block-wide float sum in a fixed order (wavefront DPP sums, then the
// wavefronts in order), the same value in every thread.
// A learned call's request role: Eq. 4 counts from the heads' per-frame
// counts (from the density test where a segment has no head), the
// descriptor z_m of every modality, Eq. 6 on [p; z_m] when an MLP is given
// (alpha from the table otherwise), then the softmax and Eq. 7.
// The descriptor: 1, rho, sum a / sum C, sum L1 / sum C, sqrt(sum L2 / sum C),
// the temporal term (0 if none), 1 if it exists, ln(1 + Ntok) / 16.
template <int NT>
__device__ void role_request_learned(const PostArgs& a, int r, PostShared<NT>& sh)
{
    const Tables& t = a.t;
    constexpr int kParts = (NT / kWave) / kNumMod;
    const int wid = threadIdx.x >> 6, m = wid % kNumMod, part = wid / kNumMod;
    const int lane = threadIdx.x & (kWave - 1);
    const RmEntry e = t.rm[r * kNumMod + m];
    // the MLP's weights of this thread's first hidden unit (the descriptor
    // columns of W1, u = W1[:, :P] p + b1 from the head launch, and w2) are
    // the same for every modality: read them now, so that their latency
    // overlaps the aggregation
    const int P = a.mlp.prompt_dim, IN = P + kDesc, H = a.mlp.hidden;
    float w1u[kDesc], uu = 0.0f, w2u = 0.0f;
    if (a.use_mlp && (int)threadIdx.x < H) {
        const float* row = a.mlp.w1 + (int64_t)threadIdx.x * IN + P;
#pragma unroll
        for (int k = 0; k < kDesc; ++k) w1u[k] = row[k];
        uu = a.mlp_u[(int64_t)r * H + threadIdx.x];
        w2u = a.mlp.w2[threadIdx.x];
    }
    uint64_t nsp = 0, ds = 0, as = 0, cs = 0;
    double l1 = 0.0, l2 = 0.0;
    for (int j = e.rng_begin; j < e.rng_end; ++j) {
        const WiRange wr = t.rm_rng[j];
        const DevSeg& sg = t.seg[wr.seg];
        const bool head = sg.head_w != nullptr;
        if (part == 0 && lane == 0) cs += (uint64_t)sg.n_tok * (uint64_t)sg.C;
        constexpr int U = 8;  // partials in flight per lane
        for (int w0 = wr.begin + part * kWave + lane; w0 < wr.end; w0 += U * kParts * kWave) {
            Partial pr[U];
            PartialX px[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int w = min(w0 + u * kParts * kWave, wr.end - 1);
                pr[u] = t.partial[w];
                px[u] = t.partial_x[w];
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (w0 + u * kParts * kWave >= wr.end) break;
                if (!head) nsp += pr[u].nsparse;
                ds += pr[u].dsum;
                as += px[u].asum;
                l1 += (double)px[u].l1;
                l2 += (double)px[u].l2;
            }
        }
        if (head)
            for (int h = sg.hb_begin + part * kWave + lane; h < sg.hb_begin + sg.T; h += kParts * kWave)
                nsp += t.head_count[h];
    }
    nsp = wave_sum_u64(nsp);
    ds = wave_sum_u64(ds);
    as = wave_sum_u64(as);
    cs = wave_sum_u64(cs);
    l1 = wave_sum_f64(l1);
    l2 = wave_sum_f64(l2);
    __syncthreads();
    if (lane == 0) {
        sh.nsp[wid] = nsp;
        sh.dsum[wid] = ds;
        sh.asum[wid] = as;
        sh.csum[wid] = cs;
        sh.l1[wid] = l1;
        sh.l2[wid] = l2;
        if (part == 0) {
            sh.ntok[m] = e.ntok;
            sh.qbits[m] = e.qbits;
        }
    }
    __syncthreads();
    RMAgg g[kNumMod];
    double z[kNumMod][kDesc];
    bool pres[kNumMod];
    MasTerms pre[kNumMod];
#pragma unroll
    for (int mm = 0; mm < kNumMod; ++mm) {
        uint64_t n1 = 0, d1 = 0, a1 = 0, c1 = 0;
        double s1 = 0.0, s2 = 0.0;
#pragma unroll
        for (int q = 0; q < kParts; ++q) {
            const int w = q * kNumMod + mm;
            n1 += sh.nsp[w];
            d1 += sh.dsum[w];
            a1 += sh.asum[w];
            c1 += sh.csum[w];
            s1 += sh.l1[w];
            s2 += sh.l2[w];
        }
        g[mm] = RMAgg{sh.ntok[mm], n1, d1, sh.qbits[mm]};
        pres[mm] = g[mm].ntok > 0;
        pre[mm] = MasTerms{0.0, 0.0, 0.0, 0.0, false};
        if (pres[mm]) pre[mm] = mas_terms(t, g[mm], 1.0, mm);  // rho and the temporal term
        modality_descriptor(pres[mm], pre[mm], a1, c1, s1, s2, g[mm].ntok, z[mm]);
    }
    // Eq. 6: alpha = w2 . relu(W1 [p; z] + b1) + b2 for every modality at
    // once: each thread sums its hidden units' terms per modality, and one
    // block reduction (each wavefront's sums, then the wavefronts in order)
    // gives the four sums
    double al[kNumMod];
#pragma unroll
    for (int mm = 0; mm < kNumMod; ++mm) al[mm] = (double)t.alpha[r * kNumMod + mm];
    if (a.use_mlp) {
        float zf[kNumMod][kDesc];
#pragma unroll
        for (int mm = 0; mm < kNumMod; ++mm)
#pragma unroll
            for (int k = 0; k < kDesc; ++k) zf[mm][k] = (float)z[mm][k];
        float ps[kNumMod] = {0.0f, 0.0f, 0.0f, 0.0f};
        auto unit = [&](const float (&w1)[kDesc], float u, float w2) {
#pragma unroll
            for (int mm = 0; mm < kNumMod; ++mm) {
                if (!pres[mm]) continue;
                float h = u;
#pragma unroll
                for (int k = 0; k < kDesc; ++k) h = fmaf(w1[k], zf[mm][k], h);
                ps[mm] = fmaf(w2, fmaxf(h, 0.0f), ps[mm]);
            }
        };
        if ((int)threadIdx.x < H) unit(w1u, uu, w2u);
        for (int j = threadIdx.x + NT; j < H; j += NT) {
            const float* row = a.mlp.w1 + (int64_t)j * IN + P;
            float w1[kDesc];
#pragma unroll
            for (int k = 0; k < kDesc; ++k) w1[k] = row[k];
            unit(w1, a.mlp_u[(int64_t)r * H + j], a.mlp.w2[j]);
        }
#pragma unroll
        for (int mm = 0; mm < kNumMod; ++mm) ps[mm] = wave_sum(ps[mm]);
        if (lane == 0) {
#pragma unroll
            for (int mm = 0; mm < kNumMod; ++mm) sh.fred4[wid][mm] = ps[mm];
        }
        __syncthreads();
#pragma unroll
        for (int mm = 0; mm < kNumMod; ++mm) {
            if (!pres[mm]) continue;
            float sum = 0.0f;
#pragma unroll
            for (int w = 0; w < NT / kWave; ++w) sum += sh.fred4[w][mm];
            al[mm] = (double)(a.mlp.b2 + sum);
        }
    }
    if (threadIdx.x != 0) return;
    double beta[kNumMod];
    modal_softmax(al, pres, beta);
#pragma unroll
    for (int mm = 0; mm < kNumMod; ++mm) {
        const int x = r * kNumMod + mm;
        const MasTerms o = pres[mm] ? mas_terms(t, g[mm], beta[mm], mm) : MasTerms{0.0, 0.0, 0.0, 0.0, false};
        if (a.req.agg) {
            a.req.agg[x * 4 + 0] = g[mm].ntok;
            a.req.agg[x * 4 + 1] = g[mm].nsparse;
            a.req.agg[x * 4 + 2] = g[mm].dsum;
            a.req.agg[x * 4 + 3] = g[mm].qbits;
        }
        if (a.req.rho) a.req.rho[x] = (float)o.rho;
        if (a.req.temporal) a.req.temporal[x] = (float)o.tterm;
        if (a.req.beta) a.req.beta[x] = (float)o.beta;
        if (a.req.mas) a.req.mas[x] = (float)o.mas;
        if (a.mas_ws) a.mas_ws[x] = (float)o.mas;
        if (a.req.present) a.req.present[x] = pres[mm] ? 1 : 0;
        if (a.alpha_out) a.alpha_out[x] = pres[mm] ? (float)al[mm] : 0.0f;
        if (a.desc_out)
            for (int k = 0; k < kDesc; ++k) a.desc_out[x * kDesc + k] = (float)z[mm][k];
    }
}

// Eq. 5 for one frame of a temporal segment: D_t = sum of d over its tokens.
template <int NT>
__device__ void role_frame(const PostArgs& a, int f, PostShared<NT>& sh)
{
    const Tables& t = a.t;
    const DevSeg& sg = t.seg[t.frame_seg[f]];
    const int tt = f - sg.frame_off;
    const int base = sg.tok_off + tt * sg.P;
    uint64_t acc = 0;
    for (int p = threadIdx.x; p < sg.P; p += blockDim.x) acc += a.d[base + p];
    const uint64_t D = block_sum_u64(acc, sh);
    if (threadIdx.x == 0) {
#pragma clang fp contract(off)
        const double sim = 1.0 - (double)D / (double)((int64_t)sg.P * sg.E);
        if (a.frm.dframe) a.frm.dframe[f] = D;
        if (a.frm.sim) a.frm.sim[f] = (float)sim;
        if (a.frm.gamma) a.frm.gamma[f] = (float)(1.0 - sim);
    }
}

// Selection key Ms*z + Mt*(E - d), order-equivalent to L_s z / C + L_t (E -
// d) / E (E = C for bit sampling, where Ms = L_s and Mt = L_t): when one
// weight is 0 the other term alone orders the tokens, so it is used unscaled.
// A learned importance as a key: larger importance first. The bits of a
// positive float grow with its value, so their complement orders it
// downwards; NaN and values not above 0 take the largest key (importance 0).
__device__ __forceinline__ uint64_t imp_key(float m)
{
    return m > 0.0f ? (uint64_t)(~__float_as_uint(m)) : 0xFFFFFFFFull;
}

__device__ __forceinline__ uint64_t sel_key(const uint32_t* __restrict__ z, const uint32_t* __restrict__ d,
                                            const float* __restrict__ imp, int g, int kind, uint64_t Ms, uint64_t Mt,
                                            uint32_t E)
{
    switch (kind) {
    case kKeyZ: return (uint64_t)z[g];
    case kKeyE: return (uint64_t)(E - d[g]);
    case kKeyFull: return Ms * (uint64_t)z[g] + Mt * (uint64_t)(E - d[g]);
    case kKeyImp: return imp_key(imp[g]);
    default: return 0ull;
    }
}

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint32_t dpp_u(uint32_t old, uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)v, CTRL, ROW_MASK, 0xF, false);
}

// Inclusive prefix sum over the 64 lanes: row_shr 1, 2, 4, 8 give every
// 16-lane row its own prefix; row_bcast:15 and row_bcast:31 then carry the
// totals of the rows before.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t x)
{
    x += dpp_u<0x111, 0xF>(0u, x);
    x += dpp_u<0x112, 0xF>(0u, x);
    x += dpp_u<0x114, 0xF>(0u, x);
    x += dpp_u<0x118, 0xF>(0u, x);
    x += dpp_u<0x142, 0xA>(0u, x);
    x += dpp_u<0x143, 0xC>(0u, x);
    return x;
}

// Block-wide exclusive scan of 32-bit counts in thread order (DPP wavefront
// scans, then the wavefront totals through LDS); *total gets the sum.
template <int NT>
__device__ __forceinline__ uint32_t block_exscan_dpp(uint32_t v, PostShared<NT>& sh, uint32_t* total)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int wid = threadIdx.x >> 6;
    const uint32_t inc = wave_incl_scan(v);
    __syncthreads();
    if (lane == kWave - 1) sh.scan[wid] = inc;
    __syncthreads();
    uint32_t before = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < (NT / kWave); ++i) {
        const uint32_t t = sh.scan[i];
        if (i < wid) before += t;
        tot += t;
    }
    *total = tot;
    return before + inc - v;
}

// Keys of tokens [0, N) of a selection staged into LDS (when in_lds), each
// also counted in the histogram of the first radix digit, key >> shift (the
// keys lie in [0, kmax], so the first digit needs no range of its own), which
// this zeroes first (every thread of the block calls it). U
// tokens per thread are loaded before any is used, so that the global loads
// of one thread overlap; indices past N are clamped (and their values
// dropped) so that no load sits behind a branch.
template <int NT, int KIND>
__device__ __forceinline__ void stage_keys(const uint32_t* __restrict__ z, const uint32_t* __restrict__ d,
                                           const float* __restrict__ imp, int N, uint64_t Ms, uint64_t Mt, uint32_t E,
                                           bool in_lds, uint64_t* keys, uint32_t* hist, int shift, bool count)
{
    constexpr int U = 8;
    if (N <= U * NT) {
        // one batch per thread: its loads are issued first and the histogram
        // is zeroed while they are in flight (one barrier before the counting)
        uint32_t zz[U], ee[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int g = min((int)threadIdx.x + u * NT, N - 1);
            zz[u] = KIND == kKeyZ || KIND == kKeyFull ? z[g] : 0u;
            ee[u] = KIND == kKeyE || KIND == kKeyFull ? E - d[g] : 0u;
            if constexpr (KIND == kKeyImp) zz[u] = (uint32_t)imp_key(imp[g]);
        }
        for (int b = threadIdx.x; b < kRadixBins; b += NT) hist[b] = 0u;
        __syncthreads();
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int i = (int)threadIdx.x + u * NT;
            if (i < N) {
                uint64_t key = 0ull;
                if constexpr (KIND == kKeyZ || KIND == kKeyImp) key = zz[u];
                else if constexpr (KIND == kKeyE) key = ee[u];
                else if constexpr (KIND == kKeyFull) key = Ms * (uint64_t)zz[u] + Mt * (uint64_t)ee[u];
                if (in_lds) keys[i] = key;
                if (count) atomicAdd(&hist[(uint32_t)(key >> shift)], 1u);
            }
        }
        return;
    }
    for (int b = threadIdx.x; b < kRadixBins; b += NT) hist[b] = 0u;
    __syncthreads();
    for (int i0 = threadIdx.x; i0 < N; i0 += U * NT) {
        uint32_t zz[U], ee[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int g = min(i0 + u * NT, N - 1);
            zz[u] = KIND == kKeyZ || KIND == kKeyFull ? z[g] : 0u;
            ee[u] = KIND == kKeyE || KIND == kKeyFull ? E - d[g] : 0u;
            if constexpr (KIND == kKeyImp) zz[u] = (uint32_t)imp_key(imp[g]);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int i = i0 + u * NT;
            if (i < N) {
                uint64_t key = 0ull;
                if constexpr (KIND == kKeyZ || KIND == kKeyImp) key = zz[u];
                else if constexpr (KIND == kKeyE) key = ee[u];
                else if constexpr (KIND == kKeyFull) key = Ms * (uint64_t)zz[u] + Mt * (uint64_t)ee[u];
                if (in_lds) keys[i] = key;
                if (count) atomicAdd(&hist[(uint32_t)(key >> shift)], 1u);
            }
        }
    }
}

// MAS-guided keep count (Eq. 11 floor): k = min(N, ceil((1 - MAS) * N)) in double.
__device__ __forceinline__ int guided_keep_count(float mas, int N)
{
#pragma clang fp contract(off)
    double kk = ceil((1.0 - (double)mas) * (double)N);
    kk = kk > (double)N ? (double)N : kk;
    kk = kk < 0.0 ? 0.0 : kk;
    return (int)kk;
}

// Where the selection keys are read from: staged in LDS, or recomputed from
// z and d for selections larger than the LDS staging area.
struct KeySrc {
    const uint64_t* keys;
    const uint32_t* z;
    const uint32_t* d;
    const float* imp;
    int kind;
    uint64_t Ms, Mt;
    uint32_t E;
    template <bool IN_LDS>
    __device__ __forceinline__ uint64_t at(int i) const
    {
        if constexpr (IN_LDS) return keys[i];
        else return sel_key(z, d, imp, i, kind, Ms, Mt, E);
    }
};

// Rank k-1 of the N keys of a selection (range [lo, hi]) by MSD radix
// select; then this block's slice [s0, s1) of keep flags (at off + i) and
// ascending kept indices (iadd + i, written from ioff). IN_LDS: every key is
// staged in LDS.
template <int NT, bool IN_LDS>
__device__ void select_and_compact(const PostArgs& a, PostShared<NT>& sh, const KeySrc& src, uint64_t* cand,
                                   int cand_cap, int N, int k, int off, int ioff, int iadd, uint64_t lo, uint64_t hi,
                                   int s0, int s1, bool first_hist_ready)
{
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid >> 6;
    constexpr int kW = NT / kWave;
    auto key_at = [&](int i) -> uint64_t { return src.at<IN_LDS>(i); };
    // radix select of the key of rank k-1 among key - lo, most significant digit
    // first. Once the candidate range holds at most cand_cap keys, the next
    // pass also copies them to cand[] and later passes read only those.
    int ncand = -1;                // -1: passes read every key
    uint32_t in_range = (uint32_t)N;
    uint64_t prefix = 0;
    uint32_t below = 0;            // keys below the current candidate range
    uint32_t rank = (uint32_t)k - 1;
    int bits = hi > lo ? 64 - __clzll((long long)(hi - lo)) : 0;
    bool built = first_hist_ready;  // the first digit's histogram was counted while staging
    constexpr int U = 4;
    while (bits > 0) {
        const int db = bits < kRadixBits ? bits : kRadixBits;
        const int shift = bits - db;
        const uint64_t mask = (1ull << db) - 1ull;
        // copy out the candidates once they are few (and fewer than half the keys)
        const bool collect = ncand < 0 && in_range <= (uint32_t)cand_cap && 2 * in_range < (uint32_t)N;
        const bool first = in_range == (uint32_t)N && below == 0u && prefix == 0ull;
        if (!built && collect && in_range <= (uint32_t)kSmallCand) {
            // so few keys are left that a copy of them and a direct rank among
            // them cost less than the remaining digit passes (their count was
            // reset by the digit scan before its barrier)
            for (int base = wid * kWave; base < N; base += U * NT) {
                uint64_t x[U];
#pragma unroll
                for (int u = 0; u < U; ++u) x[u] = key_at(min(base + u * NT + lane, N - 1)) - lo;
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const bool match = base + u * NT + lane < N && (x[u] >> bits) == prefix;
                    const uint64_t m = __ballot(match);
                    if (m) {
                        uint32_t at = 0;
                        if (lane == 0) at = atomicAdd(&sh.ncopy, (uint32_t)__popcll(m));
                        at = (uint32_t)__shfl((int)at, 0);
                        if (match) cand[at + lanes_below(m)] = x[u];
                    }
                }
            }
            __syncthreads();
            const int m = (int)sh.ncopy;
            // candidate c = (w % cw) * 64 + lane is counted against the j-range
            // part w / cw of the candidates by wavefront w; the parts' counts
            // of smaller and of not larger candidates meet in LDS
            const int cw = (m + kWave - 1) / kWave, nparts = kW / cw;
            const int c = (wid % cw) * kWave + lane, part = wid / cw;
            const int per = (m + nparts - 1) / nparts, j0 = min(m, part * per), j1 = min(m, j0 + per);
            uint32_t lt = 0, le = 0;
            if (part < nparts && c < m) {
                const uint64_t v = cand[c];
                for (int j = j0; j < j1; j += 4) {
                    uint64_t x[4];
#pragma unroll
                    for (int u = 0; u < 4; ++u) x[u] = cand[min(j + u, j1 - 1)];
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const bool in = j + u < j1;
                        lt += in && x[u] < v ? 1u : 0u;
                        le += in && x[u] <= v ? 1u : 0u;
                    }
                }
            }
            const int slot = part * cw * kWave + c;  // < kW * 64 = NT
            if (part < nparts) {
                sh.hist[slot] = lt;
                sh.hist[NT + slot] = le;
            }
            __syncthreads();
            if (tid < m) {
                const int cc = tid;
                uint32_t lt_all = 0, le_all = 0;
                for (int q = 0; q < nparts; ++q) {
                    lt_all += sh.hist[q * cw * kWave + cc];
                    le_all += sh.hist[NT + q * cw * kWave + cc];
                }
                // every candidate equal to the one of this rank writes the same values
                if (lt_all <= rank && rank < le_all) {
                    sh.vsel = cand[cc];
                    sh.below = lt_all;
                }
            }
            __syncthreads();
            prefix = sh.vsel;
            below += sh.below;
            bits = 0;
            break;
        }
        if (!built) {
            // (every thread has read the previous digit's fields, which the
            // zeroing does not touch; the histogram was last read before the
            // previous barrier)
            for (int b = tid; b < kRadixBins; b += NT) sh.hist[b] = 0u;
            if (tid == 0) sh.ncand = 0u;
            __syncthreads();
            // wave-uniform loop over the keys (or candidates), U x 64 per step
            const int nscan = ncand >= 0 ? ncand : N;
            for (int base = wid * kWave; base < nscan; base += U * NT) {
                uint64_t x[U];
                // clamped indices: every load is issued before any is used
                if (ncand >= 0) {
#pragma unroll
                    for (int u = 0; u < U; ++u) x[u] = cand[min(base + u * NT + lane, nscan - 1)];
                } else {
#pragma unroll
                    for (int u = 0; u < U; ++u) x[u] = key_at(min(base + u * NT + lane, N - 1)) - lo;
                }
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    // the first pass (no digit fixed yet) takes every key
                    const bool match = base + u * NT + lane < nscan &&
                                       (first || (bits >= 64 ? 0ull : (x[u] >> bits)) == prefix);
                    if (match) atomicAdd(&sh.hist[(x[u] >> shift) & mask], 1u);
                    if (collect) {
                        const uint64_t m = __ballot(match);
                        if (m) {
                            uint32_t at = 0;
                            if (lane == 0) at = atomicAdd(&sh.ncand, (uint32_t)__popcll(m));
                            at = (uint32_t)__shfl((int)at, 0);
                            if (match) cand[at + lanes_below(m)] = x[u];
                        }
                    }
                }
            }
            __syncthreads();
            if (collect) ncand = (int)sh.ncand;
        }
        built = false;
        // the digit of rank `rank`, found by wavefront 0 alone (lane l sums
        // bins [32 l, 32 l + 32) with eight 16-byte reads, taken in a rotated
        // order so that the lanes served together hit different banks; a
        // wavefront scan; the lane holding the rank walks its bins), so the
        // other wavefronts wait at one barrier
        if (wid == 0) {
            constexpr int BPL = kRadixBins / kWave;
            constexpr int VPL = BPL / 4;
            const post_u32x4* hv = reinterpret_cast<const post_u32x4*>(sh.hist);
            uint32_t local = 0;
#pragma unroll
            for (int j = 0; j < VPL; ++j) {
                const post_u32x4 q = hv[lane * VPL + ((j + lane + (lane >> 3)) & (VPL - 1))];
                local += (q.x + q.y) + (q.z + q.w);
            }
            const uint32_t incl = wave_incl_scan(local);
            // the lane whose run of bins holds the rank; then its BPL bins, one
            // per lane, scanned again to find the bin
            const uint64_t hit = __ballot(incl - local <= rank && rank < incl);
            const int owner = (int)__builtin_ctzll(hit | (1ull << 63));
            const uint32_t ex = (uint32_t)__builtin_amdgcn_readlane((int)(incl - local), owner);
            const uint32_t h = lane < BPL ? sh.hist[owner * BPL + lane] : 0u;
            const uint32_t hin = wave_incl_scan(h);
            const uint64_t at = __ballot(lane < BPL && rank < ex + hin);
            const int j = (int)__builtin_ctzll(at | (1ull << 63));
            if (lane == j) {
                sh.digit = (uint32_t)(owner * BPL + j);
                sh.below = ex + hin - h;
                sh.in_bin = h;
            }
            if (lane == 0) sh.ncopy = 0u;  // for a candidate copy that follows
        }
        __syncthreads();
        const uint32_t dg = sh.digit, bl = sh.below;
        in_range = sh.in_bin;
        below += bl;
        rank -= bl;
        prefix = (prefix << db) | dg;
        bits = shift;
    }
    const uint64_t vstar = lo + prefix;        // key of rank k-1
    const uint32_t ties = (uint32_t)k - below; // keys equal to vstar that are kept, lowest index first

    // counts of keys below and equal to vstar before this block's slice (the
    // prefix [0, s0) split evenly over the wavefronts), and in each
    // wavefront's contiguous range of the slice
    const int pw = (((s0 + kW - 1) / kW) + kWave - 1) / kWave * kWave;
    const int per = ((((s1 - s0) + kW - 1) / kW) + kWave - 1) / kWave * kWave;
    const int p0 = min(s0, wid * pw), p1 = min(s0, p0 + pw);
    const int b0 = min(s1, s0 + wid * per), b1 = min(s1, b0 + per);
    uint32_t plt = 0, peq = 0, nlt = 0, neq = 0;
    for (int base = p0; base < p1; base += U * kWave) {
        uint64_t kv[U];
#pragma unroll
        for (int u = 0; u < U; ++u) kv[u] = key_at(min(base + u * kWave + lane, p1 - 1));
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const bool v = base + u * kWave + lane < p1;
            plt += (uint32_t)__popcll(__ballot(v && kv[u] < vstar));
            peq += (uint32_t)__popcll(__ballot(v && kv[u] == vstar));
        }
    }
    for (int base = b0; base < b1; base += U * kWave) {
        uint64_t kv[U];
#pragma unroll
        for (int u = 0; u < U; ++u) kv[u] = key_at(min(base + u * kWave + lane, b1 - 1));
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const bool v = base + u * kWave + lane < b1;
            nlt += (uint32_t)__popcll(__ballot(v && kv[u] < vstar));
            neq += (uint32_t)__popcll(__ballot(v && kv[u] == vstar));
        }
    }
    if (lane == 0) {
        sh.wcnt[wid][0] = nlt;
        sh.wcnt[wid][1] = neq;
        sh.wcnt[wid][2] = plt;
        sh.wcnt[wid][3] = peq;
    }
    __syncthreads();
    uint32_t lt_before = 0, eq_before = 0;
#pragma unroll
    for (int q = 0; q < kW; ++q) {
        lt_before += sh.wcnt[q][2] + (q < wid ? sh.wcnt[q][0] : 0u);
        eq_before += sh.wcnt[q][3] + (q < wid ? sh.wcnt[q][1] : 0u);
    }
    uint32_t eq_run = eq_before;
    uint32_t kept_run = lt_before + min(eq_before, ties);
    for (int base = b0; base < b1; base += U * kWave) {
        uint64_t kv[U];
#pragma unroll
        for (int u = 0; u < U; ++u) kv[u] = key_at(min(base + u * kWave + lane, b1 - 1));
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int i = base + u * kWave + lane;
            const bool v = i < b1;
            const bool isl = v && kv[u] < vstar;
            const bool ise = v && kv[u] == vstar;
            const uint64_t me = __ballot(ise);
            const bool kp = isl || (ise && eq_run + lanes_below(me) < ties);
            const uint64_t mk = __ballot(kp);
            if (v && a.sel.keep) a.sel.keep[off + i] = kp ? 1 : 0;
            if (kp) a.sel.kept_idx[ioff + (int)(kept_run + lanes_below(mk))] = iadd + i;
            eq_run += (uint32_t)__popcll(me);
            kept_run += (uint32_t)__popcll(mk);
        }
    }
}

// Top-k of one selection: the k smallest (key, index) pairs of a segment, or
// of one frame of a clip under the per-frame scope, kept indices ascending
// (Sec. 4.1.1 pruning, k from the Eq. 11 floor or a fixed ratio). Keys are
// staged in LDS when they fit (keys_cap entries), then an MSD radix select
// finds the key of rank k-1 and each wavefront compacts a contiguous index
// range of the block's slice with ballot/mbcnt. A selection split over
// nparts blocks has every block find the same key from all of the keys and
// write its own slice (and its share of the -1 tail). Frame f of a clip
// keeping k_f per frame writes its kept indices at positions f k_f.. of the
// segment's range and its share, P - k_f entries, of the -1 tail after the
// T k_f kept ones.
template <int NT>
__device__ void role_select(const PostArgs& a, int unit, PostShared<NT>& sh, uint64_t* keys, int keys_cap)
{
    const Tables& t = a.t;
    const SelUnit su = t.sel_unit[unit];
    const int N = su.N, f = su.frame, tid = threadIdx.x, lane = tid & (kWave - 1);
    const bool framed = f >= 0;
    int k = su.kfix;
    if (k < 0) {
        float mas;
        if (a.mas_in) {
            mas = a.mas_in[su.request * kNumMod + su.modality];
        } else {
            RMAgg g[kNumMod];
            rm_aggregate_all(t, su.request, sh, g);
            MasTerms o[kNumMod];
            bool pres[kNumMod];
            request_terms(t, su.request, g, o, pres);
            mas = 0.0f;
#pragma unroll
            for (int m = 0; m < kNumMod; ++m)
                if (m == su.modality) mas = (float)o[m].mas;
        }
        k = guided_keep_count(mas, N);
    }
    if (tid == 0 && f <= 0 && su.part == 0) a.sel.kept_count[su.seg] = k * su.units;
    const int off = su.off;                                     // keys and keep flags
    const int ioff = su.seg_off + (framed ? f * k : 0);         // kept indices
    const int iadd = framed ? f * N : 0;                        // local index of the selection's first token
    const int fill = su.seg_off + su.units * k + (framed ? f : 0) * (N - k);
    {
        const int tail = N - k, share = (tail + su.nparts - 1) / su.nparts;
        const int t0 = min(tail, su.part * share), t1 = min(tail, t0 + share);
        for (int i = t0 + tid; i < t1; i += NT) a.sel.kept_idx[fill + i] = -1;
    }
    if (N == 0) return;
    // this block's slice of the tokens (whole wavefront chunks)
    const int slice = ((N + su.nparts - 1) / su.nparts + kWave - 1) / kWave * kWave;
    const int s0 = min(N, su.part * slice), s1 = min(N, s0 + slice);
    if (k == 0 || k == N) {
        for (int i = s0 + tid; i < s1; i += NT) {
            if (a.sel.keep) a.sel.keep[off + i] = k == N ? 1 : 0;
            if (k == N) a.sel.kept_idx[ioff + i] = iadd + i;
        }
        return;
    }
    const int kind = su.kind;
    const uint64_t Ms = su.Ms, Mt = su.Mt;
    const uint32_t E = su.E;
    const uint32_t* z = a.z + off;
    const uint32_t* d = a.d ? a.d + off : nullptr;
    const float* imp = kind == kKeyImp ? t.proj + off : nullptr;  // learned run: Eq. 3 importance
    const bool in_lds = N <= keys_cap;

    // keys (staged in LDS) in [0, kmax], counted in the first digit's histogram
    const uint64_t lo = 0ull, hi = su.kmax;
    const int bits = hi > 0 ? 64 - __clzll((long long)hi) : 0;
    const int shift0 = bits > kRadixBits ? bits - kRadixBits : 0;
    switch (kind) {
    case kKeyZ: stage_keys<NT, kKeyZ>(z, d, imp, N, Ms, Mt, E, in_lds, keys, sh.hist, shift0, bits > 0); break;
    case kKeyE: stage_keys<NT, kKeyE>(z, d, imp, N, Ms, Mt, E, in_lds, keys, sh.hist, shift0, bits > 0); break;
    case kKeyFull: stage_keys<NT, kKeyFull>(z, d, imp, N, Ms, Mt, E, in_lds, keys, sh.hist, shift0, bits > 0); break;
    case kKeyImp: stage_keys<NT, kKeyImp>(z, d, imp, N, Ms, Mt, E, in_lds, keys, sh.hist, shift0, bits > 0); break;
    default: stage_keys<NT, kKeyZero>(z, d, imp, N, Ms, Mt, E, in_lds, keys, sh.hist, shift0, false); break;
    }
    __syncthreads();

    const KeySrc src{keys, z, d, imp, kind, Ms, Mt, E};
    uint64_t* cand = keys + keys_cap;
    if (in_lds)
        select_and_compact<NT, true>(a, sh, src, cand, cand_cap_for(keys_cap), N, k, off, ioff, iadd, lo, hi, s0, s1, true);
    else
        select_and_compact<NT, false>(a, sh, src, cand, cand_cap_for(keys_cap), N, k, off, ioff, iadd, lo, hi, s0, s1, true);
}

// LR: a learned call (request role with head counts, descriptors and the
// relevance MLP; no selection); a separate instance, so that the plain
// kernel keeps its registers.
template <int NT, bool LR>
__global__ __launch_bounds__(NT) void k_post(PostArgs a)
{
    __shared__ PostShared<NT> sh;
    extern __shared__ uint64_t keys[];
    // selection blocks first: they are the longest and are dispatched first
    int b = blockIdx.x;
    if constexpr (!LR) {
        if (b < a.n_sel_blocks) {
            role_select(a, b, sh, keys, a.keys_cap);
            return;
        }
        b -= a.n_sel_blocks;
    }
    if (b < a.n_req_blocks) {
        if constexpr (LR) role_request_learned<NT>(a, b, sh);
        else role_request(a, b, sh);
        return;
    }
    b -= a.n_req_blocks;
    if (b < a.n_frame_blocks) role_frame(a, b, sh);
}

// ---------------------------------------------------------------- k_gather

#ifndef MSAO_GATHER_UNITS
#define MSAO_GATHER_UNITS 8  // 16-byte units per lane in flight per gather batch
#endif

// Kept rows [j0, j0 + kGatherRows) of a segment whose rows span NU units.
// The kept indices arrive in one vector load (lane i holds row j0 + i) and are
// read out per row, so every row's load is issued without waiting on another;
// out-of-range lanes are dropped by the store's buffer resource.
template <int NU>
__device__ __forceinline__ void gather_rows(const GatherArgs& a, const DevSeg& sg, int j0, int cnt, int lane)
{
    constexpr int RB0 = NU >= MSAO_GATHER_UNITS ? 1 : MSAO_GATHER_UNITS / NU;
    constexpr int RB = RB0 < kGatherRows ? RB0 : kGatherRows;
    const int rb = sg.nchunk * 16;
    const int voff = lane * 16;
    const int nrows = min(kGatherRows, cnt - j0);
    const int mine = lane < nrows ? a.kept_idx[sg.tok_off + j0 + lane] : -1;
    for (int i0 = 0; i0 < nrows; i0 += RB) {
        vec4 v[RB][NU];
        int src[RB];
#pragma unroll
        for (int i = 0; i < RB; ++i) {
            src[i] = i0 + i < nrows ? __builtin_amdgcn_readlane(mine, i0 + i) : -1;
            const bool ok = src[i] >= 0 && src[i] < sg.n_tok;
            const rsrc_t rs = make_rsrc(sg.data + (ok ? (int64_t)src[i] * sg.stride_bytes : 0), ok ? rb : 0);
#pragma unroll
            for (int u = 0; u < NU; ++u) v[i][u] = bload_gather(rs, voff + u * 1024);
        }
#pragma unroll
        for (int i = 0; i < RB; ++i) {
            if (src[i] < 0 || src[i] >= sg.n_tok) continue;
            const rsrc_t rd = make_rsrc(a.out + sg.out_off + (int64_t)(j0 + i0 + i) * rb, rb);
#pragma unroll
            for (int u = 0; u < NU; ++u) bstore(v[i][u], rd, voff + u * 1024);
        }
    }
}

__device__ void gather_rows_generic(const GatherArgs& a, const DevSeg& sg, int j0, int cnt, int lane)
{
    const int rb = sg.nchunk * 16;
    const int nu = (sg.nchunk + kWave - 1) / kWave;
    const int j1 = min(cnt, j0 + kGatherRows);
    for (int j = j0; j < j1; ++j) {
        const int src = uniform(a.kept_idx[sg.tok_off + j]);
        if (src < 0 || src >= sg.n_tok) continue;
        const rsrc_t rs = make_rsrc(sg.data + (int64_t)src * sg.stride_bytes, rb);
        const rsrc_t rd = make_rsrc(a.out + sg.out_off + (int64_t)j * rb, rb);
        for (int u0 = 0; u0 < nu; u0 += 8) {
            vec4 v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = bload_gather(rs, ((u0 + u) * kWave + lane) * 16);
#pragma unroll
            for (int u = 0; u < 8; ++u) bstore(v[u], rd, ((u0 + u) * kWave + lane) * 16);
        }
    }
}

template <int NT>
__global__ __launch_bounds__(NT) void k_gather(GatherArgs a)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int w = uniform(blockIdx.x * (NT / kWave) + (threadIdx.x >> 6));
    if (w >= a.t.n_gwi) return;
    const int s = uniform(a.t.gi_seg[w]);
    const DevSeg sg = a.t.seg[s];
    int cnt = uniform(a.kept_count[s]);
    cnt = min(cnt, min(sg.cap, sg.n_tok));
    const int j0 = (w - sg.g_begin) * kGatherRows;
    if (j0 >= cnt) return;
    switch ((sg.nchunk + kWave - 1) / kWave) {
    case 1: gather_rows<1>(a, sg, j0, cnt, lane); break;
    case 2: gather_rows<2>(a, sg, j0, cnt, lane); break;
    case 3: gather_rows<3>(a, sg, j0, cnt, lane); break;
    case 4: gather_rows<4>(a, sg, j0, cnt, lane); break;
    case 5: gather_rows<5>(a, sg, j0, cnt, lane); break;
    case 6: gather_rows<6>(a, sg, j0, cnt, lane); break;
    case 7: gather_rows<7>(a, sg, j0, cnt, lane); break;
    case 8: gather_rows<8>(a, sg, j0, cnt, lane); break;
    default: gather_rows_generic(a, sg, j0, cnt, lane); break;
    }
}

}  // namespace

// With ev0/ev1 (profiling), the launch records them at the kernel's own start
// and end, so their span is the kernel's execution time.
// ---------------------------------------------------------------- k_head

// u[r][j] = b1[j] + W1[j][:prompt_dim] . p_r for kMlpGroup requests per
// wavefront: the lanes stride over the row (coalesced loads of W1 and of
// the prompts, 8 strides issued before they are used, since each load is
// an L2 round trip), then one wavefront sum per request.
__device__ __forceinline__ void prompt_product(const HeadArgs& a, int blk)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int g = blk * (kHeadBlock / kWave) + (threadIdx.x >> 6);
    const int R = a.t.R, H = a.mlp.hidden, P = a.mlp.prompt_dim;
    const int ngr = (R + kMlpGroup - 1) / kMlpGroup;
    if (g >= H * ngr) return;  // wave-uniform
    const int j = g / ngr, r0 = (g % ngr) * kMlpGroup, nr = min(kMlpGroup, R - r0);
    const float* wrow = a.mlp.w1 + (int64_t)j * (P + kDesc);
    float acc[kMlpGroup];
#pragma unroll
    for (int q = 0; q < kMlpGroup; ++q) acc[q] = 0.0f;
    constexpr int U = 8;
    for (int k0 = lane; k0 < P; k0 += kWave * U) {
        float wk[U], pv[U][kMlpGroup];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int k = k0 + u * kWave;
            wk[u] = k < P ? wrow[k] : 0.0f;
#pragma unroll
            for (int q = 0; q < kMlpGroup; ++q)
                pv[u][q] = (k < P && q < nr) ? a.mlp.prompt[(int64_t)(r0 + q) * P + k] : 0.0f;
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int q = 0; q < kMlpGroup; ++q) acc[q] = fmaf(wk[u], pv[u][q], acc[q]);
    }
    const float b = a.mlp.b1[j];
#pragma unroll
    for (int q = 0; q < kMlpGroup; ++q) {
        const float s = wave_sum(acc[q]);
        if (lane == 0 && q < nr) a.u[(int64_t)(r0 + q) * H + j] = s + b;
    }
}

// Eq. 3 with a learned head for one frame of a segment (P tokens on an
// H x W grid, token q at row q / W, column q % W): importance
// M = sigmoid(mean of the projections over the pool x pool window cut to the
// grid + b), which is Conv1x1(AvgPool(F)) since the 1x1 convolution is
// linear; then the number of tokens with M < tau_s (Eq. 4).
// Blocks past the head blocks compute the MLP's prompt product.
__global__ __launch_bounds__(kHeadBlock) void k_head(HeadArgs a)
{
    extern __shared__ float ys[];
    __shared__ uint64_t cnt[kHeadBlock / kWave];
    const Tables& t = a.t;
    const int hb = blockIdx.x;
    if (hb >= t.n_hb) {
        prompt_product(a, hb - t.n_hb);
        return;
    }
    const DevSeg sg = t.seg[t.hb_seg[hb]];
    const int P = sg.P;
    const int base = sg.tok_off + (hb - sg.hb_begin) * P;
    for (int q = threadIdx.x; q < P; q += kHeadBlock) ys[q] = t.proj[base + q];
    __syncthreads();
    const int W = sg.grid_w > 0 ? sg.grid_w : P, H = P / W, r = (sg.pool - 1) / 2;
    uint64_t c = 0;
    for (int q = threadIdx.x; q < P; q += kHeadBlock) {
        const int i = q / W, j = q % W;
        const int i0 = max(0, i - r), i1 = min(H - 1, i + r), j0 = max(0, j - r), j1 = min(W - 1, j + r);
        float sum = 0.0f;
        for (int ii = i0; ii <= i1; ++ii)
            for (int jj = j0; jj <= j1; ++jj) sum += ys[ii * W + jj];
        const float v = sum / (float)((i1 - i0 + 1) * (j1 - j0 + 1)) + sg.head_b;
        const float M = 1.0f / (1.0f + expf(-v));
        if (a.importance) a.importance[base + q] = M;
        t.proj[base + q] = M;  // the frame's projections are in LDS: the slot now holds M for a selection
        c += M < t.tau_s ? 1u : 0u;
    }
    c = wave_sum_u64(c);
    if ((threadIdx.x & (kWave - 1)) == 0) cnt[threadIdx.x >> 6] = c;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint64_t total = 0;
#pragma unroll
        for (int w = 0; w < kHeadBlock / kWave; ++w) total += cnt[w];
        t.head_count[hb] = (uint32_t)total;
    }
}

template <typename Args>
static int launch(void (*kernel)(Args), dim3 grid, dim3 block, size_t lds, void* stream, const Args& a,
                  void* ev0, void* ev1)
{
    if (ev0 || ev1)
        hipExtLaunchKernelGGL(kernel, grid, block, lds, (hipStream_t)stream, (hipEvent_t)ev0, (hipEvent_t)ev1, 0, a);
    else
        hipLaunchKernelGGL(kernel, grid, block, lds, (hipStream_t)stream, a);
    return (int)hipGetLastError();
}

// k_pair's clips (work items [0, n_wi_pair)), then k_score for the rest:
// ev0 is recorded at the first launch's start, ev1 at the last one's end.
int launch_score(const ScoreArgs& a, void* stream, void* ev0, void* ev1)
{
    if (a.t.n_wi_score <= 0) return kNoLaunch;
    const int waves = kScoreBlock / kWave;
    if (a.learned) {
        if (!a.t.partial_x || !a.t.proj || a.t.n_wi_pair != 0) return (int)hipErrorInvalidValue;  // a learned plan's tables
        const unsigned grid = (unsigned)((a.t.n_wi_score + waves - 1) / waves);
        return launch(k_score<true>, dim3(grid), dim3(kScoreBlock), 0, stream, a, ev0, ev1);
    }
    const int npair = a.t.n_wi_pair;
    if (npair < 0 || npair % kPairWaves != 0 || npair > a.t.n_wi_score) return (int)hipErrorInvalidValue;
    const bool rest = a.t.n_wi_score > npair;
    if (npair > 0) {
        const int rc = launch(k_pair, dim3((unsigned)(npair / kPairWaves)), dim3(kPairWaves * kWave), 0, stream, a, ev0,
                              rest ? nullptr : ev1);
        if (rc != 0 || !rest) return rc;
    }
    ScoreArgs b = a;
    b.wi_first = npair;
    const unsigned grid = (unsigned)((a.t.n_wi_score - npair + waves - 1) / waves);
    return launch(k_score<false>, dim3(grid), dim3(kScoreBlock), 0, stream, b, npair > 0 ? nullptr : ev0, ev1);
}

template <int NT, bool LR>
static int launch_post_nt(const PostArgs& a, int blocks, size_t lds, void* stream, void* ev0, void* ev1)
{
    if (lds > 65536) {
        const hipError_t e =
            hipFuncSetAttribute((const void*)k_post<NT, LR>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return (int)e;
    }
    return launch(k_post<NT, LR>, dim3((unsigned)blocks), dim3(NT), lds, stream, a, ev0, ev1);
}

// Launches with a selection of kPostBigSegment tokens or more (the host's
// big_block; the threshold can be changed at context creation) take
// 1024-thread blocks (their loops are latency-bound with one wavefront per
// SIMD); otherwise kPostBlock threads, which leave room for the scoring of
// other batches in flight.
int launch_post(const PostArgs& a, void* stream, void* ev0, void* ev1)
{
    const int blocks = a.n_req_blocks + a.n_frame_blocks + a.n_sel_blocks;
    if (blocks <= 0) return kNoLaunch;
    const size_t lds = (size_t)(a.keys_cap + cand_cap_for(a.keys_cap)) * sizeof(uint64_t);
    if (a.learned && (!a.t.partial_x || !a.t.head_count || (a.use_mlp && !a.mlp_u))) return (int)hipErrorInvalidValue;
    if (a.learned) return launch_post_nt<kPostBlock, true>(a, a.n_req_blocks + a.n_frame_blocks, lds, stream, ev0, ev1);
    if (a.n_sel_blocks > 0 && a.big_block)
        return launch_post_nt<1024, false>(a, blocks, lds, stream, ev0, ev1);
    return launch_post_nt<kPostBlock, false>(a, blocks, lds, stream, ev0, ev1);
}

int launch_head(const HeadArgs& a, void* stream, void* ev0, void* ev1)
{
    const int blocks = a.t.n_hb + a.n_mlp_blocks;
    if (blocks <= 0) return kNoLaunch;
    if (a.t.n_hb > 0 && (!a.t.proj || !a.t.head_count || a.max_p < 1 || a.max_p > kMaxHeadFrame))
        return (int)hipErrorInvalidValue;
    if (a.n_mlp_blocks > 0 && (!a.u || !a.mlp.w1 || !a.mlp.b1 || a.mlp.hidden < 1 || a.mlp.hidden > kMaxMlpHidden ||
                               (a.mlp.prompt_dim > 0 && !a.mlp.prompt)))
        return (int)hipErrorInvalidValue;
    const size_t lds = a.t.n_hb > 0 ? (size_t)a.max_p * sizeof(float) : 0;
    if (lds > 65536) {
        const hipError_t e = hipFuncSetAttribute((const void*)k_head, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return (int)e;
    }
    return launch(k_head, dim3((unsigned)blocks), dim3(kHeadBlock), lds, stream, a, ev0, ev1);
}

int launch_gather(const GatherArgs& a, void* stream, void* ev0, void* ev1)
{
    if (a.t.n_gwi <= 0) return kNoLaunch;
    if (a.t.n_gwi <= kGatherFewItems) {
        constexpr int waves = kGatherBlockFew / kWave;
        const unsigned grid = (unsigned)((a.t.n_gwi + waves - 1) / waves);
        return launch(k_gather<kGatherBlockFew>, dim3(grid), dim3(kGatherBlockFew), 0, stream, a, ev0, ev1);
    }
    constexpr int waves = kGatherBlock / kWave;
    const unsigned grid = (unsigned)((a.t.n_gwi + waves - 1) / waves);
    return launch(k_gather<kGatherBlock>, dim3(grid), dim3(kGatherBlock), 0, stream, a, ev0, ev1);
}

}  // namespace msao
