// msao_kernels.hip -- gfx950 (CDNA4) kernels of MSAO's fine-grained sparsity
// analysis (Sec. 4.1) and of the MAS-guided token selection it drives.
//
// The path is HBM-bandwidth bound: every input byte is read once with 128-bit
// loads, no step is a dense contraction (no MFMA). Three launches:
//   k_score  one wavefront per work item (a run of rows, or one patch's run
//            of frames). Per token: activity count by ballot + scalar
//            popcount, L1/L2 by DPP wave reductions; for video the previous
//            frame's values and activity masks stay in registers, so the
//            temporal term (Eq. 5) costs no extra HBM traffic. Per work item
//            it writes integer partials (sparse-token count, sum of d), so no
//            atomics and no zeroing are needed and results are bit-stable.
//   k_post   block roles: one block per request (integer aggregation, modal
//            softmax, Eq. 4 ratio, Eq. 7 MAS), one per video frame (Eq. 5
//            per frame), one per segment (top-k by LDS radix select over
//            exact integer keys, ties by index, block-scan compaction).
//   k_gather one wavefront per few kept rows: packed bitwise copy.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "msao_internal.h"

namespace msao {
namespace {

constexpr int kWave = 64;

__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

template <int CTRL>
__device__ __forceinline__ float dpp_f(float v)
{
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

// Sum over the 64 lanes; the result is the same in every lane. Fixed order,
// so it is bit-reproducible. quad_perm [1,0,3,2], quad_perm [2,3,0,1],
// row_half_mirror and row_mirror give each 16-lane row its sum; the four
// row sums are then read out and added.
__device__ __forceinline__ float wave_sum(float v)
{
    v += dpp_f<0xB1>(v);
    v += dpp_f<0x4E>(v);
    v += dpp_f<0x141>(v);
    v += dpp_f<0x140>(v);
    const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
    const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
    const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
    const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
    return (r0 + r1) + (r2 + r3);
}

__device__ __forceinline__ uint4 ld16(const uint8_t* p) { return *reinterpret_cast<const uint4*>(p); }

// Widening of one 16-byte chunk to floats (exact).
template <int DT> struct Lane;
template <> struct Lane<kBF16> {
    static constexpr int EPC = 8;
    __device__ static __forceinline__ void widen(const uint4& v, float* x)
    {
        x[0] = __uint_as_float(v.x << 16); x[1] = __uint_as_float(v.x & 0xFFFF0000u);
        x[2] = __uint_as_float(v.y << 16); x[3] = __uint_as_float(v.y & 0xFFFF0000u);
        x[4] = __uint_as_float(v.z << 16); x[5] = __uint_as_float(v.z & 0xFFFF0000u);
        x[6] = __uint_as_float(v.w << 16); x[7] = __uint_as_float(v.w & 0xFFFF0000u);
    }
};
template <> struct Lane<kF32> {
    static constexpr int EPC = 4;
    __device__ static __forceinline__ void widen(const uint4& v, float* x)
    {
        x[0] = __uint_as_float(v.x); x[1] = __uint_as_float(v.y);
        x[2] = __uint_as_float(v.z); x[3] = __uint_as_float(v.w);
    }
};

// Active iff NOT(|x| <= tau): NaN is active, -0 is not.
__device__ __forceinline__ bool active(float x, float tau) { return !(fabsf(x) <= tau); }

// Largest s in [0, n) with prefix[s] <= w (prefix[n] is the total, > w).
__device__ __forceinline__ int find_seg(const int32_t* __restrict__ prefix, int n, int w)
{
    int lo = 0, hi = n;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (prefix[mid] <= w) lo = mid; else hi = mid;
    }
    return lo;
}

// ---------------------------------------------------------------- k_score

struct TokStat {
    uint32_t act;   // active channels
    uint32_t d;     // Hamming distance to the previous frame's activity bits
    float l1, l2, res;
};

__device__ __forceinline__ void emit_token(const TokenOut& o, const DevSeg& sg, int row, int lane,
                                           const TokStat& s, bool temporal, int mode)
{
    if (lane != 0) return;
    const int g = sg.tok_off + row;
    const uint32_t z = (uint32_t)sg.C - s.act;
    if (mode == kModeScore) {
        if (o.z) o.z[g] = z;
        if (o.l1) o.l1[g] = s.l1;
        if (o.l2) o.l2[g] = s.l2;
        if (o.info) {
            float red = sg.lam_s * (float)z;
            if (temporal) red += sg.lam_t * (float)((uint32_t)sg.C - s.d);
            o.info[g] = 1.0f - red / (float)sg.C;
        }
    }
    if (o.d) o.d[g] = temporal ? s.d : 0u;
    if (o.res) o.res[g] = temporal ? s.res : 0.0f;
}

// Rows [r0, r1) of a non-temporal segment whose rows span NU 1-KiB units
// (64 lanes x 16 B). Several short rows are loaded before any is reduced so
// that each wavefront keeps about 4 KiB in flight.
template <int DT, int NU>
__device__ __forceinline__ void score_rows(const ScoreArgs& a, const DevSeg& sg, int r0, int r1,
                                           int lane, uint32_t& nsp)
{
    using L = Lane<DT>;
    constexpr int EPC = L::EPC;
    constexpr int RPI = NU >= 4 ? 1 : 4 / NU;
    const float tau = a.t.tau;
    for (int r = r0; r < r1; r += RPI) {
        uint4 v[RPI][NU];
#pragma unroll
        for (int i = 0; i < RPI; ++i) {
            const uint8_t* row = sg.data + (int64_t)(r + i) * sg.stride_bytes;
#pragma unroll
            for (int u = 0; u < NU; ++u) {
                const int c = u * kWave + lane;
                v[i][u] = make_uint4(0u, 0u, 0u, 0u);
                if (r + i < r1 && c < sg.nchunk) v[i][u] = ld16(row + (int64_t)c * 16);
            }
        }
#pragma unroll
        for (int i = 0; i < RPI; ++i) {
            if (r + i >= r1) break;
            TokStat s{0u, 0u, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int u = 0; u < NU; ++u) {
                float x[EPC];
                L::widen(v[i][u], x);
#pragma unroll
                for (int e = 0; e < EPC; ++e) {
                    s.act += (uint32_t)__popcll(__ballot(active(x[e], tau)));
                    s.l1 += fabsf(x[e]);
                    s.l2 = fmaf(x[e], x[e], s.l2);
                }
            }
            s.l1 = wave_sum(s.l1);
            s.l2 = wave_sum(s.l2);
            emit_token(a.tok, sg, r + i, lane, s, false, kModeScore);
            nsp += s.act < (uint32_t)sg.A_s;
        }
    }
}

// Any row width: units processed in blocks of 4.
template <int DT>
__device__ void score_rows_generic(const ScoreArgs& a, const DevSeg& sg, int r0, int r1, int lane,
                                   uint32_t& nsp)
{
    using L = Lane<DT>;
    constexpr int EPC = L::EPC;
    const float tau = a.t.tau;
    const int nu = (sg.nchunk + kWave - 1) / kWave;
    for (int r = r0; r < r1; ++r) {
        const uint8_t* row = sg.data + (int64_t)r * sg.stride_bytes;
        TokStat s{0u, 0u, 0.0f, 0.0f, 0.0f};
        for (int u0 = 0; u0 < nu; u0 += 4) {
            uint4 v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int c = (u0 + u) * kWave + lane;
                v[u] = make_uint4(0u, 0u, 0u, 0u);
                if (c < sg.nchunk) v[u] = ld16(row + (int64_t)c * 16);
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                float x[EPC];
                L::widen(v[u], x);
#pragma unroll
                for (int e = 0; e < EPC; ++e) {
                    s.act += (uint32_t)__popcll(__ballot(active(x[e], tau)));
                    s.l1 += fabsf(x[e]);
                    s.l2 = fmaf(x[e], x[e], s.l2);
                }
            }
        }
        s.l1 = wave_sum(s.l1);
        s.l2 = wave_sum(s.l2);
        emit_token(a.tok, sg, r, lane, s, false, kModeScore);
        nsp += s.act < (uint32_t)sg.A_s;
    }
}

// Frames [t0, t1) of patch p of a temporal segment (rows t*P + p). The
// previous frame's values and activity ballots stay in registers; frame t+1
// is loaded before frame t is reduced. A run that starts after frame 0 first
// loads frame t0-1 (its halo).
template <int DT, int NU>
__device__ __forceinline__ void score_chain(const ScoreArgs& a, const DevSeg& sg, int p, int t0, int t1,
                                            int lane, uint32_t& nsp, uint64_t& dsum)
{
    using L = Lane<DT>;
    constexpr int EPC = L::EPC;
    constexpr int NE = NU * EPC;
    const float tau = a.t.tau;
    const int64_t fstride = (int64_t)sg.P * sg.stride_bytes;
    const uint8_t* base = sg.data + (int64_t)p * sg.stride_bytes;
    float prev[NE];
    uint64_t pmask[NE];
    {
        uint4 v[NU];
#pragma unroll
        for (int u = 0; u < NU; ++u) {
            const int c = u * kWave + lane;
            v[u] = make_uint4(0u, 0u, 0u, 0u);
            if (t0 > 0 && c < sg.nchunk) v[u] = ld16(base + (int64_t)(t0 - 1) * fstride + (int64_t)c * 16);
        }
#pragma unroll
        for (int u = 0; u < NU; ++u) {
            L::widen(v[u], &prev[u * EPC]);
#pragma unroll
            for (int e = 0; e < EPC; ++e) pmask[u * EPC + e] = __ballot(active(prev[u * EPC + e], tau));
        }
    }
    uint4 cur[NU];
#pragma unroll
    for (int u = 0; u < NU; ++u) {
        const int c = u * kWave + lane;
        cur[u] = make_uint4(0u, 0u, 0u, 0u);
        if (c < sg.nchunk) cur[u] = ld16(base + (int64_t)t0 * fstride + (int64_t)c * 16);
    }
    for (int t = t0; t < t1; ++t) {
        uint4 nxt[NU];
#pragma unroll
        for (int u = 0; u < NU; ++u) {
            const int c = u * kWave + lane;
            nxt[u] = make_uint4(0u, 0u, 0u, 0u);
            if (t + 1 < t1 && c < sg.nchunk) nxt[u] = ld16(base + (int64_t)(t + 1) * fstride + (int64_t)c * 16);
        }
        TokStat s{0u, 0u, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int u = 0; u < NU; ++u) {
            float x[EPC];
            L::widen(cur[u], x);
#pragma unroll
            for (int e = 0; e < EPC; ++e) {
                const int k = u * EPC + e;
                const uint64_t m = __ballot(active(x[e], tau));
                s.act += (uint32_t)__popcll(m);
                s.d += (uint32_t)__popcll(m ^ pmask[k]);
                pmask[k] = m;
                s.l1 += fabsf(x[e]);
                s.l2 = fmaf(x[e], x[e], s.l2);
                const float df = x[e] - prev[k];
                s.res = fmaf(df, df, s.res);
                prev[k] = x[e];
            }
        }
        s.l1 = wave_sum(s.l1);
        s.l2 = wave_sum(s.l2);
        s.res = wave_sum(s.res);
        emit_token(a.tok, sg, t * sg.P + p, lane, s, true, a.mode);
        nsp += s.act < (uint32_t)sg.A_s;
        if (t >= 1) dsum += s.d;
#pragma unroll
        for (int u = 0; u < NU; ++u) cur[u] = nxt[u];
    }
}

// Any row width: the previous frame's row is re-read (it was just read by
// this wavefront, so it is normally served by the L2).
template <int DT>
__device__ void score_chain_generic(const ScoreArgs& a, const DevSeg& sg, int p, int t0, int t1, int lane,
                                    uint32_t& nsp, uint64_t& dsum)
{
    using L = Lane<DT>;
    constexpr int EPC = L::EPC;
    const float tau = a.t.tau;
    const int64_t fstride = (int64_t)sg.P * sg.stride_bytes;
    const uint8_t* base = sg.data + (int64_t)p * sg.stride_bytes;
    const int nu = (sg.nchunk + kWave - 1) / kWave;
    for (int t = t0; t < t1; ++t) {
        TokStat s{0u, 0u, 0.0f, 0.0f, 0.0f};
        for (int u0 = 0; u0 < nu; u0 += 2) {
            uint4 v[2], w[2];
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const int c = (u0 + u) * kWave + lane;
                v[u] = make_uint4(0u, 0u, 0u, 0u);
                w[u] = make_uint4(0u, 0u, 0u, 0u);
                if (c < sg.nchunk) {
                    v[u] = ld16(base + (int64_t)t * fstride + (int64_t)c * 16);
                    if (t > 0) w[u] = ld16(base + (int64_t)(t - 1) * fstride + (int64_t)c * 16);
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
        emit_token(a.tok, sg, t * sg.P + p, lane, s, true, a.mode);
        nsp += s.act < (uint32_t)sg.A_s;
        if (t >= 1) dsum += s.d;
    }
}

template <int DT>
__device__ __forceinline__ void dispatch_rows(const ScoreArgs& a, const DevSeg& sg, int r0, int r1, int lane,
                                              uint32_t& nsp)
{
    const int nu = (sg.nchunk + kWave - 1) / kWave;
    switch (nu) {
    case 1: score_rows<DT, 1>(a, sg, r0, r1, lane, nsp); break;
    case 2: score_rows<DT, 2>(a, sg, r0, r1, lane, nsp); break;
    case 3: score_rows<DT, 3>(a, sg, r0, r1, lane, nsp); break;
    case 4: score_rows<DT, 4>(a, sg, r0, r1, lane, nsp); break;
    case 5: score_rows<DT, 5>(a, sg, r0, r1, lane, nsp); break;
    case 6: score_rows<DT, 6>(a, sg, r0, r1, lane, nsp); break;
    case 7: score_rows<DT, 7>(a, sg, r0, r1, lane, nsp); break;
    case 8: score_rows<DT, 8>(a, sg, r0, r1, lane, nsp); break;
    default: score_rows_generic<DT>(a, sg, r0, r1, lane, nsp); break;
    }
}

template <int DT>
__device__ __forceinline__ void dispatch_chain(const ScoreArgs& a, const DevSeg& sg, int p, int t0, int t1,
                                               int lane, uint32_t& nsp, uint64_t& dsum)
{
    const int nu = (sg.nchunk + kWave - 1) / kWave;
    switch (nu) {
    case 1: score_chain<DT, 1>(a, sg, p, t0, t1, lane, nsp, dsum); break;
    case 2: score_chain<DT, 2>(a, sg, p, t0, t1, lane, nsp, dsum); break;
    case 3: score_chain<DT, 3>(a, sg, p, t0, t1, lane, nsp, dsum); break;
    case 4: score_chain<DT, 4>(a, sg, p, t0, t1, lane, nsp, dsum); break;
    default: score_chain_generic<DT>(a, sg, p, t0, t1, lane, nsp, dsum); break;
    }
}

__global__ __launch_bounds__(kScoreBlock) void k_score(ScoreArgs a)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int w = uniform(blockIdx.x * (kScoreBlock / kWave) + (threadIdx.x >> 6));
    if (w >= a.t.n_wi) return;
    const int s = find_seg(a.t.seg_wi, a.t.n, w);
    const DevSeg sg = a.t.seg[s];
    const int q = w - sg.wi_begin;
    uint32_t nsp = 0;
    uint64_t dsum = 0;
    if (sg.temporal) {
        const int p = q % sg.P;
        const int t0 = (q / sg.P) * sg.per_item;
        const int t1 = min(sg.T, t0 + sg.per_item);
        if (sg.dtype == kBF16) dispatch_chain<kBF16>(a, sg, p, t0, t1, lane, nsp, dsum);
        else dispatch_chain<kF32>(a, sg, p, t0, t1, lane, nsp, dsum);
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
            dispatch_rows<kBF16>(a, sg, r0, r1, lane, nsp);
        } else {
            dispatch_rows<kF32>(a, sg, r0, r1, lane, nsp);
        }
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

// Block-wide sum of a 64-bit integer (exact, so the order does not matter).
__device__ __forceinline__ uint64_t block_sum_u64(uint64_t v, unsigned long long* sh)
{
    __syncthreads();
    if (threadIdx.x == 0) *sh = 0ull;
    __syncthreads();
    if (v) atomicAdd(sh, (unsigned long long)v);
    __syncthreads();
    return (uint64_t)*sh;
}

// Block-wide exclusive scan of 32-bit counts in thread order; *total gets the sum.
__device__ __forceinline__ uint32_t block_exscan(uint32_t v, uint32_t* sh, uint32_t* total)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int wid = threadIdx.x >> 6;
    constexpr int nw = kPostBlock / kWave;
    uint32_t x = v;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const uint32_t y = __shfl_up(x, o);
        if (lane >= o) x += y;
    }
    __syncthreads();
    if (lane == kWave - 1) sh[wid] = x;
    __syncthreads();
    uint32_t before = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < nw; ++i) {
        const uint32_t t = sh[i];
        if (i < wid) before += t;
        tot += t;
    }
    *total = tot;
    return before + x - v;
}

struct RMAgg {
    uint64_t ntok, nsparse, dsum, qbits;
};

// Sizes of (request r, modality m) from the segment table (every thread).
__device__ __forceinline__ void rm_sizes(const Tables& t, int r, int m, uint64_t& ntok, uint64_t& qbits)
{
    ntok = 0;
    qbits = 0;
    for (int j = t.rm_off[r * kNumMod + m]; j < t.rm_off[r * kNumMod + m + 1]; ++j) {
        const DevSeg& sg = t.seg[t.rm_seg[j]];
        ntok += (uint64_t)sg.n_tok;
        if (sg.temporal) qbits += (uint64_t)(sg.T - 1) * (uint64_t)sg.P * (uint64_t)sg.C;
    }
}

// Eq. 4 and Eq. 5 integer aggregates of (r, m): the work items' partials summed.
__device__ RMAgg rm_aggregate(const Tables& t, int r, int m, unsigned long long* sh)
{
    RMAgg g;
    rm_sizes(t, r, m, g.ntok, g.qbits);
    uint64_t nsp = 0, ds = 0;
    for (int j = t.rm_off[r * kNumMod + m]; j < t.rm_off[r * kNumMod + m + 1]; ++j) {
        const int s = t.rm_seg[j];
        for (int w = t.seg_wi[s] + threadIdx.x; w < t.seg_wi[s + 1]; w += blockDim.x) {
            const Partial pr = t.partial[w];
            nsp += pr.nsparse;
            ds += pr.dsum;
        }
    }
    g.nsparse = block_sum_u64(nsp, sh);
    g.dsum = block_sum_u64(ds, sh + 1);
    return g;
}

// Sec. 4.1.3: softmax of the logits over the modalities present.
__device__ void modal_softmax(const double al[kNumMod], const bool pres[kNumMod], double beta[kNumMod])
{
#pragma clang fp contract(off)
    double mx = -INFINITY;
    for (int m = 0; m < kNumMod; ++m)
        if (pres[m] && al[m] > mx) mx = al[m];
    double den = 0.0;
    for (int m = 0; m < kNumMod; ++m)
        if (pres[m]) den += exp(al[m] - mx);
    for (int m = 0; m < kNumMod; ++m) beta[m] = pres[m] ? exp(al[m] - mx) / den : 0.0;
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
        o.tterm = (t.flags & 1u) ? gamma_avg : 1.0 - gamma_avg;
    }
    double inner = 1.0 - (double)t.lam_s[m] * o.rho;
    if (o.has_t) inner = inner - (double)t.lam_t[m] * o.tterm;
    inner = inner < 0.0 ? 0.0 : inner;
    inner = inner > 1.0 ? 1.0 : inner;
    o.mas = 1.0 - beta * inner;
    return o;
}

// MAS of (r, m) as the request role computes it (all threads call; same value).
__device__ float request_mas(const Tables& t, int r, int m, unsigned long long* sh)
{
    bool pres[kNumMod];
    double al[kNumMod], beta[kNumMod];
    for (int mm = 0; mm < kNumMod; ++mm) {
        uint64_t nt, qb;
        rm_sizes(t, r, mm, nt, qb);
        pres[mm] = nt > 0;
        al[mm] = (double)t.alpha[r * kNumMod + mm];
    }
    modal_softmax(al, pres, beta);
    const RMAgg g = rm_aggregate(t, r, m, sh);
    if (!pres[m]) return 0.0f;
    return (float)mas_terms(t, g, beta[m], m).mas;
}

__device__ void role_request(const PostArgs& a, int r, unsigned long long* sh)
{
    const Tables& t = a.t;
    RMAgg g[kNumMod];
    for (int m = 0; m < kNumMod; ++m) g[m] = rm_aggregate(t, r, m, sh);
    if (threadIdx.x != 0) return;
    bool pres[kNumMod];
    double al[kNumMod], beta[kNumMod];
    for (int m = 0; m < kNumMod; ++m) {
        pres[m] = g[m].ntok > 0;
        al[m] = (double)t.alpha[r * kNumMod + m];
    }
    modal_softmax(al, pres, beta);
    for (int m = 0; m < kNumMod; ++m) {
        const int x = r * kNumMod + m;
        MasTerms o{0.0, 0.0, 0.0, 0.0, false};
        if (pres[m]) o = mas_terms(t, g[m], beta[m], m);
        if (a.temporal_only) {
            if (a.req.temporal) a.req.temporal[x] = (float)o.tterm;
            continue;
        }
        if (a.req.agg) {
            a.req.agg[x * 4 + 0] = g[m].ntok;
            a.req.agg[x * 4 + 1] = g[m].nsparse;
            a.req.agg[x * 4 + 2] = g[m].dsum;
            a.req.agg[x * 4 + 3] = g[m].qbits;
        }
        if (a.req.rho) a.req.rho[x] = (float)o.rho;
        if (a.req.temporal) a.req.temporal[x] = (float)o.tterm;
        if (a.req.beta) a.req.beta[x] = (float)o.beta;
        if (a.req.mas) a.req.mas[x] = (float)o.mas;
        if (a.req.present) a.req.present[x] = pres[m] ? 1 : 0;
    }
}

// Eq. 5 for one frame of a temporal segment: D_t = sum of d over its tokens.
__device__ void role_frame(const PostArgs& a, int f, unsigned long long* sh)
{
    const Tables& t = a.t;
    int lo = 0, hi = t.n_tseg;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (t.seg[t.tseg[mid]].frame_off <= f) lo = mid; else hi = mid;
    }
    const DevSeg& sg = t.seg[t.tseg[lo]];
    const int tt = f - sg.frame_off;
    const int base = sg.tok_off + tt * sg.P;
    uint64_t acc = 0;
    for (int p = threadIdx.x; p < sg.P; p += blockDim.x) acc += a.d[base + p];
    const uint64_t D = block_sum_u64(acc, sh);
    if (threadIdx.x == 0) {
#pragma clang fp contract(off)
        const double sim = 1.0 - (double)D / (double)((int64_t)sg.P * sg.C);
        if (a.frm.dframe) a.frm.dframe[f] = D;
        if (a.frm.sim) a.frm.sim[f] = (float)sim;
        if (a.frm.gamma) a.frm.gamma[f] = (float)(1.0 - sim);
    }
}

// Selection key, order-equivalent to Ls*z + Lt*(C - d): when one weight is 0
// the other term alone orders the tokens, so it is used unscaled.
enum { kKeyZero = 0, kKeyZ = 1, kKeyE = 2, kKeyFull = 3 };

__device__ __forceinline__ uint64_t sel_key(const uint32_t* __restrict__ z, const uint32_t* __restrict__ d,
                                            int g, int kind, uint64_t Ls, uint64_t Lt, uint32_t C)
{
    switch (kind) {
    case kKeyZ: return (uint64_t)z[g];
    case kKeyE: return (uint64_t)(C - d[g]);
    case kKeyFull: return Ls * (uint64_t)z[g] + Lt * (uint64_t)(C - d[g]);
    default: return 0ull;
    }
}

constexpr int kRadixBits = 11;
constexpr int kRadixBins = 1 << kRadixBits;
constexpr int kBinsPerThread = kRadixBins / kPostBlock;
constexpr int kScanItems = 8;

struct SelShared {
    uint32_t hist[kRadixBins];
    uint32_t scan[kPostBlock / kWave];
    unsigned long long red[2];
    unsigned long long lo, hi;
    uint32_t digit, below;
};

// Top-k of one segment: the k smallest (key, index) pairs, kept indices
// ascending (Sec. 4.1.1 pruning, k from the Eq. 11 floor or a fixed ratio).
__device__ void role_select(const PostArgs& a, int s, SelShared& sh)
{
    const Tables& t = a.t;
    const DevSeg sg = t.seg[s];
    const int N = sg.n_tok;
    int k = sg.k;
    if (k < 0) {
#pragma clang fp contract(off)
        const float mas = a.mas_in ? a.mas_in[sg.request * kNumMod + sg.modality]
                                   : request_mas(t, sg.request, sg.modality, sh.red);
        double kk = ceil((1.0 - (double)mas) * (double)N);
        kk = kk > (double)N ? (double)N : kk;
        kk = kk < 0.0 ? 0.0 : kk;
        k = (int)kk;
    }
    if (threadIdx.x == 0) a.sel.kept_count[s] = k;
    const int off = sg.tok_off;
    if (N == 0) return;
    if (k == 0 || k == N) {
        for (int i = threadIdx.x; i < N; i += blockDim.x) {
            if (a.sel.keep) a.sel.keep[off + i] = k == N ? 1 : 0;
            a.sel.kept_idx[off + i] = k == N ? i : -1;
        }
        return;
    }
    const int kind = sg.temporal && sg.L_t > 0 ? (sg.L_s > 0 ? kKeyFull : kKeyE) : (sg.L_s > 0 ? kKeyZ : kKeyZero);
    const uint64_t Ls = sg.L_s, Lt = sg.L_t;
    const uint32_t C = (uint32_t)sg.C;
    const uint32_t* z = a.z + off;
    const uint32_t* d = a.d ? a.d + off : nullptr;

    // range of the keys
    if (threadIdx.x == 0) {
        sh.lo = ~0ull;
        sh.hi = 0ull;
    }
    __syncthreads();
    {
        uint64_t lo = ~0ull, hi = 0ull;
        for (int i = threadIdx.x; i < N; i += blockDim.x) {
            const uint64_t key = sel_key(z, d, i, kind, Ls, Lt, C);
            lo = key < lo ? key : lo;
            hi = key > hi ? key : hi;
        }
        atomicMin(&sh.lo, (unsigned long long)lo);
        atomicMax(&sh.hi, (unsigned long long)hi);
    }
    __syncthreads();
    const uint64_t lo = sh.lo, hi = sh.hi;

    // radix select of the key of rank k-1 among key - lo, most significant digit first
    uint64_t prefix = 0;
    uint32_t below = 0;            // keys strictly below the current candidate range
    uint32_t rank = (uint32_t)k - 1;
    int bits = hi > lo ? 64 - __clzll((long long)(hi - lo)) : 0;
    while (bits > 0) {
        const int db = bits < kRadixBits ? bits : kRadixBits;
        const int shift = bits - db;
        const uint64_t mask = (1ull << db) - 1ull;
        for (int b = threadIdx.x; b < kRadixBins; b += blockDim.x) sh.hist[b] = 0u;
        __syncthreads();
        for (int i = threadIdx.x; i < N; i += blockDim.x) {
            const uint64_t x = sel_key(z, d, i, kind, Ls, Lt, C) - lo;
            if ((x >> bits) == prefix) atomicAdd(&sh.hist[(x >> shift) & mask], 1u);
        }
        __syncthreads();
        uint32_t local = 0;
#pragma unroll
        for (int j = 0; j < kBinsPerThread; ++j) local += sh.hist[threadIdx.x * kBinsPerThread + j];
        uint32_t tot;
        const uint32_t ex = block_exscan(local, sh.scan, &tot);
        if (ex <= rank && rank < ex + local) {
            uint32_t cum = ex;
            for (int j = 0; j < kBinsPerThread; ++j) {
                const uint32_t h = sh.hist[threadIdx.x * kBinsPerThread + j];
                if (rank < cum + h) {
                    sh.digit = (uint32_t)(threadIdx.x * kBinsPerThread + j);
                    sh.below = cum;
                    break;
                }
                cum += h;
            }
        }
        __syncthreads();
        const uint32_t dg = sh.digit, bl = sh.below;
        below += bl;
        rank -= bl;
        prefix = (prefix << db) | dg;
        bits = shift;
        __syncthreads();
    }
    const uint64_t vstar = lo + prefix;      // key of rank k-1
    const uint32_t ties = (uint32_t)k - below; // keys equal to vstar that are kept, lowest index first

    // keep flags and ascending kept indices, tile by tile in index order
    uint32_t eq_carry = 0, kept_carry = 0;
    for (int base = 0; base < N; base += kPostBlock * kScanItems) {
        const int i0 = base + threadIdx.x * kScanItems;
        uint64_t kv[kScanItems];
        uint32_t nlt = 0, neq = 0;
#pragma unroll
        for (int j = 0; j < kScanItems; ++j) {
            kv[j] = 0;
            if (i0 + j < N) {
                kv[j] = sel_key(z, d, i0 + j, kind, Ls, Lt, C);
                nlt += kv[j] < vstar;
                neq += kv[j] == vstar;
            }
        }
        uint32_t eq_tot;
        const uint32_t eq_before = block_exscan(neq, sh.scan, &eq_tot) + eq_carry;
        const uint32_t take = eq_before >= ties ? 0u : min(neq, ties - eq_before);
        uint32_t kept_tot;
        uint32_t pos = block_exscan(nlt + take, sh.scan, &kept_tot) + kept_carry;
        uint32_t er = eq_before;
#pragma unroll
        for (int j = 0; j < kScanItems; ++j) {
            const int i = i0 + j;
            if (i < N) {
                bool kp = kv[j] < vstar;
                if (kv[j] == vstar) {
                    kp = er < ties;
                    ++er;
                }
                if (a.sel.keep) a.sel.keep[off + i] = kp ? 1 : 0;
                if (kp) a.sel.kept_idx[off + (int)pos++] = i;
            }
        }
        eq_carry += eq_tot;
        kept_carry += kept_tot;
    }
    for (int i = k + threadIdx.x; i < N; i += blockDim.x) a.sel.kept_idx[off + i] = -1;
}

__global__ __launch_bounds__(kPostBlock) void k_post(PostArgs a)
{
    __shared__ SelShared sh;
    int b = blockIdx.x;
    if (b < a.n_req_blocks) {
        role_request(a, b, sh.red);
        return;
    }
    b -= a.n_req_blocks;
    if (b < a.n_frame_blocks) {
        role_frame(a, b, sh.red);
        return;
    }
    b -= a.n_frame_blocks;
    if (b < a.n_sel_blocks) role_select(a, b, sh);
}

// ---------------------------------------------------------------- k_gather

__global__ __launch_bounds__(kGatherBlock) void k_gather(GatherArgs a)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int w = uniform(blockIdx.x * (kGatherBlock / kWave) + (threadIdx.x >> 6));
    if (w >= a.t.n_gwi) return;
    const int s = find_seg(a.t.seg_gi, a.t.n, w);
    const DevSeg sg = a.t.seg[s];
    int cnt = uniform(a.kept_count[s]);
    cnt = min(cnt, min(sg.cap, sg.n_tok));
    const int j0 = (w - sg.g_begin) * kGatherRows;
    const int j1 = min(cnt, j0 + kGatherRows);
    const int64_t row_bytes = (int64_t)sg.nchunk * 16;
    for (int j = j0; j < j1; ++j) {
        const int src = uniform(a.kept_idx[sg.tok_off + j]);
        if (src < 0 || src >= sg.n_tok) continue;
        const uint8_t* in = sg.data + (int64_t)src * sg.stride_bytes;
        uint8_t* o = a.out + sg.out_off + (int64_t)j * row_bytes;
        for (int c0 = 0; c0 < sg.nchunk; c0 += 4 * kWave) {
            uint4 v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int c = c0 + u * kWave + lane;
                if (c < sg.nchunk) v[u] = ld16(in + (int64_t)c * 16);
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int c = c0 + u * kWave + lane;
                if (c < sg.nchunk) *reinterpret_cast<uint4*>(o + (int64_t)c * 16) = v[u];
            }
        }
    }
}

}  // namespace

int launch_score(const ScoreArgs& a, void* stream)
{
    if (a.t.n_wi <= 0) return 0;
    const int waves = kScoreBlock / kWave;
    const unsigned grid = (unsigned)((a.t.n_wi + waves - 1) / waves);
    hipLaunchKernelGGL(k_score, dim3(grid), dim3(kScoreBlock), 0, (hipStream_t)stream, a);
    return (int)hipGetLastError();
}

int launch_post(const PostArgs& a, void* stream)
{
    const int blocks = a.n_req_blocks + a.n_frame_blocks + a.n_sel_blocks;
    if (blocks <= 0) return 0;
    hipLaunchKernelGGL(k_post, dim3((unsigned)blocks), dim3(kPostBlock), 0, (hipStream_t)stream, a);
    return (int)hipGetLastError();
}

int launch_gather(const GatherArgs& a, void* stream)
{
    if (a.t.n_gwi <= 0) return 0;
    const int waves = kGatherBlock / kWave;
    const unsigned grid = (unsigned)((a.t.n_gwi + waves - 1) / waves);
    hipLaunchKernelGGL(k_gather, dim3(grid), dim3(kGatherBlock), 0, (hipStream_t)stream, a);
    return (int)hipGetLastError();
}

}  // namespace msao
