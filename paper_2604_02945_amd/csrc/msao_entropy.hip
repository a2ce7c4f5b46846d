// msao_entropy.hip -- gfx950 (CDNA4) kernel for the draft model's confidence
// in MSAO's speculative decoding (Sec. 4.2): per row of draft logits, the
// entropy of its softmax (Eq. 9), the greedy draft token (arg max) and the
// speculation test against the confidence threshold (Eq. 10).
//
// HBM-bound streaming reduction, one pass over the logits: one workgroup per
// row, each lane reading 16-byte chunks with nontemporal buffer loads, the
// next two batches in flight while the current one is reduced. A lane keeps a
// running maximum m, s = sum exp(x - m) and t = sum exp(x - m)(x - m) over its
// chunks, so that H = ln s - t / s needs no second pass and no cancellation
// against m. Per batch of chunks the batch maximum is taken first; only when
// it exceeds m are s and t rescaled (and the arg max searched), which after
// the first batches is rare. Lane states merge by shuffles, then across the
// block's wavefronts through LDS.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "msao_internal.h"

namespace msao {
namespace {

constexpr int kEntWave = 64;
constexpr float kLog2e = 1.4426950408889634f;
// exp(-200) is far below the smallest normal float: clamping the difference
// that multiplies exp(x - m) in t only matters for x = -inf, whose term is
// then 0 * -200 = 0 instead of 0 * -inf = NaN. A NaN logit still makes s NaN.
constexpr float kMinDiff = -200.0f;

typedef unsigned int ent_vec4 __attribute__((ext_vector_type(4)));
typedef __amdgpu_buffer_rsrc_t ent_rsrc_t;

__device__ __forceinline__ ent_rsrc_t ent_rsrc(const void* base, int bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, bytes, 0x00020000);
}

// nontemporal: every logit is read once
__device__ __forceinline__ ent_vec4 ent_load(ent_rsrc_t r, int off)
{
    return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 2);
}

// Softmax statistics of a set of logits: maximum m (first index idx),
// s = sum 2^(L (x - m)) = sum exp(x - m) and u = sum 2^(L (x - m)) L (x - m)
// with L = log2(e), i.e. u = L t for t = sum exp(x - m) (x - m). Keeping u in
// log2 units lets one fma give the exponent: L x - L m.
struct Acc {
    float m, s, u;
    int idx;
};

// Merge b into a: the larger maximum wins (the lower index on equal maxima)
// and the other side's sums are rescaled to it. Only an empty side (s == 0)
// is skipped, so a NaN sum still reaches the result.
__device__ __forceinline__ Acc acc_merge(Acc a, Acc b)
{
    if (b.m > a.m || (b.m == a.m && b.idx < a.idx)) {
        const Acc c = a;
        a = b;
        b = c;
    }
    if (b.s != 0.0f) {
        const float dm = (b.m - a.m) * kLog2e;
        const float sc = __builtin_amdgcn_exp2f(dm);
        a.u += (b.u + dm * b.s) * sc;
        a.s += b.s * sc;
    }
    return a;
}

__device__ __forceinline__ Acc acc_shfl_xor(const Acc& a, int o)
{
    Acc r;
    r.m = __shfl_xor(a.m, o);
    r.s = __shfl_xor(a.s, o);
    r.u = __shfl_xor(a.u, o);
    r.idx = __shfl_xor(a.idx, o);
    return r;
}

template <int DT> struct EntLane;
template <> struct EntLane<kBF16> {
    static constexpr int EPC = 8;  // elements per 16-byte chunk
    __device__ static __forceinline__ void widen(const ent_vec4& v, float* x)
    {
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            x[2 * w] = __uint_as_float(v[w] << 16);
            x[2 * w + 1] = __uint_as_float(v[w] & 0xFFFF0000u);
        }
    }
    __device__ static __forceinline__ float element(const uint8_t* row, int64_t i)
    {
        return __uint_as_float((uint32_t)((const uint16_t*)row)[i] << 16);
    }
};
template <> struct EntLane<kF32> {
    static constexpr int EPC = 4;
    __device__ static __forceinline__ void widen(const ent_vec4& v, float* x)
    {
#pragma unroll
        for (int w = 0; w < 4; ++w) x[w] = __uint_as_float(v[w]);
    }
    __device__ static __forceinline__ float element(const uint8_t* row, int64_t i)
    {
        return ((const float*)row)[i];
    }
};

// Add the N values x to the lane state; x[j] is element first + stride_of(j)
// (index(j) gives it), used only when the maximum moves.
template <int N, typename IndexOf>
__device__ __forceinline__ void acc_add(Acc& a, const float (&x)[N], IndexOf index)
{
    float cm = x[0];
#pragma unroll
    for (int j = 1; j < N; ++j) cm = fmaxf(cm, x[j]);
    if (cm > a.m) {
        // position of the first maximum, then its index (one computation)
        int js = 0;
#pragma unroll
        for (int j = N - 1; j >= 0; --j)
            if (x[j] == cm) js = j;
        const int at = index(js);
        if (a.s > 0.0f) {
            const float dm = (a.m - cm) * kLog2e;
            const float sc = __builtin_amdgcn_exp2f(dm);
            a.u = (a.u + dm * a.s) * sc;
            a.s *= sc;
        }
        a.m = cm;
        a.idx = at;
    }
    // While nothing finite has been seen (m = -inf) the values are -inf (they
    // contribute 0) or NaN (which must reach s): take the exponent against 0,
    // since -inf - (-inf) would turn every -inf into NaN.
    const float nml = a.m == -INFINITY ? 0.0f : -a.m * kLog2e;
    // A -inf logit gives e = 0 and d = -inf, whose product must be 0, not
    // NaN. The sums are taken without a clamp on d; a -inf then shows as a
    // NaN u beside a finite s (a NaN logit makes s NaN too), and only then is
    // u summed again with d clamped, from the values still in registers. Both
    // ways give the same bits wherever no -inf occurs.
    float s = a.s, u = a.u;
#pragma unroll
    for (int j = 0; j < N; ++j) {
        const float d = fmaf(x[j], kLog2e, nml);  // L (x - m)
        const float e = __builtin_amdgcn_exp2f(d);
        s += e;
        u = fmaf(e, d, u);
    }
    if (__ballot(__builtin_isnan(u) && !__builtin_isnan(s)) != 0) {
        u = a.u;
#pragma unroll
        for (int j = 0; j < N; ++j) {
            const float d = fmaf(x[j], kLog2e, nml);
            const float e = __builtin_amdgcn_exp2f(d);
            u = fmaf(e, fmaxf(d, kMinDiff * kLog2e), u);
        }
    }
    a.s = s;
    a.u = u;
}

template <int DT, int U>
__global__ __launch_bounds__(kEntBlock) void k_entropy(EntArgs a)
{
    using L = EntLane<DT>;
    constexpr int EPC = L::EPC;
    constexpr int STEP = U * kEntBlock;  // chunks per batch of the block
    const int row = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & (kEntWave - 1), wid = tid >> 6;
    const uint8_t* base = a.logits + (int64_t)row * a.row_bytes;
    const int nfull = a.vocab / EPC;         // whole 16-byte chunks
    const int npair = nfull / (2 * STEP) * (2 * STEP);  // chunks of whole pairs of batches
    const ent_rsrc_t rs = ent_rsrc(base, nfull * 16);
    Acc acc{-INFINITY, 0.0f, 0.0f, 0};
    float x[U * EPC];
    // batches in two register sets used in turn: once a batch is widened its
    // set loads the batch after next, so two batches are in flight while one
    // is reduced. The loads are unconditional, so that no register set needs
    // a copy and the loop has one way back to its head (whose wait is then for
    // the first set only): past the row they fall outside the buffer
    // resource, read nothing and return zeros (the offsets stay below 2^31: a
    // row is at most 2^31 - 2^20 bytes).
    ent_vec4 ba[U], bb[U];
    auto load = [&](ent_vec4 (&b)[U], int c0) {
#pragma unroll
        for (int u = 0; u < U; ++u) b[u] = ent_load(rs, (c0 + u * kEntBlock + tid) * 16);
    };
    auto reduce = [&](int c0) {
        acc_add<U * EPC>(acc, x, [&](int j) { return (c0 + (j / EPC) * kEntBlock + tid) * EPC + j % EPC; });
    };
    // widen a set whose chunks may pass the row's last whole chunk: those read as -inf
    auto widen_masked = [&](const ent_vec4 (&b)[U], int c0) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            L::widen(b[u], &x[u * EPC]);
            if (c0 + u * kEntBlock + tid >= nfull) {
#pragma unroll
                for (int j = 0; j < EPC; ++j) x[u * EPC + j] = -INFINITY;
            }
        }
    };
    load(ba, 0);
    // all of the first set's loads are issued before the second set's
    __builtin_amdgcn_sched_barrier(0);
    load(bb, STEP);
    for (int c0 = 0; c0 < npair; c0 += 2 * STEP) {
#pragma unroll
        for (int u = 0; u < U; ++u) L::widen(ba[u], &x[u * EPC]);
        load(ba, c0 + 2 * STEP);
        reduce(c0);
#pragma unroll
        for (int u = 0; u < U; ++u) L::widen(bb[u], &x[u * EPC]);
        load(bb, c0 + 3 * STEP);
        reduce(c0 + STEP);
    }
    // the rest of the whole chunks, fewer than two batches, already loaded
    if (npair < nfull) {
        widen_masked(ba, npair);
        reduce(npair);
    }
    if (npair + STEP < nfull) {
        widen_masked(bb, npair + STEP);
        reduce(npair + STEP);
    }
    // the elements past the last whole chunk, one per thread
    const int tail = a.vocab - nfull * EPC;
    if (tid < tail) {
        const int i = nfull * EPC + tid;
        float x1[1] = {L::element(base, i)};
        acc_add<1>(acc, x1, [&](int) { return i; });
    }
#pragma unroll
    for (int o = 1; o < kEntWave; o <<= 1) acc = acc_merge(acc, acc_shfl_xor(acc, o));
    __shared__ Acc part[kEntBlock / kEntWave];
    if (lane == 0) part[wid] = acc;
    __syncthreads();
    if (tid != 0) return;
    Acc r = part[0];
#pragma unroll
    for (int w = 1; w < kEntBlock / kEntWave; ++w) r = acc_merge(r, part[w]);
    // Eq. 9: H = -sum p ln p = ln s - t / s with p = exp(x - m) / s and t = u / L
    const float H = __logf(r.s) - (r.u * 0.6931471805599453f) / r.s;
    const float Hn = H * a.inv_log_vocab;
    if (a.entropy) a.entropy[row] = H;
    if (a.entropy_norm) a.entropy_norm[row] = Hn;
    if (a.draft_token) a.draft_token[row] = r.idx;
    if (a.speculate) a.speculate[row] = Hn <= a.theta ? 1 : 0;  // Eq. 10
}

}  // namespace

int launch_entropy(const EntArgs& a, void* stream, void* ev0, void* ev1)
{
    if (a.rows <= 0) return kNoLaunch;
    const dim3 grid((unsigned)a.rows), block(kEntBlock);
    if (a.dtype == kBF16) {
        if (ev0 && ev1)
            hipExtLaunchKernelGGL((k_entropy<kBF16, kEntUnits>), grid, block, 0, (hipStream_t)stream, (hipEvent_t)ev0,
                                  (hipEvent_t)ev1, 0, a);
        else
            hipLaunchKernelGGL((k_entropy<kBF16, kEntUnits>), grid, block, 0, (hipStream_t)stream, a);
    } else {
        if (ev0 && ev1)
            hipExtLaunchKernelGGL((k_entropy<kF32, kEntUnits>), grid, block, 0, (hipStream_t)stream, (hipEvent_t)ev0,
                                  (hipEvent_t)ev1, 0, a);
        else
            hipLaunchKernelGGL((k_entropy<kF32, kEntUnits>), grid, block, 0, (hipStream_t)stream, a);
    }
    return (int)hipGetLastError();
}

}  // namespace msao
