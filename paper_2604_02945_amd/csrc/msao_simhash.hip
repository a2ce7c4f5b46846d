// msao_simhash.hip -- the SimHash variant of Eq. 5 (Sec. 4.1.2) on gfx950.
//
// Charikar's random-hyperplane hash of every token of a clip: bit k of the
// token's signature is 1 iff r_k . f >= 0, for K = 16..64 caller hyperplanes.
// The projections [tokens x C] . [C x K] are the path's one dense
// contraction, so they run on the matrix cores (v_mfma_f32_16x16x32_bf16,
// or v_mfma_f32_16x16x4_f32 for fp32 data): a wavefront streams a tile of
// kHashTokens tokens once and turns the fp32 accumulators into signature
// bits with one ballot per accumulator register. A second launch compares
// each patch's signature with the previous frame's (d), sums D_t per frame
// (one block per frame) and the temporal term per request (one block per
// request). Nothing here is HBM traffic beyond one read of the rows and
// 12 bytes per token written (signature, d).
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "msao_device.h"
#include "msao_internal.h"

namespace msao {
namespace {

constexpr int kWave = 64;
constexpr int kHashBlock = 64 * kHashWaves;     // one wavefront per tile
constexpr int kMT = kHashTokens / 16;            // 16-token MFMA tiles per wavefront
constexpr int kSteps = 4;                        // 64-byte column steps per 256-byte chunk
static_assert(kHashTokens % 16 == 0 && kHashTokens <= 64, "tiles of 16, 32 or 64 tokens");

typedef unsigned int vec4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __amdgpu_buffer_rsrc_t rsrc_t;

// Raw buffer resource: loads at or past num_records return 0.
__device__ __forceinline__ rsrc_t make_rsrc(const void* base, int bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, bytes, 0x00020000);
}

// Rows are read once (nontemporal); hyperplanes are re-read by every tile.
__device__ __forceinline__ vec4 load_row(rsrc_t r, int off) { return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 2); }
__device__ __forceinline__ vec4 load_plane(rsrc_t r, int off) { return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0); }

constexpr int kOutOfRange = (int)0x80000000u;   // past any num_records of a tile

// Signatures of tokens [r0, r0 + kHashTokens) of a temporal segment.
//
// MFMA operand layout (16 x 16 output tiles): lane l holds row l % 16 of A
// and column l % 16 of B for the reduction slice of group g = l / 16, and
// rows 4 g .. 4 g + 3 of column l % 16 of the result. Since the reduction
// over channels may visit them in any order, A and B only need the same
// assignment of channels to (group, element): lane (m, g) takes the 16
// bytes at column byte 64 u + 16 g of a 256-byte chunk, for its token (A)
// and for hyperplane 16 j + m (B). bf16: one 16x16x32 MFMA per 16 bytes (8
// channels per lane); fp32: four 16x16x4 MFMAs, element e in the e-th.
//
// Reading A or B from memory in that layout would touch 16 rows x 64 bytes
// per instruction. Instead each wavefront reads its tile 256 contiguous
// bytes of 4 rows per instruction into its own LDS slice, and the block
// reads the chunk's K hyperplane rows once into a shared slice (so the four
// tiles of a block share them). Both slices have a 288-byte row pitch: with
// it the row writes and the column reads show no LDS bank conflicts
// (SQ_LDS_BANK_CONFLICT = 0), where 272 bytes conflict on 44 % of the LDS
// cycles and an unpadded 256 on three times as many cycles as it is active.
// The next chunk's loads are in flight during the MFMAs.
constexpr int kChunk = 256;                       // bytes of every row per step
constexpr int kLdsPitch = kChunk + 32;            // padded LDS row pitch
constexpr int kLoadsPerChunk = kHashTokens / 4;   // 4 rows x 256 bytes per load

template <int DT, int KT>
__device__ void hash_tile(const HashArgs& a, const DevSeg& sg, int r0, int lane, uint8_t* rows_lds,
                          uint8_t* planes_lds)
{
    constexpr int K = 16 * KT;
    constexpr int kPlaneLoads = K / 16;           // 16-byte pieces of the chunk's hyperplanes per thread
    const int m = lane & 15, g = lane >> 4;
    const int rows = uniform(max(0, min(kHashTokens, sg.n_tok - r0)));   // a tile past the end: no rows
    const int rb = sg.nchunk * 16;                       // row bytes
    const int pitch = (int)sg.stride_bytes;              // < 64 MiB (host check)
    const rsrc_t rx = make_rsrc(sg.data + (int64_t)min(r0, sg.n_tok) * sg.stride_bytes, rows * pitch);
    const rsrc_t rr = make_rsrc(sg.planes, K * rb);
    f32x4 acc[kMT][KT];
#pragma unroll
    for (int i = 0; i < kMT; ++i)
#pragma unroll
        for (int j = 0; j < KT; ++j) acc[i][j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    // tile rows: load q covers rows 4 q .. 4 q + 3; lane l takes row 4 q + l / 16, bytes 16 (l % 16) ..
    const int lrow = lane >> 4, lcol = (lane & 15) * 16;
    // hyperplanes: piece p = tid + 256 v is row p / 16, bytes 16 (p % 16) .. of the chunk
    const int tid = threadIdx.x;
    auto load_chunk = [&](int c, vec4 (&G)[kLoadsPerChunk], vec4 (&H)[kPlaneLoads]) {
        const int col = c * kChunk + lcol;               // past the row: zero
#pragma unroll
        for (int q = 0; q < kLoadsPerChunk; ++q)
            G[q] = load_row(rx, col < rb ? (4 * q + lrow) * pitch + col : kOutOfRange);
#pragma unroll
        for (int v = 0; v < kPlaneLoads; ++v) {
            const int p = tid + kHashBlock * v;
            const int pc = c * kChunk + (p & 15) * 16;
            H[v] = load_plane(rr, pc < rb ? (p >> 4) * rb + pc : kOutOfRange);
        }
    };
    const int nchunks = (rb + kChunk - 1) / kChunk;
    vec4 G[kLoadsPerChunk], H[kPlaneLoads];
    load_chunk(0, G, H);
    for (int c = 0; c < nchunks; ++c) {
#pragma unroll
        for (int q = 0; q < kLoadsPerChunk; ++q)
            *reinterpret_cast<vec4*>(rows_lds + (4 * q + lrow) * kLdsPitch + lcol) = G[q];
#pragma unroll
        for (int v = 0; v < kPlaneLoads; ++v) {
            const int p = tid + kHashBlock * v;
            *reinterpret_cast<vec4*>(planes_lds + (p >> 4) * kLdsPitch + (p & 15) * 16) = H[v];
        }
        __syncthreads();
        if (c + 1 < nchunks) load_chunk(c + 1, G, H);
        vec4 A[kSteps][kMT], B[kSteps][KT];
#pragma unroll
        for (int u = 0; u < kSteps; ++u) {
#pragma unroll
            for (int j = 0; j < KT; ++j)
                B[u][j] = *reinterpret_cast<const vec4*>(planes_lds + (16 * j + m) * kLdsPitch + 64 * u + 16 * g);
#pragma unroll
            for (int i = 0; i < kMT; ++i)
                A[u][i] = *reinterpret_cast<const vec4*>(rows_lds + (16 * i + m) * kLdsPitch + 64 * u + 16 * g);
        }
#pragma unroll
        for (int u = 0; u < kSteps; ++u)
#pragma unroll
            for (int i = 0; i < kMT; ++i)
#pragma unroll
                for (int j = 0; j < KT; ++j) {
                    if constexpr (DT == kBF16) {
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, A[u][i]),
                                                                            __builtin_bit_cast(bf16x8, B[u][j]),
                                                                            acc[i][j], 0, 0, 0);
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(A[u][i][e]),
                                                                             __uint_as_float(B[u][j][e]),
                                                                             acc[i][j], 0, 0, 0);
                    }
                }
        __syncthreads();  // every wavefront has read the slices before they are rewritten
    }
    // signature bits: the ballot of result register e of tile (i, j) holds,
    // at bit 16 g + n, the bit of hyperplane 16 j + n for token 16 i + 4 g + e;
    // lane L assembles token L's signature (NaN compares false: bit 0)
    const int li = lane >> 4, lg = (lane & 15) >> 2, le = lane & 3;
    uint64_t sig = 0;
#pragma unroll
    for (int i = 0; i < kMT; ++i)
#pragma unroll
        for (int j = 0; j < KT; ++j)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const uint64_t b = __ballot(acc[i][j][e] >= 0.0f);
                if (li == i && le == e) sig |= ((b >> (16 * lg)) & 0xFFFFull) << (16 * j);
            }
    if (lane < rows) a.sig[sg.tok_off + r0 + lane] = sig;
}

// One block per kHashBlockTokens tokens of a segment; wavefront w takes the
// w-th tile. Segments that are not temporal get zero signatures and d.
__global__ __launch_bounds__(kHashBlock) void k_simhash(HashArgs a)
{
    __shared__ __attribute__((aligned(16))) uint8_t rows_lds[kHashWaves][kHashTokens * kLdsPitch];
    __shared__ __attribute__((aligned(16))) uint8_t planes_lds[64 * kLdsPitch];
    const int lane = threadIdx.x & (kWave - 1), wave = uniform(threadIdx.x >> 6);
    const int b = blockIdx.x;
    const int s = a.t.hi_seg[b];
    const DevSeg sg = a.t.seg[s];
    const int r0 = (b - sg.hi_begin) * kHashBlockTokens + wave * kHashTokens;
    if (!sg.temporal) {
        if (lane < kHashTokens && r0 + lane < sg.n_tok) {
            a.sig[sg.tok_off + r0 + lane] = 0ull;
            a.d[sg.tok_off + r0 + lane] = 0u;
        }
        return;  // the whole block: one segment
    }
    uint8_t* mine = rows_lds[wave];
    const int kt = sg.hash_bits / 16;
    if (sg.dtype == kBF16) {
        switch (kt) {
        case 1: hash_tile<kBF16, 1>(a, sg, r0, lane, mine, planes_lds); break;
        case 2: hash_tile<kBF16, 2>(a, sg, r0, lane, mine, planes_lds); break;
        case 3: hash_tile<kBF16, 3>(a, sg, r0, lane, mine, planes_lds); break;
        default: hash_tile<kBF16, 4>(a, sg, r0, lane, mine, planes_lds); break;
        }
    } else {
        switch (kt) {
        case 1: hash_tile<kF32, 1>(a, sg, r0, lane, mine, planes_lds); break;
        case 2: hash_tile<kF32, 2>(a, sg, r0, lane, mine, planes_lds); break;
        case 3: hash_tile<kF32, 3>(a, sg, r0, lane, mine, planes_lds); break;
        default: hash_tile<kF32, 4>(a, sg, r0, lane, mine, planes_lds); break;
        }
    }
}

// ------------------------------------------------------------ k_clip

constexpr int kClipBlock = 64 * kClipWaves;

// Hyperplane slices per block: two (used in turn, one barrier per chunk)
// for K <= 32, where the block's LDS stays small enough for four 4-wavefront
// blocks per CU; one (and a second barrier per chunk) for K = 48 and 64.
template <int KT>
constexpr int kClipPlaneBufs = KT <= 2 ? 2 : 1;

// DPP row_ror:n (rotation by n lanes within each 16-lane row).
template <int N>
__device__ __forceinline__ int dpp_ror(int v)
{
    return __builtin_amdgcn_update_dpp(0, v, 0x120 + N, 0xF, 0xF, false);
}

// Sum over the 16 lanes of each row; every lane of the row gets a sum (the
// float sums of different lanes may round differently: read one fixed lane).
__device__ __forceinline__ float row16_sum(float v)
{
    v += __int_as_float(dpp_ror<8>(__float_as_int(v)));
    v += __int_as_float(dpp_ror<4>(__float_as_int(v)));
    v += __int_as_float(dpp_ror<2>(__float_as_int(v)));
    v += __int_as_float(dpp_ror<1>(__float_as_int(v)));
    return v;
}
__device__ __forceinline__ uint32_t row16_sum(uint32_t v)
{
    v += (uint32_t)dpp_ror<8>((int)v);
    v += (uint32_t)dpp_ror<4>((int)v);
    v += (uint32_t)dpp_ror<2>((int)v);
    v += (uint32_t)dpp_ror<1>((int)v);
    return v;
}

typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

// The channels of 16 bytes of a row widened to floats: the low and high
// halves of each dword for bf16 (8 channels), the dwords for fp32 (4).
struct Wide {
    float v[8];
};

template <int DT>
__device__ __forceinline__ Wide widen(const vec4& x)
{
    Wide w;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        if constexpr (DT == kBF16) {
            w.v[2 * k] = __uint_as_float(x[k] << 16);
            w.v[2 * k + 1] = __uint_as_float(x[k] & 0xFFFF0000u);
        } else {
            w.v[k] = __uint_as_float(x[k]);
        }
    }
    return w;
}

// Per-lane statistics of 16 bytes of a row x against the same bytes of its
// predecessor, given widened in pw (on return pw holds x widened, the
// predecessor of the next row): active count, L1, L2 and squared
// difference. For bf16 the active count is kept per 16-bit half: the
// threshold bits minus a channel's magnitude bits, both below 2^15 (tau is
// finite and not -0), wrap below zero, setting bit 15, exactly when the
// channel is active (NaN included); the bit shifted down is added to the
// half's count, which counts at most C / 32 channels per lane, below 2^16.
// (Written as a saturating subtraction capped at 1, the compiler turns it
// into a compare and select per half.)
template <int DT>
__device__ __forceinline__ void clip_stats(const vec4& x, Wide& pw, float tau, const Thr& th, uint32_t& act,
                                           float& l1, float& l2, float& res)
{
    const Wide xw = widen<DT>(x);
    if constexpr (DT == kBF16) {
        const u16x2 th2 = {(unsigned short)th.lo, (unsigned short)th.lo};
        const u16x2 sh15 = {15, 15};
        u16x2 cnt = __builtin_bit_cast(u16x2, act);
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            const uint32_t xv = x[w];
            const uint32_t ax = xv & 0x7FFF7FFFu;
            cnt += (th2 - __builtin_bit_cast(u16x2, ax)) >> sh15;
            l1 = dot2(ax, kBf16OnePair, l1);
            l2 = dot2(xv, xv, l2);
            const float dlo = xw.v[2 * w] - pw.v[2 * w];
            const float dhi = xw.v[2 * w + 1] - pw.v[2 * w + 1];
            res = fmaf(dlo, dlo, res);
            res = fmaf(dhi, dhi, res);
        }
        act = __builtin_bit_cast(uint32_t, cnt);
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float xf = xw.v[e];
            act += active(xf, tau) ? 1u : 0u;
            l1 += fabsf(xf);
            l2 = fmaf(xf, xf, l2);
            const float df = xf - pw.v[e];
            res = fmaf(df, df, res);
        }
    }
    pw = xw;
}

// One tile: rows r = 0..nf are frames f0 + r of patch position p (f0 =
// nf j - 1 with nf <= 15 new frames per tile; frame -1 reads as zero, rows
// past the tile or the clip too). Per 256-byte
// chunk of the rows, the wavefront stages its tile in LDS (4 rows x 256
// contiguous bytes per load), reads each row and its predecessor back for
// the statistics, and runs the tile through the matrix cores against the
// block's shared hyperplane chunk, as k_simhash does. Rows 1..nf are the
// tile's tokens; row 0 only supplies their predecessor. For the statistics
// lane group g (lanes 16 g ..) takes rows g rpg .. g rpg + rpg - 1, rpg =
// ceil(r_hi / 4), so that each row's predecessor is the row before it in the
// same lanes (read and widened once) and rows past the tile are skipped.
template <int DT, int KT>
__device__ void clip_tile(const ClipArgs& a, const DevSeg& sg, int item, int lane, uint8_t* rows_lds,
                          uint8_t* planes_lds, uint32_t& nsp, uint64_t& dsum)
{
    constexpr int K = 16 * KT;
    constexpr int kPieces = K * (kChunk / 16);                      // 16-byte pieces of a hyperplane chunk
    constexpr int kPlaneLoads = (kPieces + kClipBlock - 1) / kClipBlock;
    const int m = lane & 15, g = lane >> 4;
    const bool valid = item < sg.P * sg.ntiles;
    const int p = valid ? item / sg.ntiles : 0;
    const int j = valid ? item % sg.ntiles : 0;
    const int nf = sg.per_item;                          // new frames per tile (the frames split evenly)
    const int f0 = nf * j - 1;
    const int r_lo = f0 < 0 ? 1 : 0;                    // row 0 of the first tile: the zero frame
    const int r_hi = valid ? min(nf + 1, sg.T - f0) : 0; // rows from r_hi on: past the tile or the clip
    const int rb = sg.nchunk * 16;
    const int fstride = (int)((int64_t)sg.P * sg.stride_bytes);   // 16 x fstride <= 2^31 - 1 (host check)
    const int nrows = max(0, r_hi - r_lo);
    const rsrc_t rx = make_rsrc(sg.data + (int64_t)p * sg.stride_bytes + (int64_t)(f0 + r_lo) * fstride,
                                nrows > 0 ? (nrows - 1) * fstride + rb : 0);
    const rsrc_t rr = make_rsrc(sg.planes, K * rb);
    const float tau = a.t.tau;
    const Thr th = bf16_thresholds(tau);
    f32x4 acc[KT];
#pragma unroll
    for (int jj = 0; jj < KT; ++jj) acc[jj] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    uint32_t act[4] = {0u, 0u, 0u, 0u};
    float l1[4] = {0.0f, 0.0f, 0.0f, 0.0f}, l2[4] = {0.0f, 0.0f, 0.0f, 0.0f}, res[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    // load q covers rows 4 q .. 4 q + 3: lane l takes row 4 q + l / 16, bytes 16 (l % 16) .. of the chunk
    const int lrow = lane >> 4, lcol = (lane & 15) * 16;
    const int rpg = (r_hi + 3) >> 2;                    // statistics rows per lane group (<= 4)
    const int rg0 = lrow * rpg;                          // the group's first row (rg0 + rpg - 1 <= 15)
    const int tid = threadIdx.x;
    auto load_chunk = [&](int c, vec4 (&G)[4], vec4 (&H)[kPlaneLoads]) {
        const int col = c * kChunk + lcol;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int r = 4 * q + lrow;
            G[q] = load_row(rx, (col < rb && r >= r_lo && r < r_hi) ? (r - r_lo) * fstride + col : kOutOfRange);
        }
#pragma unroll
        for (int v = 0; v < kPlaneLoads; ++v) {
            const int pp = tid + kClipBlock * v;
            const int pc = c * kChunk + (pp & 15) * 16;
            H[v] = load_plane(rr, (pp < kPieces && pc < rb) ? (pp >> 4) * rb + pc : kOutOfRange);
        }
    };
    const int nchunks = (rb + kChunk - 1) / kChunk;
    vec4 G[4], H[kPlaneLoads];
    load_chunk(0, G, H);
    for (int c = 0; c < nchunks; ++c) {
        // the wavefront's own row slice: rewritten only after its own reads
        // of the previous chunk (one wavefront's LDS operations run in order)
#pragma unroll
        for (int q = 0; q < 4; ++q) *reinterpret_cast<vec4*>(rows_lds + (4 * q + lrow) * kLdsPitch + lcol) = G[q];
        uint8_t* const pl = planes_lds + (kClipPlaneBufs<KT> == 2 ? (c & 1) : 0) * (16 * KT * kLdsPitch);
#pragma unroll
        for (int v = 0; v < kPlaneLoads; ++v) {
            const int pp = tid + kClipBlock * v;
            if (pp < kPieces)
                *reinterpret_cast<vec4*>(pl + (pp >> 4) * kLdsPitch + (pp & 15) * 16) = H[v];
        }
        __syncthreads();
        if (c + 1 < nchunks) load_chunk(c + 1, G, H);
        // statistics: each lane's 16 bytes of rows rg0 + i against the row above
        if (rpg > 0) {
            Wide pw = widen<DT>(*reinterpret_cast<const vec4*>(rows_lds + (rg0 > 0 ? rg0 - 1 : 0) * kLdsPitch + lcol));
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                if (i >= rpg) break;
                const vec4 x = *reinterpret_cast<const vec4*>(rows_lds + (rg0 + i) * kLdsPitch + lcol);
                clip_stats<DT>(x, pw, tau, th, act[i], l1[i], l2[i], res[i]);
            }
        }
        // one 64-byte column step at a time (the operands of one step live at once)
#pragma unroll
        for (int u = 0; u < kSteps; ++u) {
            const vec4 A = *reinterpret_cast<const vec4*>(rows_lds + m * kLdsPitch + 64 * u + 16 * g);
#pragma unroll
            for (int jj = 0; jj < KT; ++jj) {
                const vec4 B = *reinterpret_cast<const vec4*>(pl + (16 * jj + m) * kLdsPitch + 64 * u + 16 * g);
                if constexpr (DT == kBF16) {
                    acc[jj] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, A),
                                                                      __builtin_bit_cast(bf16x8, B), acc[jj], 0, 0, 0);
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        acc[jj] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(A[e]), __uint_as_float(B[e]),
                                                                       acc[jj], 0, 0, 0);
                }
            }
        }
        // with one hyperplane slice, every wavefront has read it before it is
        // rewritten; with two, the next chunk writes the other one, and the
        // one after waits for the barrier above
        if constexpr (kClipPlaneBufs<KT> == 1) __syncthreads();
    }
    // signature of row L in lane L < 16: the ballot of result register e of
    // tile column block jj holds, at bit 16 lg + n, hyperplane 16 jj + n of row 4 lg + e
    const int lg = (lane & 15) >> 2, le = lane & 3;
    uint64_t sig = 0;
#pragma unroll
    for (int jj = 0; jj < KT; ++jj)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const uint64_t b = __ballot(acc[jj][e] >= 0.0f);
            if (g == 0 && le == e) sig |= ((b >> (16 * lg)) & 0xFFFFull) << (16 * jj);
        }
    // d against the row above (lane L - 1 holds it)
    const int up = lane > 0 ? lane - 1 : 0;
    const uint32_t slo = (uint32_t)__shfl((int)(uint32_t)sig, up), shi = (uint32_t)__shfl((int)(uint32_t)(sig >> 32), up);
    const uint32_t d = (uint32_t)__popcll(sig ^ (((uint64_t)shi << 32) | slo));
    // row r's sums (every lane of its group holds them): group gr = r / rpg,
    // register r - gr rpg; lane r takes them from lane 16 gr
    const int rp = max(rpg, 1), lr = lane & 15;
    const int gr = min(lr / rp, 3), qr = lr - gr * rp;
    const int src = 16 * gr;
    uint32_t A_r = 0u;
    float L1 = 0.0f, L2 = 0.0f, RS = 0.0f;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const uint32_t aq = (uint32_t)__shfl((int)row16_sum(DT == kBF16 ? (act[q] & 0xFFFFu) + (act[q] >> 16) : act[q]), src);
        const float l1q = __shfl(row16_sum(l1[q]), src);
        const float l2q = __shfl(row16_sum(l2[q]), src);
        const float rq = __shfl(row16_sum(res[q]), src);
        if (qr == q) {
            A_r = aq;
            L1 = l1q;
            L2 = l2q;
            RS = rq;
        }
    }
    const int f = f0 + lane;
    const bool out = valid && lane >= 1 && lane < r_hi;
    if (out) {
        const int tk = sg.tok_off + f * sg.P + p;
        const uint32_t z = (uint32_t)sg.C - A_r;
        const TokenOut& o = a.tok;
        if (o.z) o.z[tk] = z;
        if (o.l1) o.l1[tk] = L1;
        if (o.l2) o.l2[tk] = L2;
        if (o.res) o.res[tk] = RS;
        if (o.d) o.d[tk] = d;
        if (o.sig) o.sig[tk] = sig;
        if (o.info) {
            const float red = sg.lam_s * (float)z * __builtin_amdgcn_rcpf((float)sg.C) +
                              sg.lam_t * (float)(K - (int)d) * __builtin_amdgcn_rcpf((float)K);
            o.info[tk] = 1.0f - red;
        }
    }
    nsp += (uint32_t)__popcll(__ballot(out && A_r < (uint32_t)sg.A_s));
    uint32_t dd = (out && f >= 1) ? d : 0u;
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) dd += (uint32_t)__shfl_xor((int)dd, o);
    dsum += (uint64_t)__shfl((int)dd, 0);
}

// One block per kClipWaves work items (tiles) of one fused clip; each
// wavefront writes its work item's integer partials. One instance per
// element type and signature width, so that each holds only its own
// accumulators.
#ifndef MSAO_CLIP_WPE
#define MSAO_CLIP_WPE 1
#endif
// Block order: with 1 (the default) consecutive blocks of the plan run on
// one XCD. The hardware deals blocks to the 8 XCDs in turn, so in plan order
// the tiles of neighbouring patch positions sit in different L2s and their
// 4-byte outputs, a frame stride apart, leave as partial lines (5x the
// output bytes at L2 on the video clips; with the remap, 1.0x).
#ifndef MSAO_CLIP_XCD
#define MSAO_CLIP_XCD 1
#endif
template <int DT, int KT>
__global__ __launch_bounds__(kClipBlock) __attribute__((amdgpu_waves_per_eu(MSAO_CLIP_WPE, 8))) void k_clip(ClipArgs a)
{
    __shared__ __attribute__((aligned(16))) uint8_t rows_lds[kClipWaves][16 * kLdsPitch];
    __shared__ __attribute__((aligned(16))) uint8_t planes_lds[kClipPlaneBufs<KT> * 16 * KT * kLdsPitch];
    const int lane = threadIdx.x & (kWave - 1), wave = uniform(threadIdx.x >> 6);
    int blk = blockIdx.x;
    if (MSAO_CLIP_XCD) {  // a bijection of [0, nb): XCD x gets the x-th run of consecutive blocks
        const int nb = gridDim.x, x = blk & 7, per = nb >> 3, rem = nb & 7;
        blk = x * per + min(x, rem) + (blk >> 3);
    }
    const int s = a.t.cl_seg[blk];
    const DevSeg sg = a.t.seg[s];
    const int item = (blk - sg.cl_begin) * kClipWaves + wave;
    uint32_t nsp = 0;
    uint64_t dsum = 0;
    clip_tile<DT, KT>(a, sg, item, lane, rows_lds[wave], planes_lds, nsp, dsum);
    if (lane == 0 && item < sg.P * sg.ntiles) {
        Partial pr;
        pr.nsparse = nsp;
        pr.pad_ = 0u;
        pr.dsum = dsum;
        a.t.partial[sg.wi_begin + item] = pr;
    }
}

// ------------------------------------------------------------ k_hash_post

__device__ __forceinline__ uint64_t all_bits(int K) { return K >= 64 ? ~0ull : ((1ull << K) - 1ull); }

// Block-wide sum of a 64-bit count, the same value in every thread.
__device__ __forceinline__ uint64_t block_sum(uint64_t v, uint64_t* red)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)v, o);
        const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(v >> 32), o);
        v += ((uint64_t)hi << 32) | lo;
    }
    __syncthreads();
    if ((threadIdx.x & (kWave - 1)) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    uint64_t s = 0;
#pragma unroll
    for (int w = 0; w < kHashBlock / kWave; ++w) s += red[w];
    return s;
}

// Frame f: d of its tokens against the previous frame (frame 0 against the
// all-zero frame, all bits 1), D_t, sim = 1 - D_t / (P K), gamma. In a run
// with SimHash also the tokens' informativeness 1 - (lambda_s z / C +
// lambda_t (K - d) / K).
__device__ void hash_frame(const HashArgs& a, int f, uint64_t* red)
{
    const Tables& t = a.t;
    const DevSeg& sg = t.seg[t.frame_seg[f]];
    const int tt = f - sg.frame_off;
    const int base = sg.tok_off + tt * sg.P;
    const uint64_t ones = all_bits(sg.hash_bits);
    const float rc = __builtin_amdgcn_rcpf((float)sg.C), rk = __builtin_amdgcn_rcpf((float)sg.hash_bits);
    uint64_t acc = 0;
    for (int p = threadIdx.x; p < sg.P; p += kHashBlock) {
        const uint64_t prev = tt > 0 ? a.sig[base + p - sg.P] : ones;
        const uint32_t dd = (uint32_t)__popcll(a.sig[base + p] ^ prev);
        a.d[base + p] = dd;
        if (a.info) {
            const float red = sg.lam_s * (float)a.z[base + p] * rc + sg.lam_t * (float)(sg.hash_bits - (int)dd) * rk;
            a.info[base + p] = 1.0f - red;
        }
        acc += dd;
    }
    const uint64_t D = block_sum(acc, red);
    if (threadIdx.x == 0) {
#pragma clang fp contract(off)
        const double sim = 1.0 - (double)D / (double)((int64_t)sg.P * sg.hash_bits);
        if (a.frm.dframe) a.frm.dframe[f] = D;
        if (a.frm.sim) a.frm.sim[f] = (float)sim;
        if (a.frm.gamma) a.frm.gamma[f] = (float)(1.0 - sim);
    }
}

// Request r: per modality, the differing bits over frames 1..T-1 of its
// clips (recomputed from the signatures; written to hdsum in a run with
// SimHash) and (T - 1) P K, then the temporal term of Eq. 7.
__device__ void hash_request(const HashArgs& a, int r, uint64_t* red)
{
    const Tables& t = a.t;
    for (int m = 0; m < kNumMod; ++m) {
        const RmEntry e = t.rm[r * kNumMod + m];
        uint64_t dsum = 0, qbits = 0;
        for (int j = e.rng_begin; j < e.rng_end; ++j) {
            const DevSeg& sg = t.seg[t.rm_rng[j].seg];
            if (!sg.temporal) continue;
            qbits += (uint64_t)(sg.T - 1) * (uint64_t)sg.P * (uint64_t)sg.hash_bits;
            // 8 tokens per thread in flight (indices clamped, extras dropped)
            constexpr int U = 8;
            const uint64_t* sig = a.sig + sg.tok_off;
            for (int i0 = sg.P + threadIdx.x; i0 < sg.n_tok; i0 += U * kHashBlock) {
                uint64_t cur[U], prev[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int i = min(i0 + u * kHashBlock, sg.n_tok - 1);
                    cur[u] = sig[i];
                    prev[u] = sig[i - sg.P];
                }
#pragma unroll
                for (int u = 0; u < U; ++u)
                    if (i0 + u * kHashBlock < sg.n_tok) dsum += (uint64_t)__popcll(cur[u] ^ prev[u]);
            }
        }
        dsum = block_sum(dsum, red);
        if (threadIdx.x == 0) {
#pragma clang fp contract(off)
            float term = 0.0f;
            if (qbits > 0) {
                const double gamma_avg = (double)dsum / (double)qbits;
                term = (float)((t.flags & kFlagLiteral) ? gamma_avg : 1.0 - gamma_avg);
            }
            if (a.temporal) a.temporal[r * kNumMod + m] = term;
            if (a.hdsum) a.hdsum[r * kNumMod + m] = dsum;
        }
    }
}

__global__ __launch_bounds__(kHashBlock) void k_hash_post(HashArgs a)
{
    __shared__ uint64_t red[kHashBlock / kWave];
    const int b = blockIdx.x;
    if (b < a.n_frame_blocks) hash_frame(a, b, red);
    else hash_request(a, b - a.n_frame_blocks, red);
}

template <typename Args>
int launch(void (*kernel)(Args), dim3 grid, dim3 block, void* stream, const Args& a, void* ev0, void* ev1)
{
    if (ev0 && ev1)
        hipExtLaunchKernelGGL(kernel, grid, block, 0, (hipStream_t)stream, (hipEvent_t)ev0, (hipEvent_t)ev1, 0, a);
    else
        hipLaunchKernelGGL(kernel, grid, block, 0, (hipStream_t)stream, a);
    return (int)hipGetLastError();
}

}  // namespace

int launch_simhash(const HashArgs& a, void* stream, void* ev0, void* ev1)
{
    if (a.t.n_hi <= 0) return kNoLaunch;
    if (!a.sig || !a.d) return (int)hipErrorInvalidValue;
    return launch(k_simhash, dim3((unsigned)a.t.n_hi), dim3(kHashBlock), stream, a, ev0, ev1);
}

int launch_clip(const ClipArgs& a, void* stream, void* ev0, void* ev1)
{
    if (a.t.n_cl <= 0) return kNoLaunch;
    if (!a.tok.z || !a.tok.d || !a.tok.sig || !a.t.cl_seg) return (int)hipErrorInvalidValue;
    // every fused clip of a run has the same element type and signature width (host check)
    const dim3 grid((unsigned)a.t.n_cl), block(kClipBlock);
    switch (a.clip_dtype * 8 + a.clip_bits / 16) {
    case kBF16 * 8 + 1: return launch(k_clip<kBF16, 1>, grid, block, stream, a, ev0, ev1);
    case kBF16 * 8 + 2: return launch(k_clip<kBF16, 2>, grid, block, stream, a, ev0, ev1);
    case kBF16 * 8 + 3: return launch(k_clip<kBF16, 3>, grid, block, stream, a, ev0, ev1);
    case kBF16 * 8 + 4: return launch(k_clip<kBF16, 4>, grid, block, stream, a, ev0, ev1);
    case kF32 * 8 + 1: return launch(k_clip<kF32, 1>, grid, block, stream, a, ev0, ev1);
    case kF32 * 8 + 2: return launch(k_clip<kF32, 2>, grid, block, stream, a, ev0, ev1);
    case kF32 * 8 + 3: return launch(k_clip<kF32, 3>, grid, block, stream, a, ev0, ev1);
    case kF32 * 8 + 4: return launch(k_clip<kF32, 4>, grid, block, stream, a, ev0, ev1);
    default: return (int)hipErrorInvalidValue;
    }
}

int launch_hash_post(const HashArgs& a, void* stream, void* ev0, void* ev1)
{
    const int blocks = a.n_frame_blocks + a.n_req_blocks;
    if (blocks <= 0) return kNoLaunch;
    if (!a.sig || !a.d || (a.n_req_blocks > 0 && !a.temporal && !a.hdsum) || (a.info && !a.z))
        return (int)hipErrorInvalidValue;
    return launch(k_hash_post, dim3((unsigned)blocks), dim3(kHashBlock), stream, a, ev0, ev1);
}

}  // namespace msao
