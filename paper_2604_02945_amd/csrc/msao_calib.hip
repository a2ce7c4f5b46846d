// msao_calib.hip -- a plain streaming read of a device buffer, the ceiling
// the HBM-bound passes are measured against on the same box: each wavefront
// reads one contiguous chunk with 128-bit nontemporal buffer loads, eight
// 1-KiB units in flight, and folds the words it read into one XOR per
// wavefront (written out, so that no load can be dropped). No arithmetic of
// the analysis runs here.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "msao_device.h"
#include "msao_internal.h"

namespace msao {
namespace {

typedef unsigned int cvec4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(kReadBlock) void k_read(ReadArgs a)
{
    const int lane = threadIdx.x & 63;
    const int64_t w = (int64_t)blockIdx.x * (kReadBlock / 64) + uniform(threadIdx.x >> 6);
    if (w >= a.waves) return;
    const int64_t begin = w * a.chunk_bytes;
    const int64_t left = a.bytes - begin;
    const int n = (int)(left < a.chunk_bytes ? left : a.chunk_bytes);
    const __amdgpu_buffer_rsrc_t r =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(a.data + begin), (short)0, n, 0x00020000);
    uint32_t x = 0;
    for (int u0 = 0; u0 < a.chunk_bytes; u0 += 8 * 1024) {
        cvec4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = __builtin_amdgcn_raw_buffer_load_b128(r, u0 + u * 1024 + lane * 16, 0, 2);
#pragma unroll
        for (int u = 0; u < 8; ++u) x ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x ^= (uint32_t)__shfl_xor((int)x, o);
    if (lane == 0) a.sink[w] = x;
}

}  // namespace

int launch_read(const ReadArgs& a, void* stream, void* ev0, void* ev1)
{
    if (a.waves <= 0) return kNoLaunch;
    const int64_t blocks = (a.waves + kReadBlock / 64 - 1) / (kReadBlock / 64);
    if (ev0 && ev1)
        hipExtLaunchKernelGGL(k_read, dim3((unsigned)blocks), dim3(kReadBlock), 0, (hipStream_t)stream,
                              (hipEvent_t)ev0, (hipEvent_t)ev1, 0, a);
    else
        hipLaunchKernelGGL(k_read, dim3((unsigned)blocks), dim3(kReadBlock), 0, (hipStream_t)stream, a);
    return (int)hipGetLastError();
}

}  // namespace msao
