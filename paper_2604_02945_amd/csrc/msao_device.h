// msao_device.h -- device helpers shared by the scoring kernels and the
// fused clip pass of the SimHash run: the channel activity test (a channel
// is active iff NOT(|x| <= tau)) on floats and on bf16 bits, and the bf16
// pair dot product into fp32.
#ifndef MSAO_DEVICE_H
#define MSAO_DEVICE_H

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace msao {
namespace {

// A value every lane of the wavefront holds, moved to a scalar register so
// that what is derived from it (buffer descriptors, loop bounds, branches)
// stays scalar: the compiler treats anything computed from threadIdx as
// varying per lane, and a per-lane buffer descriptor costs a loop of
// readfirstlanes around every load.
__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

// Active iff NOT(|x| <= tau): NaN is active, -0 is not.
__device__ __forceinline__ bool active(float x, float tau) { return !(fabsf(x) <= tau); }

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Two bf16 products summed into an fp32 accumulator (products of bf16 values
// are exact in fp32).
__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c)
{
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), __builtin_bit_cast(bf16x2, b), c, false);
}

// Activity thresholds on bf16 magnitude bits. A bf16 value widens to a float
// whose bits are its 16 bits shifted up, so |x| <= tau exactly when the 15
// magnitude bits are at most lo = bits(tau) >> 16 (NaN and inf lie above).
// For the high channel of a dword the low channel's bits ride below it, hence
// hi = lo << 16 | 0xFFFF.
struct Thr {
    uint32_t hi, lo;
};

__device__ __forceinline__ Thr bf16_thresholds(float tau)
{
    const uint32_t lo = __float_as_uint(tau) >> 16;
    return Thr{(lo << 16) | 0xFFFFu, lo};
}

constexpr uint32_t kBf16OnePair = 0x3F803F80u;  // (1.0, 1.0) in bf16

}  // namespace
}  // namespace msao

#endif
