// msao_scratch.hip -- the library's own device scratch, for msao_run_noalloc.
//
// msao_run_noalloc serves callers that cannot allocate device memory (code
// under HIP graph capture, tight serving loops, harnesses that forbid
// hipMalloc): in place of a caller workspace it uses one fixed array per
// GPU, a file-scope __device__ array of kNoAllocScratchBytes that the code
// object carries (it lives until the process ends). Host code never passes
// the array's name to a kernel: in host code that name is only a stand-in,
// not a device address. Its device address is looked up once per device
// with hipGetSymbolAddress, with that device current, and kept here.
#include <hip/hip_runtime.h>

#include <mutex>

#include "msao_internal.h"

namespace msao {

static __device__ __align__(256) uint8_t scratch[kNoAllocScratchBytes];

namespace {
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices] = {};
}  // namespace

// Looks up (once) the device address of `device`'s copy of the scratch
// array. The caller has made `device` current. Returns the HIP error code.
int scratch_init(int device)
{
    if (device < 0 || device >= kMaxScratchDevices) return (int)hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[device]) return (int)hipSuccess;
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return (int)e;
    if (!p) return (int)hipErrorInvalidSymbol;
    g_scratch_ptr[device] = p;
    return (int)hipSuccess;
}

// The device address found by scratch_init for `device`, or NULL.
void* scratch_ptr(int device)
{
    if (device < 0 || device >= kMaxScratchDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    return g_scratch_ptr[device];
}

}  // namespace msao
