// Fixed device scratch for the entry point that allocates nothing
// (moe_grouped_ffn_static).  Its only scratch is the grouped GEMM's tile
// schedule, which lives in a file-scope device array instead of a caller
// workspace.  Each GPU the library runs on holds its own copy of the array
// (at its own address) until the process ends.
#include <mutex>

#include "common.h"
#include "kernels.h"

static __device__ __align__(256) unsigned char scratch[moe::kStaticScratchBytes];

namespace moe {

namespace {
constexpr int kMaxDevices = 64;
}  // namespace

// The device address of this GPU's copy of `scratch`, looked up once per
// device with that device current.  In host code the array's name is only a
// host-side stand-in; kernels must receive this address instead.
hipError_t static_scratch(void** ptr) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    static std::once_flag once[kMaxDevices];
    static void* addr[kMaxDevices];
    static hipError_t err[kMaxDevices];
    std::call_once(once[dev], [dev] {
        void* p = nullptr;
        err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        addr[dev] = err[dev] == hipSuccess ? p : nullptr;
    });
    *ptr = addr[dev];
    return err[dev];
}

}  // namespace moe
