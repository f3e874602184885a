// The static scratch array of headkv_decode_attn_noalloc and its address.
//
// One array per GPU, shared by every call on that GPU and held until the
// process ends.  In host code the array's name is only a host-side stand-in:
// kernels receive the device address that hipGetSymbolAddress returns, looked
// up once per GPU with that GPU current.
#include <hip/hip_runtime.h>

#include <mutex>

#include "scratch.h"

namespace headkv {

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

int scratch_address(void** ptr) {
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static void* addr[kMaxDevices] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return (int)e;
    if (dev < 0 || dev >= kMaxDevices) return (int)hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (addr[dev] == nullptr) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return (int)e;
        addr[dev] = p;
    }
    *ptr = addr[dev];
    return 0;
}

}  // namespace headkv
