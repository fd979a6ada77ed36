// Static device scratch for ftcnn_protected_conv_noalloc, the form of the protected layer for
// callers that cannot allocate device memory.  The array is a file-scope __device__ object of this
// file's code object; its device address is looked up once per device, with that device current,
// and only that address is ever handed to kernels or copies (in host code the array's name is a
// host-side stand-in, not a device address).  Each device that the entry point runs on holds its
// own copy of the array until the process ends.
#include <mutex>

#include "ftcnn_internal.h"

namespace ftcnn {
namespace {

__device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void *g_addr[kMaxDevices];

}  // namespace

hipError_t static_scratch(int device, void **ptr) {
    if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_addr[device]) {
        int cur = 0;
        hipError_t e = hipGetDevice(&cur);
        if (e != hipSuccess) return e;
        if (cur != device) {
            e = hipSetDevice(device);
            if (e != hipSuccess) return e;
        }
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (cur != device) {
            const hipError_t e2 = hipSetDevice(cur);
            if (e == hipSuccess) e = e2;
        }
        if (e != hipSuccess) return e;
        if (!p || reinterpret_cast<uintptr_t>(p) % 256) return hipErrorInvalidSymbol;
        g_addr[device] = p;
    }
    *ptr = g_addr[device];
    return hipSuccess;
}

}  // namespace ftcnn
