// Scratch memory of the entry point that allocates nothing
// (pqhsa_dense_decode_noalloc): one fixed device array, of which every GPU
// the library runs on holds its own copy until the process ends.
//
// In host code the array's name is only a host-side stand-in: its device
// address is looked up once per device, with that device current, and only
// that address is handed to kernels.
#include <mutex>

#include "pqhsa_internal.h"

namespace pqhsa {

constexpr size_t kStaticScratchBytes = size_t(32) << 20;   // 32 MiB
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

static std::mutex g_scratch_mu;
static void* g_scratch_ptr[kMaxDevices];   // device address per device, null until looked up

size_t static_scratch_bytes() { return kStaticScratchBytes; }

hipError_t static_scratch(void** ptr) {
    *ptr = nullptr;
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *ptr = g_scratch_ptr[dev];
    return hipSuccess;
}

}  // namespace pqhsa
