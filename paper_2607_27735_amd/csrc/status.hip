// status.hip -- the device's exchange status word.
//
// Kernels that exchange partial results between co-resident workgroups wait
// for each other with bounded polls.  A wait that gives up (the workgroups
// were not all resident, e.g. because other work held CUs) sets its kernel
// family's bit here; the host reads and clears the word in stream order.
// Each device that loads the library holds its own copy of the two words.
#include <atomic>

#include "launch.h"

namespace ssl {
namespace {

__device__ uint32_t g_exchange_status;   // bits of kStatus*, zero at load
__device__ uint32_t g_status_taken;      // the value the last take_status_kernel read

__global__ void take_status_kernel(uint32_t* word, uint32_t* taken) {
    *taken = __hip_atomic_exchange(word, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

constexpr int kMaxDevices = 64;

// The device addresses of the two words on the current device, looked up once
// per device (looking them up twice is harmless, so a race between threads is
// too).
hipError_t status_words(uint32_t** word, uint32_t** taken) {
    static std::atomic<uintptr_t> words[kMaxDevices], takens[kMaxDevices];
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    const bool cached = dev >= 0 && dev < kMaxDevices;
    uintptr_t w = cached ? words[dev].load(std::memory_order_relaxed) : 0;
    uintptr_t t = cached ? takens[dev].load(std::memory_order_relaxed) : 0;
    if (w == 0 || t == 0) {
        void* pw = nullptr;
        void* pt = nullptr;
        e = hipGetSymbolAddress(&pw, HIP_SYMBOL(g_exchange_status));
        if (e != hipSuccess) return e;
        e = hipGetSymbolAddress(&pt, HIP_SYMBOL(g_status_taken));
        if (e != hipSuccess) return e;
        w = reinterpret_cast<uintptr_t>(pw);
        t = reinterpret_cast<uintptr_t>(pt);
        if (cached) {
            words[dev].store(w, std::memory_order_relaxed);
            takens[dev].store(t, std::memory_order_relaxed);
        }
    }
    *word = reinterpret_cast<uint32_t*>(w);
    *taken = reinterpret_cast<uint32_t*>(t);
    return hipSuccess;
}

}  // namespace

hipError_t exchange_status_word(uint32_t** word) {
    uint32_t* taken = nullptr;
    return status_words(word, &taken);
}

hipError_t take_exchange_status(hipStream_t stream, uint32_t* flags) {
    uint32_t *word = nullptr, *taken = nullptr;
    hipError_t e = status_words(&word, &taken);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(take_status_kernel, dim3(1), dim3(1), 0, stream, word, taken);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    uint32_t host = 0;
    e = hipMemcpyAsync(&host, taken, sizeof host, hipMemcpyDeviceToHost, stream);
    if (e != hipSuccess) return e;
    e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return e;
    *flags = host;
    return hipSuccess;
}

}  // namespace ssl
