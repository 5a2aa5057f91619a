// static_scratch.hip -- verify attention for callers that cannot allocate.
//
// ssl_verify_attn_static is ssl_verify_attn with the library's own device
// scratch as its workspace: a file-scope array that each GPU the library runs
// on holds from the moment the library's code is loaded on it until the
// process ends.  Host code never uses the array's name as an address (on the
// host it only stands for the symbol): the array's address on a device comes
// from hipGetSymbolAddress, looked up once per device with that device
// current, and that address is what the kernels receive.
#include <atomic>

#include "../../include/sparsespec_l.h"
#include "launch.h"

namespace ssl {

int verify_attn_static_scratch(const ssl_shape* shape, const ssl_params* params,
                               const int32_t* ctx_len_host, const int32_t* q_len_host,
                               const void* q, const void* k_cache, const void* v_cache, void* out,
                               float* scores, const StaticScratch& scratch, hipStream_t stream);

namespace {

// Enough for every verify workspace of the workloads this library is measured
// on (the largest, a 70B-shaped layer of batch 4 at 64K keys, needs 105 MiB).
constexpr size_t kScratchBytes = (size_t)128 << 20;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::atomic<uintptr_t> g_scratch_ptr[kMaxDevices];   // 0: not looked up on that device yet

// The scratch's address on the current device (looking it up twice is
// harmless, so a race between threads is too).
hipError_t scratch_address(void** ptr) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    uintptr_t p = g_scratch_ptr[dev].load(std::memory_order_acquire);
    if (p == 0) {
        void* addr = nullptr;
        e = hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (addr == nullptr) return hipErrorInvalidSymbol;
        p = reinterpret_cast<uintptr_t>(addr);
        g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
    *ptr = reinterpret_cast<void*>(p);
    return hipSuccess;
}

}  // namespace
}  // namespace ssl

extern "C" int ssl_verify_attn_static(const ssl_shape* shape, const ssl_params* params,
                                      const int32_t* ctx_len_host, const int32_t* q_len_host,
                                      const void* q, const void* k_cache, const void* v_cache,
                                      void* out, float* scores, hipStream_t stream) {
    const ssl::StaticScratch s{ssl::kScratchBytes, &ssl::scratch_address};
    return ssl::verify_attn_static_scratch(shape, params, ctx_len_host, q_len_host, q, k_cache,
                                           v_cache, out, scores, s, stream);
}
