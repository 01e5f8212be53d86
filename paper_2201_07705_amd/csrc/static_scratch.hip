// Static device scratch of the allocation-free inference round
// (gemel_infer_noalloc): a file-scope device array holds that round's
// activation arena, split-K partial sums and arrival counters, so the round
// needs no device allocation. Each GPU the library runs on holds its own
// copy of the array until the process ends; every call on a GPU shares it.
#include <hip/hip_runtime.h>

#include <map>
#include <mutex>

#include "kernels.h"

namespace gemel {

namespace {

__device__ __align__(256) unsigned char scratch[GEMEL_STATIC_SCRATCH_BYTES];

struct FillArgs {
    uint32_t *p;
    uint32_t n, v;
};

__global__ __launch_bounds__(256) void fill_u32_kernel(const FillArgs a) {
    const uint32_t i = blockIdx.x * 256u + threadIdx.x;
    if (i < a.n) a.p[i] = a.v;
}

std::mutex addr_mu;
std::map<int, void *> addr;   // device -> address of that device's copy

}  // namespace

// Address of `device`'s copy of the scratch array, looked up once per device
// (the host-side name of a __device__ array is a stand-in, not a device
// address: kernels and copies must use this one). `device` must be current.
hipError_t static_scratch(int device, void **ptr) {
    std::lock_guard<std::mutex> g(addr_mu);
    auto it = addr.find(device);
    if (it != addr.end()) {
        *ptr = it->second;
        return hipSuccess;
    }
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) return e != hipSuccess ? e : hipErrorInvalidSymbol;
    addr[device] = p;
    *ptr = p;
    return hipSuccess;
}

hipError_t launch_fill_u32(uint32_t *p, size_t n, uint32_t v, const Sink &sk) {
    if (!p || n == 0 || n >= 0xffffff00ull) return hipErrorInvalidValue;
    const FillArgs a{p, (uint32_t)n, v};
    return submit(sk, reinterpret_cast<const void *>(&fill_u32_kernel), dim3((unsigned)((n + 255) / 256)), dim3(256),
                  a);
}

}  // namespace gemel
