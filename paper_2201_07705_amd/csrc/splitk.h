// Split-K partial sums and the arrival counting of the fused split-K
// reductions (conv and FC kernels).
//
// The splits of one output tile may run on different XCDs, whose L2 caches
// are not coherent with each other. Partial sums are therefore written and
// read with device-scope cache policy (sc1: the store is written through to
// the device's coherence point, the load is served from it), the access
// form the compiler itself uses for agent-scope atomics. An agent-scope
// release fence would do the same job for ordinary stores, but it writes
// back every dirty line of the XCD's L2 and, issued by every workgroup of
// a launch, costs far more than the split-K work itself.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gemel {

constexpr int kCachePolicyDevice = 16;  // sc1: device scope

// Buffer resource over `bytes` bytes of partial sums (raw addressing;
// accesses beyond `bytes` are dropped by the hardware).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t partial_rsrc(const float *p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(p), 0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ void store_partial4(__amdgpu_buffer_rsrc_t r, uint32_t byte_off, float4 v) {
    typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, v), r, byte_off, 0, kCachePolicyDevice);
}
__device__ __forceinline__ float4 load_partial4(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
    return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, kCachePolicyDevice));
}
__device__ __forceinline__ void store_partial1(float *p, float v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_partial1(const float *p) {
    return __hip_atomic_load(const_cast<float *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Arrival of one split of a split-K tile, called by every thread of the
// workgroup after its partial stores (made with the functions above). Each
// wave waits until its stores have completed at device scope, thread 0
// counts the arrival on *counter, and the workgroup that completes the
// count clears the counter for the next launch and returns true; its
// device-scope loads issued after the return see every split's partial
// sums. `flag` is one int of LDS.
__device__ __forceinline__ bool splitk_arrive(int *counter, int splits, int *flag) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (threadIdx.x == 0) {
        const int prev = __hip_atomic_fetch_add(counter, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const int last = prev == splits - 1;
        if (last) __hip_atomic_store(counter, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        *flag = last;
    }
    __syncthreads();
    return *flag != 0;
}

}  // namespace gemel
