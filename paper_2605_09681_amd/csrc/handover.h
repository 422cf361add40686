// handover.h -- passing values between the workgroups of one launch: the
// scoring reduction, the in-kernel merge of cut attention items and the FP8
// statistics all end with "the last workgroup to arrive combines what the
// others wrote".
//
// Values another workgroup of the same launch reads are written and read with
// device-scope accesses (sc1: coherent across the XCDs' L2 caches for that
// location), so the hand-over needs no cache write-back or invalidation: a
// generic agent-scope release or acquire fence writes back or invalidates the
// whole L2 of the XCD (measured ~1 us, serialised per XCD, when every
// workgroup does it).
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace fkv {

__device__ __forceinline__ void put_shared(double *p, double v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ double get_shared(const double *p) {
    return __hip_atomic_load(const_cast<double *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void put_shared(float *p, float v) {
    __hip_atomic_store((uint32_t *)p, __float_as_uint(v), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float get_shared(const float *p) {
    return __uint_as_float(
        __hip_atomic_load(const_cast<uint32_t *>((const uint32_t *)p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
}
__device__ __forceinline__ void put_shared(unsigned long long *p, uint2 v) {
    __hip_atomic_store(p, ((unsigned long long)v.y << 32) | v.x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint2 get_shared(const uint2 *p) {
    const unsigned long long v = __hip_atomic_load(const_cast<unsigned long long *>((const unsigned long long *)p),
                                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return make_uint2((uint32_t)v, (uint32_t)(v >> 32));
}

// Arrival on a device-scope counter; true in every thread of the workgroup
// that arrives last (which resets the counter to zero for the next call).
// Every wave first waits until its own stores have completed, so the last
// arrival sees all of them (and, through a chain of arrivals, everything the
// earlier arrivals saw).  flag: one word of LDS.  Every thread of the
// workgroup calls it (it contains barriers).
__device__ __forceinline__ bool arrive_last(uint32_t *counter, uint32_t expected, uint32_t *flag) {
    __builtin_amdgcn_s_waitcnt(0);   // this wave's stores (vmcnt), LDS and scalar accesses complete
    __syncthreads();
    if (threadIdx.x == 0) {
        const uint32_t old = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const bool last = old + 1 == expected;
        if (last) __hip_atomic_store(counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        *flag = last ? 1u : 0u;
    }
    __syncthreads();
    return *flag != 0;
}

}  // namespace fkv
