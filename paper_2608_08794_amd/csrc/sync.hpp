// Passing values between workgroups of one launch on MI355X.  The eight
// XCDs each have their own L2, and those caches are not coherent with one
// another, so plain loads may return a stale line that another XCD has since
// written.  Agent-scope atomic loads and stores go past the L2 to the
// device's coherence point; a device-wide fence would also work but writes
// the whole XCD's L2 back, which costs tens of microseconds per kernel.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace apack {

// Relaxed agent-scope loads and stores; ordering comes from the vmcnt wait
// and workgroup barrier around them (see arrive_last).
__device__ __forceinline__ uint32_t ld_agent(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_agent(const float* p) {
  return __uint_as_float(ld_agent(reinterpret_cast<const uint32_t*>(p)));
}
__device__ __forceinline__ float2 ld_agent(const float2* p) {
  const uint64_t v =
      __hip_atomic_load(reinterpret_cast<const uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return make_float2(__uint_as_float((uint32_t)v), __uint_as_float((uint32_t)(v >> 32)));
}
__device__ __forceinline__ void st_agent(float* p, float v) {
  __hip_atomic_store(reinterpret_cast<uint32_t*>(p), __float_as_uint(v), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_agent(float2* p, float2 v) {
  const uint64_t b = (uint64_t)__float_as_uint(v.x) | ((uint64_t)__float_as_uint(v.y) << 32);
  __hip_atomic_store(reinterpret_cast<uint64_t*>(p), b, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Arrival at a counter of `expected` workgroups; true in the last one to
// arrive (all threads of the workgroup get the same answer).  Every thread
// first waits until its own vector memory operations have completed, so the
// results the workgroup wrote with agent-scope stores or device atomics are
// visible before its arrival counts; the last workgroup reads them with
// agent-scope loads.  A full device fence here would also write back the
// XCD's L2, which costs far more on this chip.
template <int NT>
__device__ __forceinline__ bool arrive_last(uint32_t* counter, uint32_t expected) {
  __shared__ bool last;
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (threadIdx.x == 0)
    last = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == expected - 1;
  __syncthreads();
  return last;
}

}  // namespace apack
