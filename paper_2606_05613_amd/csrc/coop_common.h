// Cross-workgroup primitives of the cooperative resolve kernels.
//
// Data that one workgroup publishes for another (partial Grams, counters,
// flags, weights) crosses XCDs, whose L2 caches are not coherent with each
// other.  It moves only through agent-scope atomic loads and stores, which
// the hardware performs device-coherently (the sc1 policy); a writer drains
// its own stores (vmcnt = 0) before it moves a counter or a flag that
// releases them, and a reader issues its loads only after observing that
// counter or flag.
#pragma once

#include "internal.h"

namespace bkmoo {

namespace {

// Wait until every vector memory access this wavefront issued has completed
// (vmcnt = 0; expcnt and lgkmcnt left unconstrained).
__device__ __forceinline__ void wait_vm_complete() { __builtin_amdgcn_s_waitcnt(0x0F70); }

template <typename T>
__device__ __forceinline__ void store_agent(T *p, T v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename T>
__device__ __forceinline__ T load_agent(const T *p) {
  return __hip_atomic_load(const_cast<T *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace

}  // namespace bkmoo
