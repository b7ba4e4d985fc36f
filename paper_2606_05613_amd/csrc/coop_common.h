// Cross-workgroup primitives of the cooperative resolve kernel.
//
// Data that one workgroup publishes for another (partial Grams, counters,
// flags, weights) crosses XCDs, whose L2 caches are not coherent with each
// other.  It moves only through agent-scope atomic loads and stores, which
// the hardware performs device-coherently (the sc1 policy: every such store
// is visible device-wide once it completes, every such load bypasses the
// non-coherent caches).  What remains is ordering, and each hand-off has a
// publish point and an observe point:
//   publish  the data stores (all issued by one wavefront), publish_point(),
//            then the relaxed atomic store or add of the flag or counter;
//   observe  relaxed polls of that word until it has the awaited value,
//            observe_point(), then the loads of the data.
// Both points are inline assembly with a "memory" clobber, so the compiler
// moves no memory access across them; publish_point() also waits for every
// vector memory access of the wavefront to complete (s_waitcnt vmcnt(0)),
// so the data stores are visible before the flag can be.  The loads after
// observe_point() are issued only after the poll loop has exited, which
// needs the polled value.  Data of other wavefronts of the publishing
// workgroup reaches the publishing one through a workgroup barrier first;
// data for other wavefronts of the consuming workgroup is loaded after a
// barrier that follows the observe point.
//
// Agent-scope release and acquire fences (__builtin_amdgcn_fence) would give
// the same order in the memory model's own terms, but on gfx950 they write
// back and invalidate the XCD's whole L2 on every hand-off: measured on
// MI355X, the K=4 bf16 MGDA workload (613 buckets of 25 MiB per row) took
// 30.7 ms per step with them against 17.5 ms with these points, the K=8
// CAGrad workload 53.1 against 39.5 ms.  The build checks the generated
// code instead (paper_2606_05613_amd/build.py, handoff_order_violations):
// each publish point's next vector memory instruction is the flag or
// counter update, and each observe point directly follows a poll loop.
#pragma once

#include "internal.h"

namespace bkmoo {

namespace {

// The marker comments let the build find these points in the generated code.
__device__ __forceinline__ void publish_point() { asm volatile("s_waitcnt vmcnt(0) ; bkmoo publish" ::: "memory"); }
__device__ __forceinline__ void observe_point() { asm volatile("; bkmoo observe" ::: "memory"); }

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
