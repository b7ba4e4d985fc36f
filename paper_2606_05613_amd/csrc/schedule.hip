// Bucket schedule: validates the bucket offsets and cuts every bucket into
// chunks of C elements that never straddle a bucket boundary (the partition
// of the parameter vector into disjoint contiguous buckets, Section 3.2).
#include "internal.h"

namespace bkmoo {

namespace {

constexpr int kSchedThreads = 1024;

// One workgroup.  chunk_start[b] = sum_{b' < b} ceil(n_b' / C) and, when
// group_start is given, group_start[b] = sum_{b' < b} ceil(chunks_b' / G)
// (groups of G consecutive chunks of one bucket, the Gram finalize's unit).
// On invalid offsets every entry is 0 (so no chunk is processed) and the
// error word gets kErrOffsets.  Otherwise the error word is cleared.
__global__ __launch_bounds__(kSchedThreads) void schedule_kernel(
    const int64_t *__restrict__ offs, int B, int64_t N, int64_t C, int64_t *__restrict__ cs,
    int64_t G, int64_t *__restrict__ gs, uint32_t *__restrict__ err, uint32_t *__restrict__ sync,
    int64_t nsync) {
  __shared__ int bad;
  __shared__ int64_t scan_c[kSchedThreads];
  __shared__ int64_t scan_g[kSchedThreads];
  __shared__ int64_t carry_c, carry_g;
  const int tid = threadIdx.x;
  for (int64_t i = tid; i < nsync; i += kSchedThreads) sync[i] = 0u;
  if (tid == 0) {
    bad = (offs[0] != 0 || offs[B] != N) ? 1 : 0;
    carry_c = 0;
    carry_g = 0;
  }
  __syncthreads();
  for (int b = tid; b < B; b += kSchedThreads)
    if (offs[b + 1] < offs[b]) bad = 1;
  __syncthreads();
  if (bad) {
    for (int b = tid; b <= B; b += kSchedThreads) {
      cs[b] = 0;
      if (gs) gs[b] = 0;
    }
    if (tid == 0) *err = kErrOffsets;
    return;
  }
  for (int base = 0; base < B; base += kSchedThreads) {
    const int b = base + tid;
    const int64_t n = b < B ? offs[b + 1] - offs[b] : 0;
    const int64_t cnt = (n + C - 1) / C;
    const int64_t gcnt = (cnt + G - 1) / G;
    scan_c[tid] = cnt;
    scan_g[tid] = gcnt;
    __syncthreads();
    // Hillis-Steele inclusive scans over the tile
    for (int d = 1; d < kSchedThreads; d <<= 1) {
      const int64_t add_c = tid >= d ? scan_c[tid - d] : 0;
      const int64_t add_g = tid >= d ? scan_g[tid - d] : 0;
      __syncthreads();
      scan_c[tid] += add_c;
      scan_g[tid] += add_g;
      __syncthreads();
    }
    if (b < B) {
      cs[b] = carry_c + scan_c[tid] - cnt;
      if (gs) gs[b] = carry_g + scan_g[tid] - gcnt;
    }
    __syncthreads();
    if (tid == kSchedThreads - 1) {
      carry_c += scan_c[tid];
      carry_g += scan_g[tid];
    }
    __syncthreads();
  }
  if (tid == 0) {
    cs[B] = carry_c;
    if (gs) gs[B] = carry_g;
    *err = 0u;
  }
}

}  // namespace

hipError_t launch_schedule(const int64_t *offsets, int B, int64_t N, int64_t C, int64_t *chunk_start,
                           int64_t *group_start, uint32_t *err, uint32_t *sync, int64_t nsync,
                           hipStream_t s) {
  hipLaunchKernelGGL(schedule_kernel, dim3(1), dim3(kSchedThreads), 0, s, offsets, B, N, C,
                     chunk_start, (int64_t)kFinalizeGroup, group_start, err, sync, nsync);
  return hipGetLastError();
}

}  // namespace bkmoo
