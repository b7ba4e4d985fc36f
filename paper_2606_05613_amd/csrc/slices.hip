// Bucket slices and the slice-order sum of partial Gram matrices.
//
// Inner products add over disjoint pieces of a vector (Eq. decomp), so a
// bucket's Gram matrix is the sum of the Gram matrices of any partition of
// the bucket.  Cutting every bucket into T slices gives the pieces T ranks
// would each hold after exchanging bucket slices: each rank computes the
// partial Grams of its slices with the ordinary Gram pass, the partials are
// gathered, and every rank adds them in rank order, which is deterministic
// and identical everywhere.  On one GPU the same two calls run the sliced
// computation at its real slice shapes: the Gram pass over the B*T slice
// offsets (bucket-major), then the reduction.
#include "internal.h"

namespace bkmoo {

namespace {

constexpr int kSliceThreads = 256;

// slice t of bucket b starts at o_b + floor(t n_b / T); with n_b = q T + r
// that is o_b + t q + floor(t r / T), which never overflows.
__global__ __launch_bounds__(kSliceThreads) void slice_offsets_kernel(
    const int64_t *__restrict__ offs, int B, int T, int64_t *__restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * kSliceThreads + threadIdx.x;
  const int64_t total = (int64_t)B * T;
  if (i < total) {
    const int64_t b = i / T, t = i % T;
    const int64_t n = offs[b + 1] - offs[b];
    const int64_t q = n / T, r = n % T;
    out[i] = offs[b] + t * q + (t * r) / T;
  }
  if (i == 0) out[total] = offs[B];
}

// gram[b][e] = sum over t = 0..T-1, in that order, of the slice partials;
// rank-major partial[t][b][e] or bucket-major partial[b][t][e], e < K*K.
__global__ __launch_bounds__(kSliceThreads) void gram_reduce_kernel(
    int KK, int B, int T, const double *__restrict__ partial, int bucket_major,
    double *__restrict__ gram) {
  const int64_t i = (int64_t)blockIdx.x * kSliceThreads + threadIdx.x;
  if (i >= (int64_t)B * KK) return;
  const int64_t b = i / KK, e = i % KK;
  const int64_t step = bucket_major ? KK : (int64_t)B * KK;
  const double *p = partial + (bucket_major ? b * T * KK : b * KK) + e;
  double s = p[0];
  for (int t = 1; t < T; ++t) s += p[t * step];
  gram[i] = s;
}

}  // namespace

hipError_t launch_slice_offsets(const int64_t *offsets, int B, int T, int64_t *out, hipStream_t s) {
  const int64_t total = (int64_t)B * T + 1;
  const unsigned grid = (unsigned)((total + kSliceThreads - 1) / kSliceThreads);
  hipLaunchKernelGGL(slice_offsets_kernel, dim3(grid), dim3(kSliceThreads), 0, s, offsets, B, T, out);
  return hipGetLastError();
}

hipError_t launch_gram_reduce(int K, int B, int T, const double *partial, int bucket_major, double *gram,
                              hipStream_t s) {
  const int64_t total = (int64_t)B * K * K;
  const unsigned grid = (unsigned)((total + kSliceThreads - 1) / kSliceThreads);
  hipLaunchKernelGGL(gram_reduce_kernel, dim3(grid), dim3(kSliceThreads), 0, s, K * K, B, T, partial,
                     bucket_major, gram);
  return hipGetLastError();
}

}  // namespace bkmoo
