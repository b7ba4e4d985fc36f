// Per-bucket gradient-conflict diagnostics from the Gram matrices.
//
// Two task gradients conflict when their inner product (equivalently their
// cosine similarity) is negative (Section 2.1 and the appendix definition of
// conflicting gradients).  Figure 1 follows the mean and spread of the
// pairwise cosines and counts a conflict at a step when some pair is
// negative; per bucket these are the statistics below.  They read only the
// K x K Gram matrices the Gram pass already produced: B*K*K*8 bytes, no
// gradient traffic.  One thread per bucket walks the pairs i < j in
// lexicographic order in fp64.
#include "internal.h"

namespace bkmoo {

namespace {

constexpr int kConflictThreads = 64;

// Cosine of tasks i != j: G_ij / sqrt(G_ii G_jj) clipped to [-1, 1]; 0 when
// either gradient is zero.
__device__ __forceinline__ double pair_cos(const double *G, int K, int i, int j) {
  const double gii = G[i * K + i], gjj = G[j * K + j];
  if (!(gii > 0.0) || !(gjj > 0.0)) return 0.0;
  const double c = G[i * K + j] / sqrt(gii * gjj);
  return c < -1.0 ? -1.0 : (c > 1.0 ? 1.0 : c);
}

__global__ __launch_bounds__(kConflictThreads) void conflicts_kernel(
    int K, int B, const double *__restrict__ gram, double *__restrict__ cosines,
    double *__restrict__ summary, int32_t *__restrict__ pairs) {
  const int b = blockIdx.x * kConflictThreads + threadIdx.x;
  if (b >= B) return;
  const double *G = gram + (int64_t)b * K * K;
  double *cb = cosines ? cosines + (int64_t)b * K * K : nullptr;

  bool finite = true;
  for (int q = 0; q < K * K; ++q) finite = finite && __builtin_isfinite(G[q]);
  if (!finite) {
    const double nan = __builtin_nan("");
    if (cb)
      for (int q = 0; q < K * K; ++q) cb[q] = nan;
    if (summary) summary[3 * b] = summary[3 * b + 1] = summary[3 * b + 2] = nan;
    if (pairs) pairs[3 * b] = pairs[3 * b + 1] = pairs[3 * b + 2] = -1;
    return;
  }

  const int npairs = K * (K - 1) / 2;
  double sum = 0.0, best = 0.0;
  int bi = -1, bj = -1, count = 0;
  for (int i = 0; i < K; ++i) {
    if (cb) cb[i * K + i] = G[i * K + i] > 0.0 ? 1.0 : 0.0;
    for (int j = i + 1; j < K; ++j) {
      const double c = pair_cos(G, K, i, j);
      if (cb) cb[i * K + j] = cb[j * K + i] = c;
      sum += c;
      if (G[i * K + j] < 0.0) ++count;
      if (bi < 0 || c < best) {
        best = c;
        bi = i;
        bj = j;
      }
    }
  }
  if (summary) {
    const double mean = sum / npairs;
    double ss = 0.0;
    for (int i = 0; i < K; ++i)
      for (int j = i + 1; j < K; ++j) {
        const double d = pair_cos(G, K, i, j) - mean;
        ss += d * d;
      }
    summary[3 * b] = mean;
    summary[3 * b + 1] = sqrt(ss / npairs);
    summary[3 * b + 2] = best;
  }
  if (pairs) {
    pairs[3 * b] = bi;
    pairs[3 * b + 1] = bj;
    pairs[3 * b + 2] = count;
  }
}

}  // namespace

hipError_t launch_conflicts(int K, int B, const double *gram, double *cosines, double *summary,
                            int32_t *pairs, hipStream_t s) {
  const unsigned grid = (unsigned)((B + kConflictThreads - 1) / kConflictThreads);
  hipLaunchKernelGGL(conflicts_kernel, dim3(grid), dim3(kConflictThreads), 0, s, K, B, gram, cosines,
                     summary, pairs);
  return hipGetLastError();
}

}  // namespace bkmoo
