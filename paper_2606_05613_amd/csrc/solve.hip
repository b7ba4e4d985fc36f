// The per-bucket MOO subproblem, solved from the bucket's Gram matrix alone.
//
// One wavefront per bucket, everything in fp64 in LDS and registers (the
// solvers are in solve_impl.h).  This file is compiled without
// floating-point contraction so every scalar expression rounds exactly as
// written.
#include "solve_impl.h"

namespace bkmoo {

namespace {

__global__ __launch_bounds__(kWave) void solve_kernel(int K, const double *__restrict__ gram,
                                                      int method, int iters, double c,
                                                      const int8_t *__restrict__ order,
                                                      float *__restrict__ weights,
                                                      double *__restrict__ aux) {
  __shared__ Shared S;
  const int64_t b = blockIdx.x;
  const int t = threadIdx.x;
  solver_load_gram<WaveSync>(S, K, gram + b * K * K, t, kWave);
  double wt, ax;
  solver_run<WaveSync>(S, K, method, iters, c, order, b, t, &wt, &ax);
  if (t < K) {
    weights[b * K + t] = (float)wt;
    if (aux) aux[b * K + t] = ax;
  }
}

}  // namespace

hipError_t launch_solve(int K, int B, const double *gram, int method, int max_iter, double c,
                        const int8_t *order, float *weights, double *aux, hipStream_t s) {
  if (method == MGDA_EXACT || method == CAGRAD_EXACT)
    return launch_exact_solve(K, B, gram, method, c, weights, aux, s);
  hipLaunchKernelGGL(solve_kernel, dim3((unsigned)B), dim3(kWave), 0, s, K, gram, method, max_iter,
                     c, order, weights, aux);
  return hipGetLastError();
}

}  // namespace bkmoo
