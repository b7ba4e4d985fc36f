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

// The same with K fixed at compile time: MGDA and CAGrad run the
// lane-parallel solvers (lane i holds task i's row, O(K) arithmetic per
// step and lane), PCGrad, the mean and non-finite Grams the sequential
// code above.  A K = 2 MGDA FW-20 solve of four buckets took 12.7 us with
// the sequential code, most of the smallest workload's step.
template <int K>
__global__ __launch_bounds__(kWave) void lane_solve_kernel(const double *__restrict__ gram, int method,
                                                           int iters, double c,
                                                           const int8_t *__restrict__ order,
                                                           float *__restrict__ weights,
                                                           double *__restrict__ aux) {
  __shared__ Shared S;
  const int64_t b = blockIdx.x;
  const int t = threadIdx.x;
  solver_load_gram<WaveSync>(S, K, gram + b * K * K, t, kWave);
  double wt = 0.0, ax = 0.0;
  if (S.bad || (method != MGDA && method != CAGRAD))
    solver_run<WaveSync>(S, K, method, iters, c, order, b, t, &wt, &ax);
  else if (method == MGDA)
    wt = ax = lane_solve_mgda<K>(S.G, iters, t);
  else
    lane_solve_cagrad<K>(S.G, iters, c, t, &wt, &ax);
  if (t < K) {
    weights[b * K + t] = (float)wt;
    if (aux) aux[b * K + t] = ax;
  }
}

template <int K>
void launch_lane_solve(int B, const double *gram, int method, int max_iter, double c, const int8_t *order,
                       float *weights, double *aux, hipStream_t s) {
  hipLaunchKernelGGL(lane_solve_kernel<K>, dim3((unsigned)B), dim3(kWave), 0, s, gram, method, max_iter, c,
                     order, weights, aux);
}

}  // namespace

hipError_t launch_solve(int K, int B, const double *gram, int method, int max_iter, double c,
                        const int8_t *order, float *weights, double *aux, hipStream_t s) {
  if (method == MGDA_EXACT || method == CAGRAD_EXACT)
    return launch_exact_solve(K, B, gram, method, c, weights, aux, s);
  switch (K) {
    case 2: launch_lane_solve<2>(B, gram, method, max_iter, c, order, weights, aux, s); break;
    case 3: launch_lane_solve<3>(B, gram, method, max_iter, c, order, weights, aux, s); break;
    case 4: launch_lane_solve<4>(B, gram, method, max_iter, c, order, weights, aux, s); break;
    case 5: launch_lane_solve<5>(B, gram, method, max_iter, c, order, weights, aux, s); break;
    case 6: launch_lane_solve<6>(B, gram, method, max_iter, c, order, weights, aux, s); break;
    case 7: launch_lane_solve<7>(B, gram, method, max_iter, c, order, weights, aux, s); break;
    case 8: launch_lane_solve<8>(B, gram, method, max_iter, c, order, weights, aux, s); break;
    case 9: launch_lane_solve<9>(B, gram, method, max_iter, c, order, weights, aux, s); break;
    case 10: launch_lane_solve<10>(B, gram, method, max_iter, c, order, weights, aux, s); break;
    default:
      hipLaunchKernelGGL(solve_kernel, dim3((unsigned)B), dim3(kWave), 0, s, K, gram, method, max_iter, c,
                         order, weights, aux);
  }
  return hipGetLastError();
}

}  // namespace bkmoo
