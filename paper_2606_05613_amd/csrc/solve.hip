// The per-bucket MOO subproblem, solved from the bucket's Gram matrix alone.
//
// One wavefront per bucket, everything in fp64 in LDS and registers.  Lanes
// t < K do the per-task work (rows of G times a vector, PCGrad's task rows);
// the scalar parts of each step (argmin with lowest-index ties, line
// searches) run identically on every lane, reading LDS broadcasts, so no
// cross-lane reduction order can change a decision.  This file is compiled
// without floating-point contraction so every scalar expression rounds
// exactly as written.
#include "internal.h"

namespace bkmoo {

namespace {

enum Method : int { MGDA = 0, PCGRAD = 1, CAGRAD = 2, MEAN = 3 };

// min over gamma in [0, 1] of |gamma a + (1 - gamma) b|^2 from aa, ab, bb
// (Eq. mgda restricted to a segment): the stationary point
// (bb - ab) / (aa - 2ab + bb), clipped; gamma = 1 when a = b.
__device__ __forceinline__ double pair_gamma(double aa, double ab, double bb) {
  const double den = aa - 2.0 * ab + bb;
  if (den <= 0.0) return 1.0;
  double g = (bb - ab) / den;
  g = g < 0.0 ? 0.0 : g;
  return g > 1.0 ? 1.0 : g;
}

__device__ __forceinline__ double pair_value(double g, double aa, double ab, double bb) {
  return g * g * aa + 2.0 * g * (1.0 - g) * ab + (1.0 - g) * (1.0 - g) * bb;
}

struct Shared {
  double G[kMaxK * kMaxK];
  double C[kMaxK * kMaxK];  // PCGrad coefficient rows
  double a[kMaxK];          // simplex variable
  double v[kMaxK];          // G a
  double bvec[kMaxK];       // CAGrad: G 1 / K
  int bad;
};

// MGDA: Frank-Wolfe on min_{a in simplex} a^T G a (Eq. shard-mgda), started
// on the best pair of tasks, fixed iteration count.
__device__ void solve_mgda(Shared &S, int K, int iters, int t) {
  if (t == 0) {
    double best = 0.0, bg = 1.0;
    int bi = 0, bj = 1;
    bool first = true;
    for (int i = 0; i < K; ++i)
      for (int j = i + 1; j < K; ++j) {
        const double aa = S.G[i * K + i], ab = S.G[i * K + j], bb = S.G[j * K + j];
        const double g = pair_gamma(aa, ab, bb);
        const double val = pair_value(g, aa, ab, bb);
        if (first || val < best) {
          first = false;
          best = val;
          bi = i;
          bj = j;
          bg = g;
        }
      }
    for (int i = 0; i < K; ++i) S.a[i] = 0.0;
    S.a[bi] = bg;
    S.a[bj] = 1.0 - bg;
  }
  __syncthreads();
  for (int it = 0; it < iters; ++it) {
    if (t < K) {
      double s = 0.0;
      for (int j = 0; j < K; ++j) s += S.G[t * K + j] * S.a[j];
      S.v[t] = s;
    }
    __syncthreads();
    int ts = 0;
    double m = S.v[0];
    for (int i = 1; i < K; ++i)
      if (S.v[i] < m) {
        m = S.v[i];
        ts = i;
      }
    double aa = 0.0;
    for (int i = 0; i < K; ++i) aa += S.a[i] * S.v[i];
    const double g = pair_gamma(aa, S.v[ts], S.G[ts * K + ts]);
    __syncthreads();
    if (t < K) {
      double na = g * S.a[t];
      if (t == ts) na += 1.0 - g;
      S.a[t] = na;
    }
    __syncthreads();
  }
}

// PCGrad (Algorithm 1): lane t owns task t's coefficient row; a projection
// of d_t off g_j only changes C[t][j], and every inner product uses the
// original g_j, so the K tasks are independent.
__device__ void solve_pcgrad(Shared &S, int K, const int8_t *order, int b, int t) {
  if (t < K) {
    for (int i = 0; i < K; ++i) S.C[t * K + i] = i == t ? 1.0 : 0.0;
    uint32_t seen = 1u << t;
    for (int q = 0; q < K - 1; ++q) {
      int j = q < t ? q : q + 1;
      if (order) {
        j = order[((int64_t)b * K + t) * (K - 1) + q];
        if (j < 0 || j >= K || ((seen >> j) & 1u)) {
          S.bad = 1;
          break;
        }
        seen |= 1u << j;
      }
      double p = 0.0;
      for (int i = 0; i < K; ++i) p += S.C[t * K + i] * S.G[i * K + j];
      if (p < 0.0) S.C[t * K + j] -= p / S.G[j * K + j];
    }
  }
  __syncthreads();
  if (t < K) {
    double w = 0.0;
    for (int r = 0; r < K; ++r) w += S.C[r * K + t];
    S.a[t] = w;
  }
  __syncthreads();
}

// CAGrad through its dual min_{w in simplex} F(w) = b^T w + r sqrt(w^T G w)
// (b = G 1 / K, r = c |g_avg|), Frank-Wolfe from the uniform point with an
// exact line search; primal d = g_avg + r g_w / |g_w|.
__device__ void solve_cagrad(Shared &S, int K, int iters, double c, int t) {
  const double invK = 1.0 / (double)K;
  if (t < K) {
    double s = 0.0;
    for (int j = 0; j < K; ++j) s += S.G[t * K + j];
    S.bvec[t] = s / (double)K;
    S.a[t] = invK;
  }
  __syncthreads();
  double tot = 0.0;
  for (int i = 0; i < K * K; ++i) tot += S.G[i];
  double g0sq = tot / (double)(K * K);
  g0sq = g0sq > 0.0 ? g0sq : 0.0;
  const double r = c * sqrt(g0sq);

  for (int it = 0; it < iters; ++it) {
    if (t < K) {
      double s = 0.0;
      for (int j = 0; j < K; ++j) s += S.G[t * K + j] * S.a[j];
      S.v[t] = s;
    }
    __syncthreads();
    double cq = 0.0, bw = 0.0;
    for (int i = 0; i < K; ++i) cq += S.a[i] * S.v[i];
    for (int i = 0; i < K; ++i) bw += S.bvec[i] * S.a[i];
    const double nrm = sqrt(cq > 0.0 ? cq : 0.0);
    int sidx = 0;
    double m = 0.0;
    for (int i = 0; i < K; ++i) {
      const double gi = S.bvec[i] + (nrm > 1e-300 ? r * S.v[i] / nrm : 0.0);
      if (i == 0 || gi < m) {
        m = gi;
        sidx = i;
      }
    }
    const double beta1 = S.bvec[sidx] - bw;
    const double A = S.G[sidx * K + sidx] - 2.0 * S.v[sidx] + cq;
    const double Bq = S.v[sidx] - cq;
    double cand[4] = {0.0, 1.0, 0.0, 0.0};
    int nc = 2;
    const double D = r * r * A - beta1 * beta1;
    if (A > 0.0 && D > 0.0) {
      const double disc = (A * cq - Bq * Bq) / D;
      if (disc >= 0.0) {
        const double root = fabs(beta1) * sqrt(disc);
        const double g1 = (-Bq - root) / A, g2 = (-Bq + root) / A;
        if (g1 > 0.0 && g1 < 1.0) cand[nc++] = g1;
        if (g2 > 0.0 && g2 < 1.0) cand[nc++] = g2;
      }
    }
    // ascending order, then the first least F
    for (int i = 1; i < nc; ++i)
      for (int j = i; j > 0 && cand[j] < cand[j - 1]; --j) {
        const double tmp = cand[j];
        cand[j] = cand[j - 1];
        cand[j - 1] = tmp;
      }
    double gamma = cand[0], fbest = 0.0;
    for (int i = 0; i < nc; ++i) {
      const double g = cand[i];
      double q = A * g * g + 2.0 * Bq * g + cq;
      q = q > 0.0 ? q : 0.0;
      const double f = bw + beta1 * g + r * sqrt(q);
      if (i == 0 || f < fbest) {
        fbest = f;
        gamma = g;
      }
    }
    __syncthreads();
    if (t < K) {
      double na = (1.0 - gamma) * S.a[t];
      if (t == sidx) na += gamma;
      S.a[t] = na;
    }
    __syncthreads();
  }
  // primal weights
  if (t < K) {
    double s = 0.0;
    for (int j = 0; j < K; ++j) s += S.G[t * K + j] * S.a[j];
    S.v[t] = s;
  }
  __syncthreads();
  double q = 0.0, dmax = 0.0;
  for (int i = 0; i < K; ++i) q += S.a[i] * S.v[i];
  for (int i = 0; i < K; ++i) dmax = S.G[i * K + i] > dmax ? S.G[i * K + i] : dmax;
  const double nrm = sqrt(q > 0.0 ? q : 0.0);
  const double scale = sqrt(dmax);
  const bool degenerate = r == 0.0 || nrm <= 1e-12 * scale || nrm == 0.0;
  __syncthreads();
  if (t < K) S.C[t] = degenerate ? invK : invK + (r / nrm) * S.a[t];  // weights
  __syncthreads();
}

__global__ __launch_bounds__(kWave) void solve_kernel(int K, const double *__restrict__ gram,
                                                      int method, int iters, double c,
                                                      const int8_t *__restrict__ order,
                                                      float *__restrict__ weights,
                                                      double *__restrict__ aux) {
  __shared__ Shared S;
  const int b = blockIdx.x;
  const int t = threadIdx.x;
  if (t == 0) S.bad = 0;
  __syncthreads();
  for (int i = t; i < K * K; i += kWave) {
    const double g = gram[(int64_t)b * K * K + i];
    S.G[i] = g;
    if (!__builtin_isfinite(g)) S.bad = 1;
  }
  __syncthreads();
  const double nan = __builtin_nan("");
  if (S.bad) {
    if (t < K) {
      weights[(int64_t)b * K + t] = (float)nan;
      if (aux) aux[(int64_t)b * K + t] = nan;
    }
    return;
  }
  double wt = 0.0, ax = 0.0;
  switch (method) {
    case MGDA:
      solve_mgda(S, K, iters, t);
      if (t < K) wt = ax = S.a[t];
      break;
    case PCGRAD:
      solve_pcgrad(S, K, order, b, t);
      if (t < K) wt = ax = S.bad ? nan : S.a[t];
      break;
    case CAGRAD:
      solve_cagrad(S, K, iters, c, t);
      if (t < K) {
        wt = S.C[t];
        ax = S.a[t];
      }
      break;
    default:
      wt = ax = 1.0 / (double)K;
      break;
  }
  if (t < K) {
    weights[(int64_t)b * K + t] = (float)wt;
    if (aux) aux[(int64_t)b * K + t] = ax;
  }
}

}  // namespace

hipError_t launch_solve(int K, int B, const double *gram, int method, int max_iter, double c,
                        const int8_t *order, float *weights, double *aux, hipStream_t s) {
  hipLaunchKernelGGL(solve_kernel, dim3((unsigned)B), dim3(kWave), 0, s, K, gram, method, max_iter,
                     c, order, weights, aux);
  return hipGetLastError();
}

}  // namespace bkmoo
