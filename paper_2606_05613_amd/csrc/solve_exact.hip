// Exact solvers for the per-bucket problems, by support enumeration: the
// minimum-norm point of the simplex hull of the task gradients (Eq. mgda /
// Eq. shard-mgda over the simplex) and the minimiser of the CAGrad dual
// F(w) = b^T w + r ||g_w|| over the simplex (the local problem of Eq.
// cagrad through its dual), both from the bucket's Gram matrix alone.
//
// One wavefront per bucket, fp64, K <= 10.  The 2^K - 1 supports S are
// spread over the 64 lanes.  Each lane writes its support's small linear
// system into LDS (the 64 lanes' copies interleaved, so one access of the
// wavefront touches 64 consecutive words) and solves it by Gaussian
// elimination with partial pivoting; a support whose system has an exactly
// zero pivot is skipped.  Candidates are ranked in the order "by support
// size, then lexicographically", which fixes every tie-break:
//
// MGDA.  On S the stationarity conditions G_SS a_S = mu 1, 1^T a_S = 1 form
// a bordered (|S|+1)-square system (non-singular exactly when the g_t, t in
// S, are affinely independent, which the smallest optimal support is).  A
// solution is kept if a_S >= -1e-10 and |sum a_S - 1| <= 1e-9; clipped at 0
// and renormalised it must satisfy (G a)_t >= a^T G a - 1e-9 for every t
// (the minimum-norm property); G is first divided by its largest diagonal
// entry.  Scanning the kept candidates in rank order, a later one replaces
// the current choice only if its a^T G a is smaller by more than 1e-12.  If
// none is kept (numerically degenerate input), 5000 Frank-Wolfe iterations
// of the iterative solver stand in.
//
// CAGrad.  Candidates are the K vertices and, when r > 0, for every S with
// |S| >= 2 the points v_S = G_SS^{-1} (lam 1 - b_S) / r for the two roots
// lam of v_S^T G_SS v_S = 1 (a quadratic in lam), kept if v_S >= -1e-12 and
// sum v_S > 0, clipped at 0 and normalised onto the simplex.  The candidate
// of least F wins, the first in rank order (vertices first, smaller root
// first) on exact ties.
#include "solve_impl.h"

namespace bkmoo {

namespace {

__device__ __forceinline__ int binom(int n, int k) {
  if (k < 0 || k > n) return 0;
  int r = 1;
  for (int i = 1; i <= k; ++i) r = r * (n - k + i) / i;  // C(n-k+i, i), exact
  return r;
}

// Position of support `m` (bit t = task t) among the non-empty subsets of
// {0..K-1} ordered by size, then lexicographically.
__device__ int support_rank(uint32_t m, int K) {
  const int s = __builtin_popcount(m);
  int r = 0;
  for (int t = 1; t < s; ++t) r += binom(K, t);
  int prev = -1, i = 0;
  for (int c = 0; c < K; ++c)
    if ((m >> c) & 1u) {
      ++i;
      for (int j = prev + 1; j < c; ++j) r += binom(K - 1 - j, s - i);
      prev = c;
    }
  return r;
}

// This lane's matrix, rows of `stride` entries: entry (r, c) at
// M[(r * stride + c) * kWave].
struct LaneMat {
  double *M;
  int stride;
  __device__ __forceinline__ double &operator()(int r, int c) const {
    return M[(r * stride + c) * kWave];
  }
};

// Gaussian elimination with partial pivoting (the first entry of largest
// magnitude) on an n x ncols augmented matrix (ncols - n right-hand sides).
// False if a pivot is exactly zero; otherwise the solutions overwrite
// columns n .. ncols - 1.
__device__ bool lane_solve(const LaneMat &A, int n, int ncols) {
  for (int k = 0; k < n; ++k) {
    int p = k;
    double pv = fabs(A(k, k));
    for (int r = k + 1; r < n; ++r) {
      const double v = fabs(A(r, k));
      if (v > pv) {
        pv = v;
        p = r;
      }
    }
    if (pv == 0.0) return false;
    if (p != k)
      for (int c = k; c < ncols; ++c) {
        const double tmp = A(k, c);
        A(k, c) = A(p, c);
        A(p, c) = tmp;
      }
    const double piv = A(k, k);
    for (int r = k + 1; r < n; ++r) {
      const double f = A(r, k) / piv;
      for (int c = k + 1; c < ncols; ++c) A(r, c) -= f * A(k, c);
      A(r, k) = 0.0;
    }
  }
  for (int j = n; j < ncols; ++j)
    for (int r = n - 1; r >= 0; --r) {
      double s = A(r, j);
      for (int c = r + 1; c < n; ++c) s -= A(r, c) * A(c, j);
      A(r, j) = s / A(r, r);
    }
  return true;
}

// MGDA on support m of the normalised Gram Gn: solves the bordered system
// and runs the feasibility and minimum-norm checks.  On success the support's
// simplex weights (clipped, renormalised) are in column |S|+1 of rows
// 0..|S|-1, in increasing task order, and *q = a^T Gn a.
__device__ bool mgda_support(const double *Gn, int K, uint32_t m, const LaneMat &A, double *q) {
  int idx[kExactMaxK];
  int s = 0;
  for (int t = 0; t < K; ++t)
    if ((m >> t) & 1u) idx[s++] = t;
  const int n = s + 1, sol = s + 1;
  for (int u = 0; u < s; ++u) {
    for (int v = 0; v < s; ++v) A(u, v) = Gn[idx[u] * K + idx[v]];
    A(u, s) = 1.0;
    A(u, sol) = 0.0;
  }
  for (int v = 0; v < s; ++v) A(s, v) = 1.0;
  A(s, s) = 0.0;
  A(s, sol) = 1.0;
  if (!lane_solve(A, n, s + 2)) return false;
  double amin = s < K ? 0.0 : A(0, sol), sum = 0.0;
  for (int u = 0; u < s; ++u) {
    const double a = A(u, sol);
    amin = a < amin ? a : amin;
    sum += a;
  }
  if (!(amin >= -1e-10) || !(fabs(sum - 1.0) <= 1e-9)) return false;
  double csum = 0.0;
  for (int u = 0; u < s; ++u) {
    const double a = A(u, sol) > 0.0 ? A(u, sol) : 0.0;
    A(u, sol) = a;
    csum += a;
  }
  for (int u = 0; u < s; ++u) A(u, sol) = A(u, sol) / csum;
  // (Gn a)_t over every task, a^T Gn a, and the minimum-norm check
  double qq = 0.0;
  for (int u = 0; u < s; ++u) {
    double g = 0.0;
    for (int v = 0; v < s; ++v) g += Gn[idx[u] * K + idx[v]] * A(v, sol);
    qq += A(u, sol) * g;
  }
  for (int t = 0; t < K; ++t) {
    double g = 0.0;
    for (int v = 0; v < s; ++v) g += Gn[t * K + idx[v]] * A(v, sol);
    if (!(g >= qq - 1e-9)) return false;
  }
  *q = qq;
  return true;
}

// CAGrad candidate `root` (0: smaller lam, 1: larger) on support m (|m| >= 2):
// on success the simplex point w_S is in column |S| of rows 0..|S|-1 and *F is
// its dual objective.
__device__ bool cagrad_support(const double *G, const double *bvec, double r, int K, uint32_t m,
                               int root, const LaneMat &A, double *F) {
  int idx[kExactMaxK];
  int s = 0;
  for (int t = 0; t < K; ++t)
    if ((m >> t) & 1u) idx[s++] = t;
  const int c1 = s, cb = s + 1;  // columns of H 1 and H b_S
  for (int u = 0; u < s; ++u) {
    for (int v = 0; v < s; ++v) A(u, v) = G[idx[u] * K + idx[v]];
    A(u, c1) = 1.0;
    A(u, cb) = bvec[idx[u]];
  }
  if (!lane_solve(A, s, s + 2)) return false;
  double qa = 0.0, h1b = 0.0, hbb = 0.0;
  for (int u = 0; u < s; ++u) {
    qa += A(u, c1);
    h1b += A(u, c1) * bvec[idx[u]];
    hbb += bvec[idx[u]] * A(u, cb);
  }
  const double qb = -2.0 * h1b, qc = hbb - r * r;
  const double disc = qb * qb - 4.0 * qa * qc;
  if (!(qa > 0.0) || !(disc >= 0.0)) return false;
  const double sq = sqrt(disc);
  const double lam = root == 0 ? (-qb - sq) / (2.0 * qa) : (-qb + sq) / (2.0 * qa);
  double vmin = 0.0, vsum = 0.0;
  for (int u = 0; u < s; ++u) {
    const double v = (lam * A(u, c1) - A(u, cb)) / r;
    A(u, c1) = v;  // v_S, then w_S, in column |S|
    vmin = u == 0 || v < vmin ? v : vmin;
    vsum += v;
  }
  if (!(vmin >= -1e-12) || !(vsum > 0.0)) return false;
  double csum = 0.0;
  for (int u = 0; u < s; ++u) {
    const double w = A(u, c1) > 0.0 ? A(u, c1) : 0.0;
    A(u, c1) = w;
    csum += w;
  }
  double bw = 0.0, q = 0.0;
  for (int u = 0; u < s; ++u) A(u, c1) = A(u, c1) / csum;
  for (int u = 0; u < s; ++u) {
    bw += bvec[idx[u]] * A(u, c1);
    double g = 0.0;
    for (int v = 0; v < s; ++v) g += A(v, c1) * G[idx[v] * K + idx[u]];
    q += g * A(u, c1);
  }
  const double f = bw + r * sqrt(q > 0.0 ? q : 0.0);
  if (!__builtin_isfinite(f)) return false;
  *F = f;
  return true;
}

// (F, slot) is lexicographically smaller than (G, other).
__device__ __forceinline__ bool before(double f, int slot, double g, int other) {
  return f < g || (f == g && slot < other);
}

template <int K>
__global__ __launch_bounds__(kWave) void exact_solve_kernel(const double *__restrict__ gram, int method,
                                                            double c, float *__restrict__ weights,
                                                            double *__restrict__ aux) {
  constexpr int NSUB = (1 << K) - 1;
  constexpr int COLS = K + 2;
  __shared__ Shared S;
  __shared__ double mats[(K + 1) * COLS * kWave];
  __shared__ double Gn[K * K];
  __shared__ double qv[NSUB];
  __shared__ uint32_t ok[NSUB];  // mask | kept << 16
  __shared__ int choice;
  const int64_t b = blockIdx.x;
  const int t = threadIdx.x;
  const LaneMat A{mats + t, COLS};
  solver_load_gram<WaveSync>(S, K, gram + b * K * K, t, kWave);
  if (S.bad) {
    if (t < K) {
      weights[b * K + t] = __builtin_nanf("");
      if (aux) aux[b * K + t] = __builtin_nan("");
    }
    return;
  }
  double wt = 0.0, ax = 0.0;
  if (method == MGDA_EXACT) {
    double dmax = S.G[0];
    for (int i = 1; i < K; ++i) dmax = S.G[i * K + i] > dmax ? S.G[i * K + i] : dmax;
    const double scale = dmax > 1e-300 ? dmax : 1e-300;
    for (int i = t; i < K * K; i += kWave) Gn[i] = S.G[i] / scale;
    WaveSync()();
    for (uint32_t m = t + 1; m <= (uint32_t)NSUB; m += kWave) {
      double q = 0.0;
      const bool kept = mgda_support(Gn, K, m, A, &q);
      const int rk = support_rank(m, K);
      qv[rk] = q;
      ok[rk] = m | (kept ? 1u << 16 : 0u);
    }
    WaveSync()();
    if (t == 0) {
      int best = -1;
      double bq = 0.0;
      for (int rk = 0; rk < NSUB; ++rk)
        if ((ok[rk] >> 16) && (best < 0 || qv[rk] < bq - 1e-12)) {
          best = rk;
          bq = qv[rk];
        }
      choice = best;
      if (best >= 0) {
        const uint32_t m = ok[best] & 0xFFFFu;
        double q;
        mgda_support(Gn, K, m, A, &q);
        const int s = __builtin_popcount(m);
        int u = 0;
        for (int i = 0; i < K; ++i) S.a[i] = ((m >> i) & 1u) ? A(u++, s + 1) : 0.0;
      }
    }
    WaveSync()();
    if (choice < 0) solve_mgda<WaveSync>(S, K, 5000, t);
    if (t < K) wt = ax = S.a[t];
  } else {  // CAGRAD_EXACT
    const double invK = 1.0 / (double)K;
    if (t < K) {
      double s = 0.0;
      for (int j = 0; j < K; ++j) s += S.G[t * K + j];
      S.bvec[t] = s / (double)K;
    }
    WaveSync()();
    double tot = 0.0;
    for (int i = 0; i < K * K; ++i) tot += S.G[i];
    double g0sq = tot / (double)(K * K);
    g0sq = g0sq > 0.0 ? g0sq : 0.0;
    const double r = c * sqrt(g0sq);
    // this lane's best candidate: slot t < K are the vertices; support rank
    // rk >= K gives slots K + 2 (rk - K) + root
    double bf = __builtin_inf();
    int bslot = 0x7fffffff;
    uint32_t bmask = 0;
    if (t < K) {
      const double gtt = S.G[t * K + t];
      bf = S.bvec[t] + r * sqrt(gtt > 0.0 ? gtt : 0.0);
      bslot = t;
    }
    if (r > 0.0)
      for (uint32_t m = t + 1; m <= (uint32_t)NSUB; m += kWave) {
        if (__builtin_popcount(m) < 2) continue;
        const int rk = support_rank(m, K);
        for (int root = 0; root < 2; ++root) {
          double f;
          if (cagrad_support(S.G, S.bvec, r, K, m, root, A, &f)) {
            const int slot = K + 2 * (rk - K) + root;
            if (before(f, slot, bf, bslot)) {
              bf = f;
              bslot = slot;
              bmask = m;
            }
          }
        }
      }
    for (int off = kWave / 2; off >= 1; off >>= 1) {
      const double of = __shfl_xor(bf, off, kWave);
      const int os = __shfl_xor(bslot, off, kWave);
      const uint32_t om = (uint32_t)__shfl_xor((int)bmask, off, kWave);
      if (before(of, os, bf, bslot)) {
        bf = of;
        bslot = os;
        bmask = om;
      }
    }
    // every lane now holds the winner; lane 0 rebuilds its point
    if (t == 0) {
      if (bslot < K) {
        for (int i = 0; i < K; ++i) S.a[i] = i == bslot ? 1.0 : 0.0;
      } else {
        const int root = (bslot - K) & 1;
        const uint32_t m = bmask;
        double f;
        cagrad_support(S.G, S.bvec, r, K, m, root, A, &f);
        const int s = __builtin_popcount(m);
        int u = 0;
        for (int i = 0; i < K; ++i) S.a[i] = ((m >> i) & 1u) ? A(u++, s) : 0.0;
      }
    }
    WaveSync()();
    cagrad_primal<WaveSync>(S, K, r, invK, t);
    if (t < K) {
      wt = S.C[t];
      ax = S.a[t];
    }
  }
  if (t < K) {
    weights[b * K + t] = (float)wt;
    if (aux) aux[b * K + t] = ax;
  }
}

template <int K>
void launch_exact_t(int B, const double *gram, int method, double c, float *weights, double *aux,
                    hipStream_t s) {
  hipLaunchKernelGGL(exact_solve_kernel<K>, dim3((unsigned)B), dim3(kWave), 0, s, gram, method, c,
                     weights, aux);
}

}  // namespace

hipError_t launch_exact_solve(int K, int B, const double *gram, int method, double c, float *weights,
                              double *aux, hipStream_t s) {
  switch (K) {
    case 2: launch_exact_t<2>(B, gram, method, c, weights, aux, s); break;
    case 3: launch_exact_t<3>(B, gram, method, c, weights, aux, s); break;
    case 4: launch_exact_t<4>(B, gram, method, c, weights, aux, s); break;
    case 5: launch_exact_t<5>(B, gram, method, c, weights, aux, s); break;
    case 6: launch_exact_t<6>(B, gram, method, c, weights, aux, s); break;
    case 7: launch_exact_t<7>(B, gram, method, c, weights, aux, s); break;
    case 8: launch_exact_t<8>(B, gram, method, c, weights, aux, s); break;
    case 9: launch_exact_t<9>(B, gram, method, c, weights, aux, s); break;
    case 10: launch_exact_t<10>(B, gram, method, c, weights, aux, s); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace bkmoo
