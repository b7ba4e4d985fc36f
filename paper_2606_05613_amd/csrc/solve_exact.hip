// Exact solvers for the per-bucket problems, by support enumeration: the
// minimum-norm point of the simplex hull of the task gradients (Eq. mgda /
// Eq. shard-mgda over the simplex) and the minimiser of the CAGrad dual
// F(w) = b^T w + r ||g_w|| over the simplex (the local problem of Eq.
// cagrad through its dual), both from the bucket's Gram matrix alone.
//
// One wavefront per bucket, fp64, K <= 10.  The 2^K - 1 supports S are
// ranked in the order "by support size, then lexicographically", which fixes
// every tie-break, and dealt to the 64 lanes in rank order, so the lanes of
// a wavefront mostly hold supports of one size.  Each lane builds its
// support's small linear system in registers (a solver instantiated per
// support size, fully unrolled, row exchanges done by selects so every index
// is static) and solves it by Gaussian elimination with partial pivoting; a
// support whose system has an exactly zero pivot is skipped:
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

// Rank -> support (bit t = task t) tables for every K, built at compile
// time: the non-empty subsets of {0..K-1} ordered by size, then
// lexicographically (each size's combinations from {0..s-1} by the usual
// successor: raise the last index that can still rise, reset the rest
// right after it).  A lookup replaces unranking through binomial sums,
// whose integer divisions took half of the kernel's time (K=10, 6,564
// buckets: 2.45 -> 1.27 ms, identical results).
struct SupportTables {
  uint16_t m[kExactMaxK + 1][(1 << kExactMaxK) - 1];
};
constexpr SupportTables make_support_tables() {
  SupportTables T{};
  for (int K = 1; K <= kExactMaxK; ++K) {
    int r = 0;
    for (int s = 1; s <= K; ++s) {
      int c[kExactMaxK] = {};
      for (int i = 0; i < s; ++i) c[i] = i;
      for (;;) {
        uint16_t m = 0;
        for (int i = 0; i < s; ++i) m = (uint16_t)(m | (1u << c[i]));
        T.m[K][r++] = m;
        int i = s - 1;
        while (i >= 0 && c[i] == K - s + i) --i;
        if (i < 0) break;
        ++c[i];
        for (int j = i + 1; j < s; ++j) c[j] = c[j - 1] + 1;
      }
    }
  }
  return T;
}
__constant__ SupportTables kSupportTables = make_support_tables();

// Gaussian elimination with partial pivoting (the first entry of largest
// magnitude) on the N x (N + M) augmented matrix A, fully unrolled.  False if
// a pivot is exactly zero; otherwise the solutions overwrite columns N..N+M-1.
template <int N, int M>
__device__ __forceinline__ bool ge_solve(double (&A)[N][N + M]) {
  bool ok = true;
#pragma unroll
  for (int k = 0; k < N; ++k) {
    double pv = fabs(A[k][k]);
    int p = k;
#pragma unroll
    for (int r = k + 1; r < N; ++r) {
      const double v = fabs(A[r][k]);
      const bool gt = v > pv;
      pv = gt ? v : pv;
      p = gt ? r : p;
    }
    ok = ok && pv != 0.0;
#pragma unroll
    for (int r = k + 1; r < N; ++r) {
      const bool sw = p == r;
#pragma unroll
      for (int c = k; c < N + M; ++c) {
        const double x = A[k][c], y = A[r][c];
        A[k][c] = sw ? y : x;
        A[r][c] = sw ? x : y;
      }
    }
    const double piv = pv != 0.0 ? A[k][k] : 1.0;
#pragma unroll
    for (int r = k + 1; r < N; ++r) {
      const double f = A[r][k] / piv;
#pragma unroll
      for (int c = k + 1; c < N + M; ++c) A[r][c] -= f * A[k][c];
      A[r][k] = 0.0;
    }
  }
#pragma unroll
  for (int j = N; j < N + M; ++j)
#pragma unroll
    for (int r = N - 1; r >= 0; --r) {
      double s = A[r][j];
#pragma unroll
      for (int c = r + 1; c < N; ++c) s -= A[r][c] * A[c][j];
      A[r][j] = s / (A[r][r] != 0.0 ? A[r][r] : 1.0);
    }
  return ok;
}

// Tasks of support m in increasing order.
template <int S>
__device__ __forceinline__ void support_tasks(uint32_t m, int (&idx)[S]) {
#pragma unroll
  for (int u = 0; u < S; ++u) {
    idx[u] = __builtin_ctz(m);
    m &= m - 1u;
  }
}

// MGDA on a support of S tasks of the normalised Gram Gn: solves the
// bordered system and runs the feasibility and minimum-norm checks.  On
// success a[0..S) holds the clipped, renormalised weights of the support's
// tasks in increasing task order and *q = a^T Gn a.
template <int S>
__device__ bool mgda_support(const double *Gn, int K, uint32_t m, double (&a)[S], double *q) {
  int idx[S];
  support_tasks<S>(m, idx);
  double A[S + 1][S + 2];
#pragma unroll
  for (int u = 0; u < S; ++u) {
#pragma unroll
    for (int v = 0; v < S; ++v) A[u][v] = Gn[idx[u] * K + idx[v]];
    A[u][S] = 1.0;
    A[u][S + 1] = 0.0;
  }
#pragma unroll
  for (int v = 0; v < S; ++v) A[S][v] = 1.0;
  A[S][S] = 0.0;
  A[S][S + 1] = 1.0;
  if (!ge_solve<S + 1, 1>(A)) return false;
  double amin = S < K ? 0.0 : A[0][S + 1], sum = 0.0;
#pragma unroll
  for (int u = 0; u < S; ++u) {
    amin = A[u][S + 1] < amin ? A[u][S + 1] : amin;
    sum += A[u][S + 1];
  }
  if (!(amin >= -1e-10) || !(fabs(sum - 1.0) <= 1e-9)) return false;
  double csum = 0.0;
#pragma unroll
  for (int u = 0; u < S; ++u) {
    a[u] = A[u][S + 1] > 0.0 ? A[u][S + 1] : 0.0;
    csum += a[u];
  }
#pragma unroll
  for (int u = 0; u < S; ++u) a[u] = a[u] / csum;
  // (Gn a)_t over every task, a^T Gn a, and the minimum-norm check
  double qq = 0.0;
#pragma unroll
  for (int u = 0; u < S; ++u) {
    double g = 0.0;
#pragma unroll
    for (int v = 0; v < S; ++v) g += Gn[idx[u] * K + idx[v]] * a[v];
    qq += a[u] * g;
  }
  for (int t = 0; t < K; ++t) {
    double g = 0.0;
#pragma unroll
    for (int v = 0; v < S; ++v) g += Gn[t * K + idx[v]] * a[v];
    if (!(g >= qq - 1e-9)) return false;
  }
  *q = qq;
  return true;
}

// CAGrad candidate `root` (0: smaller lam, 1: larger) on a support of S >= 2
// tasks: on success w[0..S) holds the simplex point on the support's tasks
// and *F its dual objective.
template <int S>
__device__ bool cagrad_support(const double *G, const double *bvec, double r, int K, uint32_t m,
                               int root, double (&w)[S], double *F) {
  int idx[S];
  support_tasks<S>(m, idx);
  double A[S][S + 2];  // [G_SS | 1 | b_S]
#pragma unroll
  for (int u = 0; u < S; ++u) {
#pragma unroll
    for (int v = 0; v < S; ++v) A[u][v] = G[idx[u] * K + idx[v]];
    A[u][S] = 1.0;
    A[u][S + 1] = bvec[idx[u]];
  }
  if (!ge_solve<S, 2>(A)) return false;
  double qa = 0.0, h1b = 0.0, hbb = 0.0;
#pragma unroll
  for (int u = 0; u < S; ++u) {
    qa += A[u][S];
    h1b += A[u][S] * bvec[idx[u]];
    hbb += bvec[idx[u]] * A[u][S + 1];
  }
  const double qb = -2.0 * h1b, qc = hbb - r * r;
  const double disc = qb * qb - 4.0 * qa * qc;
  if (!(qa > 0.0) || !(disc >= 0.0)) return false;
  const double sq = sqrt(disc);
  const double lam = root == 0 ? (-qb - sq) / (2.0 * qa) : (-qb + sq) / (2.0 * qa);
  double vmin = 0.0, vsum = 0.0;
#pragma unroll
  for (int u = 0; u < S; ++u) {
    const double v = (lam * A[u][S] - A[u][S + 1]) / r;
    w[u] = v;
    vmin = u == 0 || v < vmin ? v : vmin;
    vsum += v;
  }
  if (!(vmin >= -1e-12) || !(vsum > 0.0)) return false;
  double csum = 0.0;
#pragma unroll
  for (int u = 0; u < S; ++u) {
    w[u] = w[u] > 0.0 ? w[u] : 0.0;
    csum += w[u];
  }
  double bw = 0.0, q = 0.0;
#pragma unroll
  for (int u = 0; u < S; ++u) w[u] = w[u] / csum;
#pragma unroll
  for (int u = 0; u < S; ++u) {
    bw += bvec[idx[u]] * w[u];
    double g = 0.0;
#pragma unroll
    for (int v = 0; v < S; ++v) g += w[v] * G[idx[v] * K + idx[u]];
    q += g * w[u];
  }
  const double f = bw + r * sqrt(q > 0.0 ? q : 0.0);
  if (!__builtin_isfinite(f)) return false;
  *F = f;
  return true;
}

// Size dispatch: run the support-size instantiation for |m| and, if `dst`
// is given, scatter its point onto the K tasks.
__device__ bool mgda_any(const double *Gn, int K, uint32_t m, double *q, double *dst) {
  switch (__builtin_popcount(m)) {
#define BKMOO_MGDA_CASE(n)                                                 \
  case n: {                                                                \
    double a[n];                                                           \
    if (!mgda_support<n>(Gn, K, m, a, q)) return false;                    \
    if (dst) {                                                             \
      int idx[n];                                                          \
      support_tasks<n>(m, idx);                                            \
      for (int i = 0; i < K; ++i) dst[i] = 0.0;                            \
      _Pragma("unroll") for (int u = 0; u < n; ++u) dst[idx[u]] = a[u];    \
    }                                                                      \
    return true;                                                           \
  }
    BKMOO_MGDA_CASE(1) BKMOO_MGDA_CASE(2) BKMOO_MGDA_CASE(3) BKMOO_MGDA_CASE(4) BKMOO_MGDA_CASE(5)
    BKMOO_MGDA_CASE(6) BKMOO_MGDA_CASE(7) BKMOO_MGDA_CASE(8) BKMOO_MGDA_CASE(9) BKMOO_MGDA_CASE(10)
#undef BKMOO_MGDA_CASE
    default: return false;
  }
}

__device__ bool cagrad_any(const double *G, const double *bvec, double r, int K, uint32_t m, int root,
                           double *F, double *dst) {
  switch (__builtin_popcount(m)) {
#define BKMOO_CAGRAD_CASE(n)                                                   \
  case n: {                                                                    \
    double w[n];                                                               \
    if (!cagrad_support<n>(G, bvec, r, K, m, root, w, F)) return false;        \
    if (dst) {                                                                 \
      int idx[n];                                                              \
      support_tasks<n>(m, idx);                                                \
      for (int i = 0; i < K; ++i) dst[i] = 0.0;                                \
      _Pragma("unroll") for (int u = 0; u < n; ++u) dst[idx[u]] = w[u];        \
    }                                                                          \
    return true;                                                               \
  }
    BKMOO_CAGRAD_CASE(2) BKMOO_CAGRAD_CASE(3) BKMOO_CAGRAD_CASE(4) BKMOO_CAGRAD_CASE(5)
    BKMOO_CAGRAD_CASE(6) BKMOO_CAGRAD_CASE(7) BKMOO_CAGRAD_CASE(8) BKMOO_CAGRAD_CASE(9)
    BKMOO_CAGRAD_CASE(10)
#undef BKMOO_CAGRAD_CASE
    default: return false;
  }
}

// (F, slot) is lexicographically smaller than (G, other).
__device__ __forceinline__ bool before(double f, int slot, double g, int other) {
  return f < g || (f == g && slot < other);
}

constexpr int kMaxSupports = (1 << kExactMaxK) - 1;

__global__ __launch_bounds__(kWave) void exact_solve_kernel(int K, const double *__restrict__ gram,
                                                            int method, double c,
                                                            float *__restrict__ weights,
                                                            double *__restrict__ aux) {
  __shared__ Shared S;
  __shared__ double Gn[kExactMaxK * kExactMaxK];
  __shared__ double qv[kMaxSupports];
  __shared__ uint32_t ok[kMaxSupports];  // mask | kept << 16
  __shared__ int choice;
  const int64_t b = blockIdx.x;
  const int t = threadIdx.x;
  const int nsub = (1 << K) - 1;
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
    for (int rk = t; rk < nsub; rk += kWave) {
      const uint32_t m = kSupportTables.m[K][rk];
      double q = 0.0;
      const bool kept = mgda_any(Gn, K, m, &q, nullptr);
      qv[rk] = q;
      ok[rk] = m | (kept ? 1u << 16 : 0u);
    }
    WaveSync()();
    if (t == 0) {
      int best = -1;
      double bq = 0.0;
      for (int rk = 0; rk < nsub; ++rk)
        if ((ok[rk] >> 16) && (best < 0 || qv[rk] < bq - 1e-12)) {
          best = rk;
          bq = qv[rk];
        }
      choice = best;
      if (best >= 0) {
        double q;
        mgda_any(Gn, K, ok[best] & 0xFFFFu, &q, S.a);
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
      for (int rk = K + t; rk < nsub; rk += kWave) {
        const uint32_t m = kSupportTables.m[K][rk];
        for (int root = 0; root < 2; ++root) {
          double f;
          if (cagrad_any(S.G, S.bvec, r, K, m, root, &f, nullptr)) {
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
        double f;
        cagrad_any(S.G, S.bvec, r, K, bmask, (bslot - K) & 1, &f, S.a);
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

}  // namespace

hipError_t launch_exact_solve(int K, int B, const double *gram, int method, double c, float *weights,
                              double *aux, hipStream_t s) {
  if (K < kMinK || K > kExactMaxK) return hipErrorInvalidValue;
  hipLaunchKernelGGL(exact_solve_kernel, dim3((unsigned)B), dim3(kWave), 0, s, K, gram, method, c, weights,
                     aux);
  return hipGetLastError();
}

}  // namespace bkmoo
