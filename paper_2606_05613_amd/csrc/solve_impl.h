// Per-bucket MOO solvers shared by the solve kernel and the pipelined
// resolve kernel.  Every function is called by all threads of one wavefront
// (WaveSync) or of the workgroup (BlockSync); lanes t < K do the per-task
// work, the scalar steps run redundantly on every lane from LDS broadcasts.
// Translation units that include this are compiled without floating-point
// contraction so every scalar expression rounds as written.
#pragma once

#include "internal.h"

namespace bkmoo {

namespace {

// Synchronisation between the steps of a solver.  BlockSync: every thread
// of the workgroup runs the solver.  WaveSync: a single wavefront runs it;
// its LDS accesses execute in order, so a fence that keeps the compiler from
// moving memory operations across the step (and waits for LDS) suffices.
struct BlockSync {
  __device__ __forceinline__ void operator()() const { __syncthreads(); }
};
struct WaveSync {
  __device__ __forceinline__ void operator()() const {
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
    __builtin_amdgcn_wave_barrier();
  }
};

enum Method : int { MGDA = 0, PCGRAD = 1, CAGRAD = 2, MEAN = 3, MGDA_EXACT = 4, CAGRAD_EXACT = 5 };

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
template <typename Sync>
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
  Sync()();
  for (int it = 0; it < iters; ++it) {
    if (t < K) {
      double s = 0.0;
      for (int j = 0; j < K; ++j) s += S.G[t * K + j] * S.a[j];
      S.v[t] = s;
    }
    Sync()();
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
    Sync()();
    if (t < K) {
      double na = g * S.a[t];
      if (t == ts) na += 1.0 - g;
      S.a[t] = na;
    }
    Sync()();
  }
}

// PCGrad (Algorithm 1): lane t owns task t's coefficient row; a projection
// of d_t off g_j only changes C[t][j], and every inner product uses the
// original g_j, so the K tasks are independent.
template <typename Sync>
__device__ void solve_pcgrad(Shared &S, int K, const int8_t *order, int64_t b, int t) {
  if (t < K) {
    for (int i = 0; i < K; ++i) S.C[t * K + i] = i == t ? 1.0 : 0.0;
    uint32_t seen = 1u << t;
    for (int q = 0; q < K - 1; ++q) {
      int j = q < t ? q : q + 1;
      if (order) {
        j = order[(b * K + t) * (K - 1) + q];
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
  Sync()();
  if (t < K) {
    double w = 0.0;
    for (int r = 0; r < K; ++r) w += S.C[r * K + t];
    S.a[t] = w;
  }
  Sync()();
}

// CAGrad's primal weights from the dual point w = S.a: d = g_avg + r g_w /
// |g_w|, i.e. weights 1/K + (r / |g_w|) w_t, or 1/K when r = 0 or g_w
// vanishes relative to the largest gradient.  Writes S.C[0..K).
template <typename Sync>
__device__ void cagrad_primal(Shared &S, int K, double r, double invK, int t) {
  if (t < K) {
    double s = 0.0;
    for (int j = 0; j < K; ++j) s += S.G[t * K + j] * S.a[j];
    S.v[t] = s;
  }
  Sync()();
  double q = 0.0, dmax = 0.0;
  for (int i = 0; i < K; ++i) q += S.a[i] * S.v[i];
  for (int i = 0; i < K; ++i) dmax = S.G[i * K + i] > dmax ? S.G[i * K + i] : dmax;
  const double nrm = sqrt(q > 0.0 ? q : 0.0);
  const double scale = sqrt(dmax);
  const bool degenerate = r == 0.0 || nrm <= 1e-12 * scale || nrm == 0.0;
  Sync()();
  if (t < K) S.C[t] = degenerate ? invK : invK + (r / nrm) * S.a[t];  // weights
  Sync()();
}

// CAGrad through its dual min_{w in simplex} F(w) = b^T w + r sqrt(w^T G w)
// (b = G 1 / K, r = c |g_avg|), Frank-Wolfe from the uniform point with an
// exact line search; primal d = g_avg + r g_w / |g_w|.
template <typename Sync>
__device__ void solve_cagrad(Shared &S, int K, int iters, double c, int t) {
  const double invK = 1.0 / (double)K;
  if (t < K) {
    double s = 0.0;
    for (int j = 0; j < K; ++j) s += S.G[t * K + j];
    S.bvec[t] = s / (double)K;
    S.a[t] = invK;
  }
  Sync()();
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
    Sync()();
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
    Sync()();
    if (t < K) {
      double na = (1.0 - gamma) * S.a[t];
      if (t == sidx) na += gamma;
      S.a[t] = na;
    }
    Sync()();
  }
  cagrad_primal<Sync>(S, K, r, invK, t);
}

// ---- register-only solvers for a compile-time K --------------------------
// The same algorithms, operation for operation, as solve_mgda and
// solve_cagrad above, with G and the iterate held in registers by every
// lane (each lane computes the same scalars): no LDS round trips and no
// synchronisation between steps.  Used where one bucket's solve sits on a
// critical path.

template <int K>
__device__ __forceinline__ double pick(const double (&x)[K], int idx) {
  double r = x[0];
#pragma unroll
  for (int i = 1; i < K; ++i) r = i == idx ? x[i] : r;
  return r;
}

template <int K>
__device__ void reg_solve_mgda(const double (&G)[K][K], int iters, double (&a)[K]) {
  double best = 0.0, bg = 1.0;
  int bi = 0, bj = 1;
  bool first = true;
#pragma unroll
  for (int i = 0; i < K; ++i)
#pragma unroll
    for (int j = i + 1; j < K; ++j) {
      const double aa = G[i][i], ab = G[i][j], bb = G[j][j];
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
#pragma unroll
  for (int i = 0; i < K; ++i) a[i] = i == bi ? bg : i == bj ? 1.0 - bg : 0.0;
  for (int it = 0; it < iters; ++it) {
    double v[K];
#pragma unroll
    for (int i = 0; i < K; ++i) {
      double s = 0.0;
#pragma unroll
      for (int j = 0; j < K; ++j) s += G[i][j] * a[j];
      v[i] = s;
    }
    int ts = 0;
    double m = v[0];
#pragma unroll
    for (int i = 1; i < K; ++i)
      if (v[i] < m) {
        m = v[i];
        ts = i;
      }
    double aa = 0.0;
#pragma unroll
    for (int i = 0; i < K; ++i) aa += a[i] * v[i];
    double gts = G[0][0];
#pragma unroll
    for (int i = 1; i < K; ++i) gts = i == ts ? G[i][i] : gts;
    const double g = pair_gamma(aa, pick<K>(v, ts), gts);
#pragma unroll
    for (int i = 0; i < K; ++i) {
      double na = g * a[i];
      if (i == ts) na += 1.0 - g;
      a[i] = na;
    }
  }
}

template <int K>
__device__ void reg_solve_cagrad(const double (&G)[K][K], int iters, double c, double (&wt)[K],
                                 double (&w)[K]) {
  const double invK = 1.0 / (double)K;
  double b[K];
#pragma unroll
  for (int i = 0; i < K; ++i) {
    double s = 0.0;
#pragma unroll
    for (int j = 0; j < K; ++j) s += G[i][j];
    b[i] = s / (double)K;
    w[i] = invK;
  }
  double tot = 0.0;
#pragma unroll
  for (int i = 0; i < K; ++i)
#pragma unroll
    for (int j = 0; j < K; ++j) tot += G[i][j];
  double g0sq = tot / (double)(K * K);
  g0sq = g0sq > 0.0 ? g0sq : 0.0;
  const double r = c * sqrt(g0sq);
  for (int it = 0; it < iters; ++it) {
    double v[K];
#pragma unroll
    for (int i = 0; i < K; ++i) {
      double s = 0.0;
#pragma unroll
      for (int j = 0; j < K; ++j) s += G[i][j] * w[j];
      v[i] = s;
    }
    double cq = 0.0, bw = 0.0;
#pragma unroll
    for (int i = 0; i < K; ++i) cq += w[i] * v[i];
#pragma unroll
    for (int i = 0; i < K; ++i) bw += b[i] * w[i];
    const double nrm = sqrt(cq > 0.0 ? cq : 0.0);
    int sidx = 0;
    double m = 0.0;
#pragma unroll
    for (int i = 0; i < K; ++i) {
      const double gi = b[i] + (nrm > 1e-300 ? r * v[i] / nrm : 0.0);
      if (i == 0 || gi < m) {
        m = gi;
        sidx = i;
      }
    }
    double gss = G[0][0];
#pragma unroll
    for (int i = 1; i < K; ++i) gss = i == sidx ? G[i][i] : gss;
    const double vs = pick<K>(v, sidx);
    const double beta1 = pick<K>(b, sidx) - bw;
    const double A = gss - 2.0 * vs + cq;
    const double Bq = vs - cq;
    // candidates in ascending order: 0, the interior stationary points
    // (g1 <= g2 since A > 0), 1; the first of least F wins
    double g1 = -1.0, g2 = -1.0;
    const double D = r * r * A - beta1 * beta1;
    if (A > 0.0 && D > 0.0) {
      const double disc = (A * cq - Bq * Bq) / D;
      if (disc >= 0.0) {
        const double root = fabs(beta1) * sqrt(disc);
        g1 = (-Bq - root) / A;
        g2 = (-Bq + root) / A;
      }
    }
    const bool h1 = g1 > 0.0 && g1 < 1.0, h2 = g2 > 0.0 && g2 < 1.0;
    double gamma = 0.0, fbest = 0.0;
    {
      double q = A * 0.0 * 0.0 + 2.0 * Bq * 0.0 + cq;
      q = q > 0.0 ? q : 0.0;
      fbest = bw + beta1 * 0.0 + r * sqrt(q);
    }
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      const bool has = k == 0 ? h1 : k == 1 ? h2 : true;
      const double g = k == 0 ? g1 : k == 1 ? g2 : 1.0;
      if (has) {
        double q = A * g * g + 2.0 * Bq * g + cq;
        q = q > 0.0 ? q : 0.0;
        const double f = bw + beta1 * g + r * sqrt(q);
        if (f < fbest) {
          fbest = f;
          gamma = g;
        }
      }
    }
#pragma unroll
    for (int i = 0; i < K; ++i) {
      double na = (1.0 - gamma) * w[i];
      if (i == sidx) na += gamma;
      w[i] = na;
    }
  }
  double v[K];
#pragma unroll
  for (int i = 0; i < K; ++i) {
    double s = 0.0;
#pragma unroll
    for (int j = 0; j < K; ++j) s += G[i][j] * w[j];
    v[i] = s;
  }
  double q = 0.0, dmax = 0.0;
#pragma unroll
  for (int i = 0; i < K; ++i) q += w[i] * v[i];
#pragma unroll
  for (int i = 0; i < K; ++i) dmax = G[i][i] > dmax ? G[i][i] : dmax;
  const double nrm = sqrt(q > 0.0 ? q : 0.0);
  const double scale = sqrt(dmax);
  const bool degenerate = r == 0.0 || nrm <= 1e-12 * scale || nrm == 0.0;
#pragma unroll
  for (int i = 0; i < K; ++i) wt[i] = degenerate ? invK : invK + (r / nrm) * w[i];
}

// ---- lane-parallel solvers for a compile-time K <= 16 ---------------------
// The same algorithms as solve_mgda and solve_cagrad above (same start,
// steps, tie rules, line searches and fixed iteration counts), run by one
// whole wavefront with lane i < K holding task i's row of G, its entry of
// G a and its variable, so a step costs O(K) instead of O(K^2) arithmetic
// per lane.  Cross-lane steps use DPP within the first row of 16 lanes
// (quad butterflies, then rotations by 4 and 8), and lane 0's result is
// broadcast; sums are therefore added in a different (fixed) order than the
// sequential loops above, so results agree with them to rounding, not
// bitwise.  Used where one bucket's solve sits on a critical path.

template <int CTRL>
__device__ __forceinline__ int dpp_i32(int x) {
  return __builtin_amdgcn_update_dpp(0, x, CTRL, 0xf, 0xf, false);
}
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double x) {
  const long long u = __double_as_longlong(x);
  const int lo = dpp_i32<CTRL>((int)u), hi = dpp_i32<CTRL>((int)(u >> 32));
  return __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) | (unsigned)lo));
}
// x of lane l (l uniform across the wavefront).
__device__ __forceinline__ double lane_f64(double x, int l) {
  const long long u = __double_as_longlong(x);
  const int lo = __builtin_amdgcn_readlane((int)u, l), hi = __builtin_amdgcn_readlane((int)(u >> 32), l);
  return __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) | (unsigned)lo));
}
// DPP controls: quad_perm xor 1, quad_perm xor 2, row rotations by 4 and 8.
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppRor4 = 0x124, kDppRor8 = 0x128;

// Sum of x over lanes 0..K-1 (x must be 0 on lanes K..15), broadcast.
template <int K>
__device__ __forceinline__ double row_sum(double x) {
  static_assert(K <= 16, "one row of lanes");
  x += dpp_f64<kDppXor1>(x);
  x += dpp_f64<kDppXor2>(x);
  if constexpr (K > 4) {
    x += dpp_f64<kDppRor4>(x);
    x += dpp_f64<kDppRor8>(x);
  }
  return lane_f64(x, 0);
}

template <int CTRL>
__device__ __forceinline__ void argmin_step(double &v, int &idx) {
  const double ov = dpp_f64<CTRL>(v);
  const int oi = dpp_i32<CTRL>(idx);
  const bool take = ov < v || (ov == v && oi < idx);
  v = take ? ov : v;
  idx = take ? oi : idx;
}
// Lowest index among the least v over lanes 0..K-1 (v must be +inf and idx
// above K on lanes K..15), broadcast.
template <int K>
__device__ __forceinline__ int row_argmin(double v, int idx) {
  static_assert(K <= 16, "one row of lanes");
  argmin_step<kDppXor1>(v, idx);
  argmin_step<kDppXor2>(v, idx);
  if constexpr (K > 4) {
    argmin_step<kDppRor4>(v, idx);
    argmin_step<kDppRor8>(v, idx);
  }
  return __builtin_amdgcn_readlane(idx, 0);
}

// First pair (i < j, lexicographic) of least two-point norm and its step:
// lane l < K(K-1)/2 evaluates pair l, then a wavefront-wide lexicographic
// (value, pair) minimum.  Every lane returns the same (bi, bj, bg).
template <int K>
__device__ __forceinline__ void lane_best_pair(const double *G, int lane, int &bi, int &bj, double &bg) {
  constexpr int NP = K * (K - 1) / 2;
  static_assert(NP <= kWave, "one pair per lane");
  int pi = 0, rem = lane < NP ? lane : 0;
  while (rem >= K - 1 - pi) {
    rem -= K - 1 - pi;
    ++pi;
  }
  const int pj = pi + 1 + rem;
  const double aa = G[pi * K + pi], ab = G[pi * K + pj], bb = G[pj * K + pj];
  const double g = pair_gamma(aa, ab, bb);
  double val = lane < NP ? pair_value(g, aa, ab, bb) : __builtin_inf();
  int idx = lane < NP ? lane : kWave;
#pragma unroll
  for (int off = kWave / 2; off >= 1; off >>= 1) {
    const double ov = __shfl_xor(val, off, kWave);
    const int oi = __shfl_xor(idx, off, kWave);
    const bool take = ov < val || (ov == val && oi < idx);
    val = take ? ov : val;
    idx = take ? oi : idx;
  }
  const int best = __builtin_amdgcn_readfirstlane(idx);
  bi = __builtin_amdgcn_readlane(pi, best);
  bj = __builtin_amdgcn_readlane(pj, best);
  bg = lane_f64(g, best);
}

// MGDA (as solve_mgda).  G: K x K row-major, readable by every lane (LDS).
// Lane i < K returns task i's simplex weight.  G a and a^T G a are summed
// for the starting pair's point and then carried: with a' = g a + (1 - g)
// e_t, (G a')_i = g (G a)_i + (1 - g) G_it and a'^T G a' = g^2 a^T G a +
// 2 g (1 - g) (G a)_t + (1 - g)^2 G_tt (exact for g = 1 and g = 0).
template <int K>
__device__ double lane_solve_mgda(const double *G, int iters, int lane) {
  const bool task = lane < K;
  const int me = task ? lane : 0;
  double gi[K];
  double gd = 0.0;
#pragma unroll
  for (int j = 0; j < K; ++j) {
    gi[j] = task ? G[me * K + j] : 0.0;
    gd = j == me ? gi[j] : gd;
  }
  int bi, bj;
  double bg;
  lane_best_pair<K>(G, lane, bi, bj, bg);
  double own = task ? (me == bi ? bg : me == bj ? 1.0 - bg : 0.0) : 0.0;
  double v = 0.0;  // (G a)_i
#pragma unroll
  for (int j = 0; j < K; ++j) v += gi[j] * (j == bi ? bg : j == bj ? 1.0 - bg : 0.0);
  double aa = row_sum<K>(task ? own * v : 0.0);  // a^T G a
  for (int it = 0; it < iters; ++it) {
    const int t = row_argmin<K>(task ? v : __builtin_inf(), task ? lane : kWave);
    const double git = task ? G[me * K + t] : 0.0;
    const double vt = lane_f64(v, t), gtt = lane_f64(gd, t);
    const double g = pair_gamma(aa, vt, gtt);
    const double h = 1.0 - g;
    aa = g * g * aa + 2.0 * g * h * vt + h * h * gtt;
    v = g * v + h * git;
    double no = g * own;
    if (task && lane == t) no += h;
    own = no;
  }
  return own;
}

// CAGrad (as solve_cagrad and cagrad_primal).  Lane i < K returns task i's
// combine weight in *wt and dual variable in *w_out.  The step's
// quantities are carried from one iteration to the next instead of being
// summed again: with w' = (1 - gamma) w + gamma e_s, (G w')_i = (1 - gamma)
// (G w)_i + gamma G_is, w'^T G w' is the line search's quadratic at gamma
// and b^T w' = (1 - gamma) b^T w + gamma b_s (exact for gamma = 0 and, but
// for the quadratic, gamma = 1); the first iterate's sums are computed as
// before.
template <int K>
__device__ void lane_solve_cagrad(const double *G, int iters, double c, int lane, double *wt, double *w_out) {
  const bool task = lane < K;
  const int me = task ? lane : 0;
  const double invK = 1.0 / (double)K;
  double gi[K];
  double gd = 0.0, rs = 0.0;
#pragma unroll
  for (int j = 0; j < K; ++j) {
    gi[j] = task ? G[me * K + j] : 0.0;
    gd = j == me ? gi[j] : gd;
    rs += gi[j];
  }
  const double bo = rs / (double)K;  // b_i = (G 1)_i / K
  double g0sq = row_sum<K>(task ? rs : 0.0) / (double)(K * K);
  g0sq = g0sq > 0.0 ? g0sq : 0.0;
  const double r = c * sqrt(g0sq);
  double own = task ? invK : 0.0;
  double v = 0.0;  // (G w)_i
#pragma unroll
  for (int j = 0; j < K; ++j) v += gi[j] * invK;
  double cq = row_sum<K>(task ? own * v : 0.0);   // w^T G w
  double bw = row_sum<K>(task ? bo * own : 0.0);  // b^T w
  for (int it = 0; it < iters; ++it) {
    const double nrm = sqrt(cq > 0.0 ? cq : 0.0);
    const double grad = bo + (nrm > 1e-300 ? r * v / nrm : 0.0);
    const int s = row_argmin<K>(task ? grad : __builtin_inf(), task ? lane : kWave);
    const double gis = task ? G[me * K + s] : 0.0;
    const double vs = lane_f64(v, s);
    const double bs = lane_f64(bo, s);
    const double beta1 = bs - bw;
    const double A = lane_f64(gd, s) - 2.0 * vs + cq;
    const double Bq = vs - cq;
    double g1 = -1.0, g2 = -1.0;
    const double D = r * r * A - beta1 * beta1;
    if (A > 0.0 && D > 0.0) {
      const double disc = (A * cq - Bq * Bq) / D;
      if (disc >= 0.0) {
        const double root = fabs(beta1) * sqrt(disc);
        g1 = (-Bq - root) / A;
        g2 = (-Bq + root) / A;
      }
    }
    // candidates in ascending order on lanes 0..3: 0, the interior
    // stationary points (g1 <= g2 since A > 0), 1; the first of least F wins
    const int q4 = lane & 3;
    const double gc = q4 == 0 ? 0.0 : q4 == 1 ? g1 : q4 == 2 ? g2 : 1.0;
    const bool valid = lane < 4 && (q4 == 0 || q4 == 3 || (gc > 0.0 && gc < 1.0));
    const double qraw = A * gc * gc + 2.0 * Bq * gc + cq;
    const double qq = qraw > 0.0 ? qraw : 0.0;
    const double f = valid ? bw + beta1 * gc + r * sqrt(qq) : __builtin_inf();
    double fv = f;
    int fi = valid ? q4 : kWave;
    argmin_step<kDppXor1>(fv, fi);
    argmin_step<kDppXor2>(fv, fi);
    const int win = __builtin_amdgcn_readlane(fi, 0);
    const double gamma = lane_f64(gc, win);
    cq = lane_f64(qraw, win);
    v = (1.0 - gamma) * v + gamma * gis;
    bw = (1.0 - gamma) * bw + gamma * bs;
    double no = (1.0 - gamma) * own;
    if (task && lane == s) no += gamma;
    own = no;
  }
  const double q = row_sum<K>(task ? own * v : 0.0);
  double dmax = 0.0;
#pragma unroll
  for (int l = 0; l < K; ++l) {
    const double x = lane_f64(gd, l);
    dmax = x > dmax ? x : dmax;
  }
  const double nrm = sqrt(q > 0.0 ? q : 0.0);
  const double scale = sqrt(dmax);
  const bool degenerate = r == 0.0 || nrm <= 1e-12 * scale || nrm == 0.0;
  *wt = degenerate ? invK : invK + (r / nrm) * own;
  *w_out = own;
}

// Load one bucket's Gram matrix (fp64, row-major K x K) into S and flag a
// non-finite entry.  Returns through S.bad.
template <typename Sync>
__device__ void solver_load_gram(Shared &S, int K, const double *__restrict__ g, int t, int nthreads) {
  if (t == 0) S.bad = 0;
  Sync()();
  for (int i = t; i < K * K; i += nthreads) {
    const double v = g[i];
    S.G[i] = v;
    if (!__builtin_isfinite(v)) S.bad = 1;
  }
  Sync()();
}

// Run `method` on S.G; afterwards lane t < K holds (weight, aux) in
// (*wt, *ax).  NaN for a non-finite Gram or an invalid PCGrad order.
template <typename Sync>
__device__ void solver_run(Shared &S, int K, int method, int iters, double c, const int8_t *order,
                           int64_t b, int t, double *wt, double *ax) {
  const double nan = __builtin_nan("");
  *wt = *ax = 0.0;
  if (S.bad) {
    *wt = *ax = nan;
    return;
  }
  switch (method) {
    case MGDA:
      solve_mgda<Sync>(S, K, iters, t);
      if (t < K) *wt = *ax = S.a[t];
      break;
    case PCGRAD:
      solve_pcgrad<Sync>(S, K, order, b, t);
      if (t < K) *wt = *ax = S.bad ? nan : S.a[t];
      break;
    case CAGRAD:
      solve_cagrad<Sync>(S, K, iters, c, t);
      if (t < K) {
        *wt = S.C[t];
        *ax = S.a[t];
      }
      break;
    default:
      *wt = *ax = 1.0 / (double)K;
      break;
  }
}

}  // namespace

}  // namespace bkmoo
