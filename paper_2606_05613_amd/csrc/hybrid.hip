// Pipelined, partly resident resolve: one cooperative kernel in which the
// Gram pass of bucket b+1 runs while the weights of bucket b are computed,
// and part of each bucket (about half at K <= 4) is held on chip between its
// Gram pass and its combine.
//
// Why.  The two-pass path reads every gradient twice, (2K+1)*s*N bytes.  A
// kernel that held a whole bucket on chip (a 25 MiB K=4 bf16 bucket is ~60%
// of the chip's registers and LDS) would leave room for nothing else: every
// workgroup would idle while the bucket's Gram is reduced and its problem
// solved.  Holding about half of each workgroup's share of a bucket leaves
// room for two buckets: the data of bucket b+1 streams in while bucket b's
// weights are produced, and bucket b's combine re-reads only the part it did
// not keep.
//
// How.  K <= 8.  Workgroups of 256 threads, two per CU (two can sit in
// different phases, so one computes while the other streams).  The first
// kHybridSolvers workgroups of the grid hold no data: solver j takes buckets
// j, j + kHybridSolvers, ...; it waits until every data workgroup
// has stored its partial Gram of the bucket, adds the partials in a fixed
// order, solves on one wavefront and publishes the weights with a flag.  A
// data workgroup owns one segment slot of every bucket, or none (the host's
// HybLayout: GD data workgroups; segments are whole multiples of one vector
// per thread; equal, or longer for the workgroups dispatched first onto
// their CU when the host asks for a skew; with long solves the solvers' CU
// mates hold no segment).  Of its segment it
// keeps the first NB = NR + NL vectors per task row and thread in one of two
// buffers (registers and LDS) and streams the rest, NS vectors per row at a
// time (hyb_regs, hyb_lds, hyb_stream).  Per workgroup the order is
//   Gram(0) -> A, Gram(1) -> B, Combine(0) <- A, Gram(2) -> A, Combine(1) <- B, ...
// A Gram phase computes the segment's partial Gram (the same fp32 arithmetic
// and fixed-order reductions as the streaming pass), stores it in the
// segment's slot and arrives at the bucket's counter.  A combine phase waits
// for the bucket's flag (bounded) and writes the update from the buffer and
// from a second read of the streamed part.  A wait that runs out sets the
// error word's timeout bit and the bucket's weights (solver) or the
// workgroup's copy of them (data workgroup) become NaN, so the call ends and
// the affected update is NaN instead of silently wrong.  The Gram phase reads
// the first ~170 MiB of a bucket's streamed part with the temporal cache
// policy, so that second read mostly hits the Infinity Cache, and the rest
// with the streaming one; solver waves, and data waves in a combine phase,
// run at raised wave priority.
//
// No cycle of waits: a data workgroup waits for bucket b's weights only after
// it has arrived for bucket b+1, every data workgroup arrives for bucket b
// before it waits for bucket b-1's, and the solvers wait only for arrivals;
// the cooperative launch keeps every workgroup resident.  Two sets of
// partial slots suffice (bucket b uses set b & 1): a data workgroup writes
// bucket b+2's partial in Gram(b+2), after its Combine(b) saw bucket b's
// flag, which a solver sets only after it has read bucket b's partials; a
// workgroup with no segment in bucket b skips that wait, and its slot is
// one the solver of bucket b does not read (slots past the bucket's last
// segment).  The solver sets kFlagCopies copies of each flag; data
// workgroup w polls copy w % kFlagCopies.
// Cross-workgroup data moves through the agent-scope primitives of
// coop_common.h, each hand-off a publish point and an observe point.
//
// The segments depend on the number of data workgroups (and on the skew), so
// results are reproducible on a given device but may differ in the last bits
// between devices with different CU counts (unlike the streaming passes).
#include "combine_impl.h"
#include "coop_common.h"
#include "solve_impl.h"

namespace bkmoo {

namespace {

constexpr int kHybThreads = 256;  // two workgroups per CU
constexpr int kHybWaves = kHybThreads / kWave;
// Partials a solver thread loads at once: with one segment per data
// workgroup (~508) and 25 threads per Gram entry, one round trip.
constexpr int kHybRedBatch = 24;

// Vectors per task row and thread kept in each of the two buffers: registers
// (NR) and LDS (NL), and streamed per row and Gram-phase step (NS).  At
// K <= 4 the two buffers together hold about what the single-read kernel
// holds for one bucket.  Above that registers run short, and keeping loads
// in flight comes first: a wavefront streams NS * K vectors at a time, and
// with fewer than ~10 in flight the kernel falls behind the two passes
// (K = 5 and 6 with NS = 1: 5-25% slower; with NS = 2 and NR = 2: 8-30%
// faster).  K = 8 fits only NR = NL = NS = 1 (its 8 loads in flight).
// With the lane-parallel solvers one more register vector fits without
// spills at K = 5 (bf16, 25 MiB per row, MGDA FW-20: 4.44-4.49 against 5.40
// ms) and at K = 4 with fp32 in and out (GPT-2 shape, PCGrad: 0.515-0.524
// against 0.528-0.541 ms; 1% slower with 41 buckets of 100 MiB).
constexpr int hyb_regs(int K, int DT, int ODT) {
  return K <= 2 ? 9 : K == 3 ? 6 : K == 4 ? (DT == F32 && ODT == F32 ? 5 : 4) : K == 5 ? 3 : K == 6 ? 2 : 1;
}
constexpr int hyb_lds(int K) { return K <= 2 ? 4 : K <= 4 ? 2 : 1; }
constexpr int hyb_stream(int K) { return K <= 7 ? 2 : 1; }
// Streamed bytes per bucket (all data workgroups) read with the temporal
// policy.  Llama-3-8B-shaped K=8 bf16, 25 MiB per row (11 streamed vectors
// per row and thread), ms, CAGrad FW-20 / mean: all temporal 37.10 / 37.55,
// 10 (166 MB) 36.67 / 35.91, 9 36.77 / 35.61, 8 37.05 / 35.62, 7 37.36 /
// 35.97, 5 38.5 / 37.7, none 43.5.  K=4 (at most ~70 MB streamed) is fastest
// with all of it temporal (4-8 of its vectors: 0.7-1.6 ms slower).
constexpr double kHybTemporalMiB = 170.0;

struct HybArgs {
  const int64_t *offs;  // [B+1]
  int B;
  int shift;
  int method, iters;
  double c;
  const int8_t *order;
  double *gram;      // [B][K][K]
  float *weights;    // [B][K]
  double *aux;       // [B][K] or null
  void *out;
  double *partials;  // [2][GD][P]: slot set b & 1 holds bucket b's segment partials
  uint32_t *arrive;  // [B] at stride kSyncStride, zero at launch
  uint32_t *flags;   // [kFlagCopies][B] at stride kSyncStride, zero at launch
  uint32_t *err;
  uint32_t spin_limit;
  HybLayout lay;      // which data workgroup holds which segment
  int tslots;         // streamed vectors per row and thread read with the temporal policy (the rest streaming)
};

// buf_load16 with the default (temporal) cache policy: the line may stay in
// the last-level cache (the 256 MB Infinity Cache), which pays off for data
// read again soon after.
__device__ __forceinline__ u32x4 buf_load16_keep(Rsrc r, uint32_t voff, uint32_t soff) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, 0);
}

// Bounded wait until *p reaches `target` (thread 0 only), SLEEP x 64 cycles
// between polls; on timeout the error word gets kErrTimeout and false is
// returned.  The solvers poll their arrival counters closely (the hand-off
// starts there); data workgroups poll the weights flags about once a
// microsecond, which costs a waiting workgroup little against a ~30 us
// bucket and keeps ~500 pollers off the memory channels.
template <int SLEEP>
__device__ bool wait_at_least(const uint32_t *p, uint32_t target, const HybArgs &a) {
  uint32_t spins = 0;
  while (load_agent(p) < target) {
    __builtin_amdgcn_s_sleep(SLEEP);
    if (++spins >= a.spin_limit) {
      __hip_atomic_fetch_or(a.err, kErrTimeout, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      return false;
    }
  }
  return true;
}

template <int K, int DT, int ODT>
struct Hybrid {
  static constexpr int V = vec_elems(DT);
  static constexpr int NR = hyb_regs(K, DT, ODT);
  static constexpr int NL = hyb_lds(K);
  static constexpr int NB = NR + NL;
  static constexpr int NS = hyb_stream(K);
  static constexpr int P = pairs(K);
  static constexpr int T = kHybThreads;
  static constexpr int EB = elem_bytes(DT);
  static constexpr int NG = T / P;                     // reduction groups per Gram entry

  struct Smem {
    u32x4 lds[2][NL][K][T];
    double red[kHybWaves][P];
    double red2[P][NG];
    Shared S;
    // the bucket's weights, one copy per buffer: Combine(b) and Combine(b+1)
    // can follow each other with no barrier in between (no Gram(b+2) at the
    // end), so thread 0 must not overwrite what other waves may still read
    float wsh[2][K];
  };

  // Gram phase of bucket b into buffer X (reg, hs and sm.lds[X]).
  static __device__ __forceinline__ void gram(const Rows<K> &rows, const HybArgs &a, Smem &sm, int b, int w, int GD,
                              int X, u32x4 (&reg)[NR][K], float (&hs)[K]) {
    const int t = threadIdx.x, lane = t & (kWave - 1), wave = t / kWave;
    const int slot = a.lay.slot(w);
    int64_t lo, hi, nseg;
    a.lay.segment(a.offs[b + 1] - a.offs[b], slot, (int64_t)T * V, lo, hi, nseg);
    lo += a.offs[b];
    hi += a.offs[b];
    const bool has = lo < hi;  // uniform over the workgroup; implies slot >= 0
    float acc[P];
#pragma unroll
    for (int p = 0; p < P; ++p) acc[p] = 0.0f;
    if (has) {
      const Split<V> sp(lo, hi, a.shift);
      if (t < sp.nh + sp.nt) {
        const int64_t n = t < sp.nh ? lo + t : sp.hi_a + (t - sp.nh);
#pragma unroll
        for (int i = 0; i < K; ++i) hs[i] = load_elem<DT>(rows.p[i], n);
        accumulate<K>(acc, hs);
      }
      Rsrc rs[K];
#pragma unroll
      for (int i = 0; i < K; ++i)
        rs[i] = make_rsrc(static_cast<const char *>(rows.p[i]) + sp.lo_a * EB, (uint32_t)sp.nv * 16u);
      const uint32_t voff = (uint32_t)t * 16u;
      // kept vectors (loads past the segment's last vector read zeros)
#pragma unroll
      for (int j = 0; j < NR; ++j) {
#pragma unroll
        for (int i = 0; i < K; ++i) reg[j][i] = buf_load16(rs[i], voff, (uint32_t)(j * T * 16));
      }
      {
        u32x4 stage[NL][K];
#pragma unroll
        for (int j = 0; j < NL; ++j) {
#pragma unroll
          for (int i = 0; i < K; ++i) stage[j][i] = buf_load16(rs[i], voff, (uint32_t)((NR + j) * T * 16));
        }
#pragma unroll
        for (int j = 0; j < NL; ++j) {
#pragma unroll
          for (int i = 0; i < K; ++i) sm.lds[X][j][i][t] = stage[j][i];
        }
      }
      // streamed vectors, NS per row at a time.  The first tslots are
      // loaded with the temporal policy so that the combine's re-read, one
      // bucket later, is mostly served by the last-level cache instead of
      // HBM; the rest with the streaming policy, so that a bucket whose
      // streamed part exceeds that cache does not push them out.
      const int nslot = (sp.nv + T - 1) / T;
      const int jt = NB + a.tslots < nslot ? NB + a.tslots : nslot;
      int j0 = NB;
      for (; j0 < jt; j0 += NS) {
        u32x4 q[NS][K];
#pragma unroll
        for (int u = 0; u < NS; ++u) {
#pragma unroll
          for (int i = 0; i < K; ++i) q[u][i] = buf_load16_keep(rs[i], voff, (uint32_t)((j0 + u) * T * 16));
        }
#pragma unroll
        for (int u = 0; u < NS; ++u) accumulate_vec(acc, q[u]);
      }
      for (; j0 < nslot; j0 += NS) {
        u32x4 q[NS][K];
#pragma unroll
        for (int u = 0; u < NS; ++u) {
#pragma unroll
          for (int i = 0; i < K; ++i) q[u][i] = buf_load16(rs[i], voff, (uint32_t)((j0 + u) * T * 16));
        }
#pragma unroll
        for (int u = 0; u < NS; ++u) accumulate_vec(acc, q[u]);
      }
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        u32x4 q[K];
#pragma unroll
        for (int i = 0; i < K; ++i) q[i] = j < NR ? reg[j < NR ? j : 0][i] : sm.lds[X][j < NR ? 0 : j - NR][i][t];
        accumulate_vec(acc, q);
      }
    }
    // fixed-order reduction: xor butterfly in the wave, waves in order
#pragma unroll
    for (int off = kWave / 2; off >= 1; off >>= 1) {
#pragma unroll
      for (int p = 0; p < P; ++p) acc[p] += __shfl_xor(acc[p], off, kWave);
    }
    if (lane == 0) {
#pragma unroll
      for (int p = 0; p < P; ++p) sm.red[wave][p] = (double)acc[p];
    }
    __syncthreads();
    if (has && t < P) {
      double v = sm.red[0][t];
#pragma unroll
      for (int q = 1; q < kHybWaves; ++q) v += sm.red[q][t];
      store_agent(&a.partials[((int64_t)(b & 1) * GD + slot) * P + t], v);
    }
    __syncthreads();
    if (t == 0) {
      publish_point();  // the slot (stored by wave 0, before the barrier) before the arrival
      __hip_atomic_fetch_add(&a.arrive[(int64_t)b * kSyncStride], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }

  static __device__ __forceinline__ void accumulate_vec(float (&acc)[P], const u32x4 (&q)[K]) {
    float x[K][V];
#pragma unroll
    for (int i = 0; i < K; ++i) decode<DT>(q[i], x[i]);
#pragma unroll
    for (int e = 0; e < V; ++e) {
      float xe[K];
#pragma unroll
      for (int i = 0; i < K; ++i) xe[i] = x[i][e];
      accumulate<K>(acc, xe);
    }
  }

  // The update of one vector, stored with one 16-byte non-temporal global
  // store (the lanes of a wavefront write 1 KiB contiguously) when v < nv.
  static __device__ __forceinline__ void combine_vec(const float (&wv)[K], const u32x4 (&q)[K], void *out,
                                                     int64_t first, bool in_range) {
    float x[K][V];
#pragma unroll
    for (int i = 0; i < K; ++i) decode<DT>(q[i], x[i]);
    float y[V];
#pragma unroll
    for (int e = 0; e < V; ++e) {
      float xe[K];
#pragma unroll
      for (int i = 0; i < K; ++i) xe[i] = x[i][e];
      y[e] = wsum<K, ODT>(wv, xe);
    }
    if (in_range) store_vec<ODT, V>(out, first, y);
  }

  // Combine phase of bucket b from buffer X.
  static __device__ __forceinline__ void combine(const Rows<K> &rows, const HybArgs &a, Smem &sm, int b, int w, int GD,
                                 int X, const u32x4 (&reg)[NR][K], const float (&hs)[K]) {
    const int t = threadIdx.x;
    int64_t lo, hi, nseg;
    a.lay.segment(a.offs[b + 1] - a.offs[b], a.lay.slot(w), (int64_t)T * V, lo, hi, nseg);
    lo += a.offs[b];
    hi += a.offs[b];
    if (lo >= hi) return;  // no segment in this bucket: no weights needed (uniform)
    const Split<V> sp(lo, hi, a.shift);
    Rsrc rs[K];
#pragma unroll
    for (int i = 0; i < K; ++i)
      rs[i] = make_rsrc(static_cast<const char *>(rows.p[i]) + sp.lo_a * EB, (uint32_t)sp.nv * 16u);
    const uint32_t voff = (uint32_t)t * 16u;
    const int nslot = (sp.nv + T - 1) / T;
    // The first re-read vector does not depend on the weights: loading it
    // before the wait for them takes its latency off the combine, and the
    // loop below keeps one vector per row in flight ahead of the one it
    // combines (loads past the segment read zeros and are not used).
    u32x4 qn[K];
#pragma unroll
    for (int i = 0; i < K; ++i) qn[i] = buf_load16(rs[i], voff, (uint32_t)(NB * T * 16));
    if (t == 0) {
      const bool ok =
          wait_at_least<32>(&a.flags[((int64_t)(w % kFlagCopies) * a.B + b) * kSyncStride], 1u, a);
      observe_point();  // the weights after the flag
#pragma unroll
      for (int i = 0; i < K; ++i)
        sm.wsh[X][i] = ok ? load_agent(&a.weights[(int64_t)b * K + i]) : __builtin_nanf("");
    }
    __syncthreads();
    // The two workgroups of a CU drift into different phases, and the wave
    // arbiter favours the older one; the combine (whose end releases the
    // next Gram phase and whose writes are the slowest traffic) goes first.
    __builtin_amdgcn_s_setprio(1);
    float wv[K];
#pragma unroll
    for (int i = 0; i < K; ++i) wv[i] = sm.wsh[X][i];
    if (t < sp.nh + sp.nt) {
      const int64_t n = t < sp.nh ? lo + t : sp.hi_a + (t - sp.nh);
      store_elem<ODT>(a.out, n, wsum<K, ODT>(wv, hs));
    }
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      u32x4 q[K];
#pragma unroll
      for (int i = 0; i < K; ++i) q[i] = j < NR ? reg[j < NR ? j : 0][i] : sm.lds[X][j < NR ? 0 : j - NR][i][t];
      const int v = j * T + t;
      combine_vec(wv, q, a.out, sp.lo_a + (int64_t)v * V, v < sp.nv);
    }
    // the re-read is the data's last use: streaming policy
    for (int j0 = NB; j0 < nslot; ++j0) {
      u32x4 q[K];
#pragma unroll
      for (int i = 0; i < K; ++i) q[i] = qn[i];
#pragma unroll
      for (int i = 0; i < K; ++i) qn[i] = buf_load16(rs[i], voff, (uint32_t)((j0 + 1) * T * 16));
      const int v = j0 * T + t;
      combine_vec(wv, q, a.out, sp.lo_a + (int64_t)v * V, v < sp.nv);
    }
    __builtin_amdgcn_s_setprio(0);
  }

  // Solver workgroup: buckets j, j + kHybridSolvers, ... (j = w - GD).
  static __device__ void solve(const HybArgs &a, Smem &sm, int w, int GD) {
    const int t = threadIdx.x, wave = t / kWave;
    __shared__ int ok_sh;
    // a solve sits on the critical path of every data workgroup and shares
    // its CU with one: its waves go first
    __builtin_amdgcn_s_setprio(3);
    for (int b = w - GD; b < a.B; b += kHybridSolvers) {
      if (t == 0) {
        ok_sh = wait_at_least<1>(&a.arrive[(int64_t)b * kSyncStride], (uint32_t)GD, a) ? 1 : 0;
        observe_point();  // the partial slots after the arrivals (loaded after the barrier)
      }
      __syncthreads();
      int64_t slo, shi, nseg;
      a.lay.segment(a.offs[b + 1] - a.offs[b], 0, (int64_t)T * V, slo, shi, nseg);
      // segment slots in a fixed order: group g of entry p sums segments
      // g, g+NG, ... ascending, then entry p sums its groups ascending
      if (t < P * NG) {
        const int p = t / NG, g = t % NG;
        double v = 0.0;
        for (int64_t s = g; s < nseg; s += kHybRedBatch * NG) {  // device-coherent loads in flight
          double q[kHybRedBatch];
#pragma unroll
          for (int u = 0; u < kHybRedBatch; ++u) {
            const int64_t ss = s + (int64_t)u * NG;
            q[u] = ss < nseg ? load_agent(&a.partials[((int64_t)(b & 1) * GD + ss) * P + p]) : 0.0;
          }
#pragma unroll
          for (int u = 0; u < kHybRedBatch; ++u) v += q[u];
        }
        sm.red2[p][g] = v;
      }
      if (t == 0) sm.S.bad = ok_sh ? 0 : 1;
      __syncthreads();
      if (t < P) {
        double v = 0.0;
        for (int g = 0; g < NG; ++g) v += sm.red2[t][g];
        if (!ok_sh) v = __builtin_nan("");  // some partials may be missing
        int i = 0, rem = t;
        while (rem >= K - i) {
          rem -= K - i;
          ++i;
        }
        const int j = i + rem;
        sm.S.G[i * K + j] = v;
        sm.S.G[j * K + i] = v;
        a.gram[((int64_t)b * K + i) * K + j] = v;
        a.gram[((int64_t)b * K + j) * K + i] = v;
        if (!__builtin_isfinite(v)) sm.S.bad = 1;
      }
      __syncthreads();
      if (wave == 0) {
        double wt = 0.0, ax = 0.0;
        if (a.method == PCGRAD || sm.S.bad) {
          solver_run<WaveSync>(sm.S, K, a.method, a.iters, a.c, a.order, b, t, &wt, &ax);
        } else if (a.method == MGDA) {
          wt = ax = lane_solve_mgda<K>(sm.S.G, a.iters, t);
        } else if (a.method == CAGRAD) {
          lane_solve_cagrad<K>(sm.S.G, a.iters, a.c, t, &wt, &ax);
        } else {
          wt = ax = 1.0 / (double)K;
        }
        // lane i < K holds task i's weight and variable; thread 0 gathers them
        // and publishes the weights, then the flag
        float wk[K];
        double xk[K];
#pragma unroll
        for (int i = 0; i < K; ++i) {
          wk[i] = (float)__shfl(wt, i, kWave);
          xk[i] = __shfl(ax, i, kWave);
        }
        if (t == 0) {
#pragma unroll
          for (int i = 0; i < K; ++i) {
            store_agent(&a.weights[(int64_t)b * K + i], wk[i]);
            if (a.aux) a.aux[(int64_t)b * K + i] = xk[i];
          }
          publish_point();  // the weights before the flags
#pragma unroll
          for (int r = 0; r < kFlagCopies; ++r) store_agent(&a.flags[((int64_t)r * a.B + b) * kSyncStride], 1u);
        }
      }
      __syncthreads();
    }
  }
};

template <int K, int DT, int ODT>
__global__ __launch_bounds__(kHybThreads, 2) void hybrid_kernel(Rows<K> rows, HybArgs a) {
  using H = Hybrid<K, DT, ODT>;
  __shared__ typename H::Smem sm;
  // the solvers are the lowest block indices: dispatched first, they are the
  // older workgroup on their CU, which the wave arbiter favours
  const int G = gridDim.x, GD = G - kHybridSolvers;
  const int w = (int)blockIdx.x < kHybridSolvers ? GD + (int)blockIdx.x : (int)blockIdx.x - kHybridSolvers;
  if (*a.err & kErrOffsets) {
    // the schedule rejected the offsets: NaN Gram and weights, no update
    if (w == 0) {
      const double nan = __builtin_nan("");
      for (int64_t i = threadIdx.x; i < (int64_t)a.B * K * K; i += kHybThreads) a.gram[i] = nan;
      for (int64_t i = threadIdx.x; i < (int64_t)a.B * K; i += kHybThreads) {
        a.weights[i] = (float)nan;
        if (a.aux) a.aux[i] = nan;
      }
    }
    return;
  }
  if (w >= GD) {
    H::solve(a, sm, w, GD);
    return;
  }
  u32x4 regA[H::NR][K], regB[H::NR][K];
  float hsA[K], hsB[K];
  if (a.B > 0) H::gram(rows, a, sm, 0, w, GD, 0, regA, hsA);
  for (int b = 0; b < a.B; b += 2) {
    if (b + 1 < a.B) H::gram(rows, a, sm, b + 1, w, GD, 1, regB, hsB);
    H::combine(rows, a, sm, b, w, GD, 0, regA, hsA);
    if (b + 1 < a.B) {
      if (b + 2 < a.B) H::gram(rows, a, sm, b + 2, w, GD, 0, regA, hsA);
      H::combine(rows, a, sm, b + 1, w, GD, 1, regB, hsB);
    }
  }
}

template <int K, int DT, int ODT>
hipError_t launch_hybrid_t(const void *const *row_ptrs, const HybArgs &a, int grid, hipStream_t s) {
  Rows<K> rows;
  for (int i = 0; i < K; ++i) rows.p[i] = row_ptrs[i];
  HybArgs args = a;
  void *kargs[] = {&rows, &args};
  return hipLaunchCooperativeKernel(reinterpret_cast<const void *>(&hybrid_kernel<K, DT, ODT>),
                                    dim3((unsigned)grid), dim3(kHybThreads), kargs, 0, s);
}

template <int K, int DT, int ODT>
int hybrid_grid_t() {
  int occ = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, hybrid_kernel<K, DT, ODT>, kHybThreads, 0) !=
      hipSuccess)
    return 0;
  // two workgroups per CU, the layout the kernel is built for (a lighter
  // instantiation could fit three, which only adds contention)
  const int g = (occ < 2 ? occ : 2) * device_cu_count();
  return g > 2 * kHybridSolvers ? g : 0;
}

}  // namespace

int hybrid_grid(int K, int dt, int out_dt) {
#define BKMOO_HYB_CASE(k)                                                                           \
  case k:                                                                                           \
    if (dt == F32) return out_dt == F32 ? hybrid_grid_t<k, F32, F32>() : hybrid_grid_t<k, F32, BF16>(); \
    return out_dt == F32 ? hybrid_grid_t<k, BF16, F32>() : hybrid_grid_t<k, BF16, BF16>();
  switch (K) {
    BKMOO_HYB_CASE(2)
    BKMOO_HYB_CASE(3)
    BKMOO_HYB_CASE(4)
    BKMOO_HYB_CASE(5)
    BKMOO_HYB_CASE(6)
    BKMOO_HYB_CASE(7)
    BKMOO_HYB_CASE(8)
    default: return 0;
  }
#undef BKMOO_HYB_CASE
}

int hybrid_data_workgroups(int grid) { return grid - kHybridSolvers; }

// The dispatcher gives every CU one workgroup before it gives any a second,
// so with two per CU the first (cu count - solvers) data workgroups are the
// older resident of their CU.
int hybrid_older_workgroups(int grid) {
  const int cus = device_cu_count();
  return grid == 2 * cus && cus > kHybridSolvers ? cus - kHybridSolvers : 0;
}

int64_t hybrid_held_elems(int K, int dt, int out_dt) {
  return (int64_t)kHybThreads * (hyb_regs(K, dt, out_dt) + hyb_lds(K)) * vec_elems(dt);
}

int64_t hybrid_unit_elems(int dt) { return (int64_t)kHybThreads * vec_elems(dt); }

hipError_t launch_hybrid(int K, int dt, int out_dt, const void *const *rows, const int64_t *offs, int B,
                         int shift, int method, int iters, double c, const int8_t *order, double *gram,
                         float *weights, double *aux, void *out, double *partials, uint32_t *arrive,
                         uint32_t *flags, uint32_t *err, uint32_t spin_limit, int grid,
                         const HybLayout &layout, hipStream_t s) {
  const double per_slot = (double)(layout.nslots > 0 ? layout.nslots : 1) * kHybThreads * 16.0 * K;
  const HybArgs a{offs, B, shift, method, iters, c, order, gram, weights, aux, out,
                  partials, arrive, flags, err, spin_limit, layout,
                  (int)(kHybTemporalMiB * (1 << 20) / per_slot)};
#define BKMOO_HYB_CASE(k)                                                                        \
  case k:                                                                                        \
    if (dt == F32)                                                                               \
      return out_dt == F32 ? launch_hybrid_t<k, F32, F32>(rows, a, grid, s)                      \
                           : launch_hybrid_t<k, F32, BF16>(rows, a, grid, s);                    \
    return out_dt == F32 ? launch_hybrid_t<k, BF16, F32>(rows, a, grid, s)                       \
                         : launch_hybrid_t<k, BF16, BF16>(rows, a, grid, s);
  switch (K) {
    BKMOO_HYB_CASE(2)
    BKMOO_HYB_CASE(3)
    BKMOO_HYB_CASE(4)
    BKMOO_HYB_CASE(5)
    BKMOO_HYB_CASE(6)
    BKMOO_HYB_CASE(7)
    BKMOO_HYB_CASE(8)
    default: return hipErrorInvalidValue;
  }
#undef BKMOO_HYB_CASE
}

}  // namespace bkmoo
