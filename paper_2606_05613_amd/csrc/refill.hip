// Single-buffer pipelined resolve ("refill"): one cooperative kernel that
// keeps most of each bucket on chip in one buffer, refilled slot by slot
// with the next bucket as the current one is combined.
//
// Why.  The two-buffer pipelined kernel (hybrid.hip) holds part of two
// buckets at once, so each bucket keeps at most half of what fits on chip
// and the rest is read twice.  Here the part of bucket b+1 that is not kept
// is read first, while bucket b's weights are being produced; then each kept
// slot of bucket b is combined and immediately reloaded with the same slot
// of bucket b+1.  Only one bucket's kept part is ever resident, so the kept
// share can be about twice as large; the price is a shorter window to hide
// the per-bucket hand-off in (the streamed parts of two buckets instead of a
// whole Gram phase), so the hand-off is cut to the fewest memory round trips.
//
// How.  K <= 10.  Workgroups of 256 threads, two per CU.  The first
// `nsolv` workgroups of the grid hold no data and solve buckets j, j + nsolv,
// ...; every other workgroup owns one segment slot of every bucket (equal
// segments in whole units of one vector per thread, the host's HybLayout).
// Of its segment a data workgroup keeps the first `keep` vectors per task row
// and thread (at most NR in registers plus NL in LDS) and streams the rest.
// Per data workgroup and bucket b the order is
//   G1(b+1)   stream the not-kept part of bucket b+1 (Gram sums only; the
//             temporal cache policy leaves it in the last-level cache)
//   wait      bucket b's weights
//   C1/G2     for each kept slot: combine bucket b's slot, then load bucket
//             b+1's slot into the same registers or LDS and add its products
//   arrive    bucket b+1's partial Gram to its slot
//   C2(b)     re-read bucket b's streamed part and combine it
// so bucket b+1's hand-off runs under C2(b) and G1(b+2).
//
// Hand-offs.  A data workgroup stores its partial Gram in its slot with
// agent-scope stores, waits for them (publish point) and bumps the bucket's
// arrival counter; the bucket's solver waits for every segment's arrival,
// adds the partials in a fixed order, solves on one wavefront and stores the
// K weights with agent-scope stores into kFlagCopies records that were
// filled with "pending" marks (signalling NaNs, which no conversion
// produces) before the launch; data workgroup w polls record w % kFlagCopies
// until no weight is pending, so the weights arrive with the poll.  Two sets
// of partial slots suffice (bucket b uses set b & 1): a data workgroup
// writes bucket b+2's partial after it has seen bucket b's weights (it
// waits for them in the period before), which the solver stores only after
// it has read bucket b's partials.  A workgroup with no segment in a bucket
// neither arrives nor waits for it; its slot is one the bucket's solver
// does not read.  Every wait is bounded: a solver whose wait runs out
// publishes NaN weights, a data workgroup whose wait runs out combines with
// NaN weights, and both set the error word's timeout bit.
//
// No cycle of waits: bucket b's weights need every arrival for b, and a data
// workgroup arrives for b right after its wait for bucket b-1's weights;
// solvers wait only for arrivals; the cooperative launch keeps every
// workgroup resident.
#include "combine_impl.h"
#include "coop_common.h"
#include "refill.h"
#include "solve_impl.h"

namespace bkmoo {

namespace {

constexpr int kRefThreads = 256;  // two workgroups per CU
constexpr int kRefWaves = kRefThreads / kWave;
constexpr int kRefMaxSlots = 512;  // segment slots (data workgroups) per bucket at most
constexpr int kRefMaxSlotsEst = 508;  // data workgroups of a 256-CU device
// Pending mark of a weight: a signalling NaN with payload 1, which an fp64
// -> fp32 conversion never produces (a NaN comes out quiet).
constexpr uint32_t kWeightPending = 0x7f800001u;

// Vectors per task row and thread kept on chip (registers NR, LDS NL),
// streamed per row and step (NS), and kept slots between a refill load and
// the addition of its products (lag): the registers and LDS the two-buffer
// kernel spreads over two buckets, as far as they compile without spills.
// At K = 4 eight kept register vectors with a lag of one slot beat seven
// with a lag of two (K=4 bf16 25 MiB MGDA FW-20, two groups: 16.82-16.92
// against 17.13-17.18 ms), and nine (4 VGPRs spilled: three scratch
// stores and three loads in the kernel) beat eight (alternating processes:
// 16.27-16.50 against 16.56-16.89 ms); ten spill 20 VGPRs and lose
// (17.05-17.55 ms).  At K = 9 and 10 with fp32 in and out a second kept
// register vector (13 VGPRs spilled at K = 10) beat one (K=10 fp32, MGDA
// FW-20, alternating processes: 1 MiB buckets 16.5-16.6 against 18.2-18.3
// ms, 5 MiB 17.5 against 18.8, 25 MiB 19.2 against 20.3-20.5, 100 MiB 21.5
// against 24.7); with bf16 on either side it spills 80-140 VGPRs (bf16 in
// and out spills 50 already with one).
// At K = 5..7 more register vectors fit without spills (bf16, 5 MiB per
// row, MGDA FW-20: K=5 six 4.60 against four 4.89 ms, K=7 three 4.75
// against two 4.95; K=6 five spill 2-12 VGPRs and gain nothing).
constexpr int ref_regs(int K, int DT, int ODT) {
  return K <= 2 ? 16 : K == 3 ? 10 : K == 4 ? 9 : K == 5 ? 6 : K == 6 ? 4 : K == 7 ? 3 : K == 8 ? 2
       : DT == F32 && ODT == F32 ? 2 : 1;
}
constexpr int ref_lds(int K) { return K <= 2 ? 8 : K <= 4 ? 4 : K <= 8 ? 2 : 1; }
constexpr int ref_stream(int K) { return K <= 7 ? 2 : 1; }
constexpr int ref_lag(int K) { return K <= 3 ? 2 : 1; }
// Vectors per row and thread every segment streams rather than keeps: the
// streamed parts of two buckets are the window that hides a bucket's
// hand-off (at K <= 4, 2..6 measured alike: the one-bucket loop, not the
// window, sets the pace there; above K = 4 the kept share is capped by NB
// first).
constexpr int kRefStreamMin = 4;
// Streamed bytes per round read with the temporal policy.  K=10 fp32, 25
// MiB per row (263 buckets, one group), CAGrad FW-20, ms: all 11 streamed
// vectors per row temporal 22.23, 8 (166 MB a round) 20.58, 5 20.97, 3
// 21.60, none 23.45; 5 and 1 MiB per row (their whole streamed part, 183
// and 117 MB a round) lose 0.3-1 ms with fewer.
constexpr double kRefTemporalMiB = 170.0;
// Partial entries a solver thread loads at once (16-byte device-coherent
// loads in flight): all of its share of the slots, at most 24 (registers).
constexpr int ref_red_batch(int ng) { return (kRefMaxSlotsEst + ng - 1) / ng < 24 ? (kRefMaxSlotsEst + ng - 1) / ng : 24; }

struct RefArgs {
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
  double *partials;  // [2][nslots][P rounded up to even]
  uint32_t *arrive;  // [B] at stride kSyncStride, zero at launch (hint)
  uint32_t *recs;    // [kFlagCopies][B] records of K weights at stride kSyncStride, pending-marked
  uint32_t *err;
  uint32_t spin_limit;
  HybLayout lay;     // segment slots of one group (equal segments)
  int nsolv;         // solver workgroups
  int groups;        // data workgroup groups: group g takes buckets g, g + groups, ...
  int tslots;        // streamed vectors per row and thread read with the temporal policy (the rest streaming)
};

// Cache policy of device-coherent loads (sc1, as agent-scope atomic loads).
constexpr int kCoherent = 16;

__device__ __forceinline__ u32x4 buf_load16_keep(Rsrc r, uint32_t voff, uint32_t soff) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, 0);
}

__device__ __forceinline__ void note_timeout(const RefArgs &a) {
  __hip_atomic_fetch_or(a.err, kErrTimeout, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Bounded poll of a weight record until none of its K words is pending;
// x receives the words.  SLEEP x 64 cycles between polls.
template <int K, int SLEEP>
__device__ bool poll_record(const uint32_t *rec, uint32_t (&x)[K], const RefArgs &a) {
  uint32_t spins = 0;
  for (;;) {
    bool ready = true;
#pragma unroll
    for (int i = 0; i < K; ++i) {
      x[i] = load_agent(rec + i);
      ready = ready && x[i] != kWeightPending;
    }
    if (ready) return true;
    __builtin_amdgcn_s_sleep(SLEEP);
    if (++spins >= a.spin_limit) {
      note_timeout(a);
      return false;
    }
  }
}

template <int K, int DT, int ODT>
struct Refill {
  static constexpr int V = vec_elems(DT);
  static constexpr int NR = ref_regs(K, DT, ODT);
  static constexpr int NL = ref_lds(K);
  static constexpr int NB = NR + NL;
  static constexpr int NS = ref_stream(K);
  static constexpr int LAG = ref_lag(K);
  static constexpr int P = pairs(K);
  static constexpr int T = kRefThreads;
  static constexpr int EB = elem_bytes(DT);
  // partial slots hold P entries at a stride of PP (even): a solver thread
  // reads a pair of entries with one 16-byte load
  static constexpr int PP = P + (P & 1);
  static constexpr int P2 = PP / 2;
  static constexpr int NG = T / P2;  // solver threads per pair of entries
  static constexpr int RB = ref_red_batch(NG);

  struct Smem {
    u32x4 lds[NL][K][T];   // kept vectors; thread t only touches column t
    double red[2][kRefWaves][P];
    double red2[P][NG];
    Shared S;
    float wsh[2][K];
  };

  // One data workgroup's share of a bucket.
  struct Geo {
    Rsrc rs[K];
    int64_t lo, lo_a, hi_a;
    int nv, nh, nt, nslot, keep;
    bool has;
  };

  static __device__ __forceinline__ Geo geo(const Rows<K> &rows, const RefArgs &a, int b, int slot) {
    Geo g;
    int64_t lo, hi, nseg;
    a.lay.segment(a.offs[b + 1] - a.offs[b], slot, (int64_t)T * V, lo, hi, nseg);
    lo += a.offs[b];
    hi += a.offs[b];
    g.has = lo < hi;
    const Split<V> sp(lo, hi, a.shift);
    g.lo = lo;
    g.lo_a = sp.lo_a;
    g.hi_a = sp.hi_a;
    g.nv = g.has ? sp.nv : 0;
    g.nh = g.has ? sp.nh : 0;
    g.nt = g.has ? sp.nt : 0;
    g.nslot = (g.nv + T - 1) / T;
    int keep = g.nslot - kRefStreamMin;
    g.keep = keep < 0 ? 0 : keep > NB ? NB : keep;
#pragma unroll
    for (int i = 0; i < K; ++i)
      g.rs[i] = make_rsrc(static_cast<const char *>(rows.p[i]) + sp.lo_a * EB, (uint32_t)g.nv * 16u);
    return g;
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

  // The scalar head and tail elements (held in hs) and the streamed
  // vectors [keep, nslot) of a share: Gram sums only.  The first `tslots`
  // are read with the temporal policy, so that their second read (C2) finds
  // them in the last-level cache; the rest with the streaming policy, so
  // that they do not push those out.
  static __device__ __forceinline__ void stream_in(const Rows<K> &rows, const Geo &g, int tslots, float (&acc)[P],
                                                   float (&hs)[K]) {
    const int t = threadIdx.x;
    if (t < g.nh + g.nt) {
      const int64_t n = t < g.nh ? g.lo + t : g.hi_a + (t - g.nh);
#pragma unroll
      for (int i = 0; i < K; ++i) hs[i] = load_elem<DT>(rows.p[i], n);
      accumulate<K>(acc, hs);
    }
    const uint32_t voff = (uint32_t)t * 16u;
    const int jt = g.keep + tslots < g.nslot ? g.keep + tslots : g.nslot;
    int j0 = g.keep;
    for (; j0 < jt; j0 += NS) {
      u32x4 q[NS][K];
#pragma unroll
      for (int u = 0; u < NS; ++u) {
#pragma unroll
        for (int i = 0; i < K; ++i) q[u][i] = buf_load16_keep(g.rs[i], voff, (uint32_t)((j0 + u) * T * 16));
      }
#pragma unroll
      for (int u = 0; u < NS; ++u) accumulate_vec(acc, q[u]);
    }
    for (; j0 < g.nslot; j0 += NS) {
      u32x4 q[NS][K];
#pragma unroll
      for (int u = 0; u < NS; ++u) {
#pragma unroll
        for (int i = 0; i < K; ++i) q[u][i] = buf_load16(g.rs[i], voff, (uint32_t)((j0 + u) * T * 16));
      }
#pragma unroll
      for (int u = 0; u < NS; ++u) accumulate_vec(acc, q[u]);
    }
  }

  // First bucket only: load the kept vectors [0, keep) and add their products.
  static __device__ __forceinline__ void keep_in(const Geo &g, Smem &sm, u32x4 (&reg)[NR][K], float (&acc)[P]) {
    const int t = threadIdx.x;
    const uint32_t voff = (uint32_t)t * 16u;
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      if (j < g.keep) {
#pragma unroll
        for (int i = 0; i < K; ++i) {
          const u32x4 x = buf_load16(g.rs[i], voff, (uint32_t)(j * T * 16));
          if (j < NR) reg[j < NR ? j : 0][i] = x;
          else sm.lds[j < NR ? 0 : j - NR][i][t] = x;
        }
      }
    }
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      if (j < g.keep) {
        u32x4 q[K];
#pragma unroll
        for (int i = 0; i < K; ++i) q[i] = j < NR ? reg[j < NR ? j : 0][i] : sm.lds[j < NR ? 0 : j - NR][i][t];
        accumulate_vec(acc, q);
      }
    }
  }

  // C1(b) / G2(b+1): combine the kept slot j of the current share (cur),
  // then load slot j of the next share (nxt) into the same storage; the
  // products of slot j are added kRefLag slots later.
  static __device__ __forceinline__ void refill(const RefArgs &a, const Geo &gc, const Geo &gn, const float (&wv)[K],
                                                Smem &sm, u32x4 (&reg)[NR][K], float (&acc)[P]) {
    const int t = threadIdx.x;
    const uint32_t voff = (uint32_t)t * 16u;
    u32x4 stage[LAG][K];
#pragma unroll
    for (int j = 0; j < NB + LAG; ++j) {
      const int jj = j - LAG;
      if (jj >= 0 && jj < gn.keep) {
        const int r = jj >= 0 && jj < NR ? jj : 0;
        const int l = jj >= NR ? jj - NR : 0;
        const int s = jj >= 0 ? jj % LAG : 0;
        u32x4 q[K];
#pragma unroll
        for (int i = 0; i < K; ++i) q[i] = jj < NR ? reg[r][i] : stage[s][i];
        if (jj >= NR) {
#pragma unroll
          for (int i = 0; i < K; ++i) sm.lds[l][i][t] = stage[s][i];
        }
        accumulate_vec(acc, q);
      }
      if (j < NB) {
        const int r = j < NR ? j : 0;
        const int l = j >= NR && j < NB ? j - NR : 0;
        if (j < gc.keep) {
          u32x4 q[K];
#pragma unroll
          for (int i = 0; i < K; ++i) q[i] = j < NR ? reg[r][i] : sm.lds[l][i][t];
          const int v = j * T + t;
          combine_vec(wv, q, a.out, gc.lo_a + (int64_t)v * V, v < gc.nv);
        }
        if (j < gn.keep) {
#pragma unroll
          for (int i = 0; i < K; ++i) {
            const u32x4 x = buf_load16(gn.rs[i], voff, (uint32_t)(j * T * 16));
            if (j < NR) reg[r][i] = x;
            else stage[j % LAG][i] = x;
          }
        }
      }
    }
  }

  // C2(b): the head/tail elements (from hs) and the re-read of the streamed
  // vectors [keep, nslot), one vector per row in flight ahead.
  static __device__ __forceinline__ void reread(const RefArgs &a, const Geo &g, const float (&wv)[K],
                                                const float (&hs)[K]) {
    const int t = threadIdx.x;
    if (t < g.nh + g.nt) {
      const int64_t n = t < g.nh ? g.lo + t : g.hi_a + (t - g.nh);
      store_elem<ODT>(a.out, n, wsum<K, ODT>(wv, hs));
    }
    if (g.keep >= g.nslot) return;
    const uint32_t voff = (uint32_t)t * 16u;
    u32x4 qn[K];
#pragma unroll
    for (int i = 0; i < K; ++i) qn[i] = buf_load16(g.rs[i], voff, (uint32_t)(g.keep * T * 16));
    for (int j0 = g.keep; j0 < g.nslot; ++j0) {
      u32x4 q[K];
#pragma unroll
      for (int i = 0; i < K; ++i) q[i] = qn[i];
#pragma unroll
      for (int i = 0; i < K; ++i) qn[i] = buf_load16(g.rs[i], voff, (uint32_t)((j0 + 1) * T * 16));
      const int v = j0 * T + t;
      combine_vec(wv, q, a.out, g.lo_a + (int64_t)v * V, v < g.nv);
    }
  }

  // Parity of bucket b in its group's sequence (selects the partial-slot set
  // and the LDS copies), and the first partial slot of bucket b's group in
  // that set: slots [set][group][slot].
  static __device__ __forceinline__ int par(const RefArgs &a, int b) { return (b / a.groups) & 1; }
  static __device__ __forceinline__ int64_t slot0(const RefArgs &a, int b) {
    return ((int64_t)par(a, b) * a.groups + b % a.groups) * a.lay.nslots;
  }

  // Bucket b's partial Gram of this share: fixed-order reductions (xor
  // butterfly in the wave, waves in order), one agent-scope store per entry
  // into slot `slot` of its group's set (all by wavefront 0), then the
  // arrival.
  static __device__ __forceinline__ void arrive(const RefArgs &a, Smem &sm, int b, int slot, float (&acc)[P]) {
    const int q2 = par(a, b);
    const int t = threadIdx.x, lane = t & (kWave - 1), wave = t / kWave;
#pragma unroll
    for (int off = kWave / 2; off >= 1; off >>= 1) {
#pragma unroll
      for (int p = 0; p < P; ++p) acc[p] += __shfl_xor(acc[p], off, kWave);
    }
    if (lane == 0) {
#pragma unroll
      for (int p = 0; p < P; ++p) sm.red[q2][wave][p] = (double)acc[p];
    }
    __syncthreads();
    if (t < P) {
      double v = sm.red[q2][0][t];
#pragma unroll
      for (int q = 1; q < kRefWaves; ++q) v += sm.red[q2][q][t];
      store_agent(&a.partials[(slot0(a, b) + slot) * PP + t], v);
    }
    if (t == 0) {
      publish_point();  // the slot before the arrival
      __hip_atomic_fetch_add(&a.arrive[(int64_t)b * kSyncStride], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }

  // Bucket b's weights from record w % kFlagCopies (thread 0 polls, the
  // workgroup reads them from LDS after a barrier).
  static __device__ __forceinline__ void wait_weights(const RefArgs &a, Smem &sm, int b, int w, float (&wv)[K]) {
    const int t = threadIdx.x;
    if (t == 0) {
      uint32_t x[K];
      const bool ok = poll_record<K, 32>(a.recs + ((int64_t)(w % kFlagCopies) * a.B + b) * kSyncStride, x, a);
#pragma unroll
      for (int i = 0; i < K; ++i) sm.wsh[par(a, b)][i] = ok ? __uint_as_float(x[i]) : __builtin_nanf("");
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < K; ++i) wv[i] = sm.wsh[par(a, b)][i];
  }

  // Data workgroup w: group w % groups, slot w / groups of that group's
  // buckets (none when the grid does not divide evenly).
  static __device__ void data(const Rows<K> &rows, const RefArgs &a, Smem &sm, int w) {
    const int G = a.groups, grp = w % G, slot = w / G;
    if (slot >= a.lay.nslots || grp >= a.B) return;
    u32x4 reg[NR][K];
    float hs_cur[K], hs_nxt[K];
#pragma unroll
    for (int i = 0; i < K; ++i) hs_cur[i] = hs_nxt[i] = 0.0f;
    float acc[P];
    Geo gn = geo(rows, a, grp, slot);
    if (gn.has) {
#pragma unroll
      for (int p = 0; p < P; ++p) acc[p] = 0.0f;
      stream_in(rows, gn, a.tslots, acc, hs_nxt);
      keep_in(gn, sm, reg, acc);
      arrive(a, sm, grp, slot, acc);
    }
    for (int b = grp; b < a.B; b += G) {
      const Geo gc = gn;
#pragma unroll
      for (int i = 0; i < K; ++i) hs_cur[i] = hs_nxt[i];
      if (b + G < a.B) {
        gn = geo(rows, a, b + G, slot);
      } else {
        gn.has = false;
        gn.keep = gn.nslot = gn.nv = gn.nh = gn.nt = 0;
      }
#pragma unroll
      for (int p = 0; p < P; ++p) acc[p] = 0.0f;
      if (gn.has) stream_in(rows, gn, a.tslots, acc, hs_nxt);
      float wv[K];
#pragma unroll
      for (int i = 0; i < K; ++i) wv[i] = 0.0f;
      if (gc.has) wait_weights(a, sm, b, w, wv);
      // the combine (whose end releases the next bucket's arrival and whose
      // writes are the slowest traffic) runs at raised wave priority
      __builtin_amdgcn_s_setprio(1);
      refill(a, gc, gn, wv, sm, reg, acc);
      if (gn.has) arrive(a, sm, b + G, slot, acc);
      if (gc.has) reread(a, gc, wv, hs_cur);
      __builtin_amdgcn_s_setprio(0);
    }
  }

  // Solver workgroup j: buckets j, j + nsolv, ...
  static __device__ void solve(const RefArgs &a, Smem &sm, int j) {
    const int t = threadIdx.x, wave = t / kWave;
    // a solve sits on the critical path of every data workgroup and shares
    // its CU with one: its waves go first
    __builtin_amdgcn_s_setprio(3);
    for (int b = j; b < a.B; b += a.nsolv) {
      int64_t slo, shi, nseg;
      a.lay.segment(a.offs[b + 1] - a.offs[b], 0, (int64_t)T * V, slo, shi, nseg);
      __shared__ int ok_sh;
      if (t == 0) {
        uint32_t spins = 0;
        bool ok = true;
        while (load_agent(&a.arrive[(int64_t)b * kSyncStride]) < (uint32_t)nseg) {
          __builtin_amdgcn_s_sleep(1);
          if (++spins >= a.spin_limit) {
            note_timeout(a);
            ok = false;
            break;
          }
        }
        observe_point();  // the partial slots after the arrivals (loaded after the barrier)
        ok_sh = ok ? 1 : 0;
      }
      __syncthreads();
      // segment slots in a fixed order: group g of entry pair q sums
      // segments g, g+NG, ... ascending (device-coherent 16-byte loads, RB in
      // flight), then each entry sums its groups ascending
      if (t < P2 * NG) {
        const int q = t / NG, g = t % NG;
        const Rsrc rp = make_rsrc(a.partials + slot0(a, b) * PP, (uint32_t)(a.lay.nslots * PP * 8));
        double v0 = 0.0, v1 = 0.0;
        for (int64_t s0 = g; s0 < nseg; s0 += (int64_t)RB * NG) {
          u32x4 x[RB];
#pragma unroll
          for (int u = 0; u < RB; ++u) {
            const int64_t ss = s0 + (int64_t)u * NG;
            x[u] = ss < nseg ? __builtin_amdgcn_raw_buffer_load_b128(rp, (int)((ss * PP + 2 * q) * 8), 0, kCoherent)
                             : u32x4{0u, 0u, 0u, 0u};
          }
#pragma unroll
          for (int u = 0; u < RB; ++u) {
            v0 += __longlong_as_double((long long)(((uint64_t)x[u].y << 32) | x[u].x));
            v1 += __longlong_as_double((long long)(((uint64_t)x[u].w << 32) | x[u].z));
          }
        }
        const double nan = __builtin_nan("");
        sm.red2[2 * q][g] = ok_sh ? v0 : nan;
        if (2 * q + 1 < P) sm.red2[2 * q + 1][g] = ok_sh ? v1 : nan;
      }
      __syncthreads();
      if (t < P) {
        double v = 0.0;
        for (int g = 0; g < NG; ++g) v += sm.red2[t][g];
        int i = 0, rem = t;
        while (rem >= K - i) {
          rem -= K - i;
          ++i;
        }
        const int jj = i + rem;
        sm.S.G[i * K + jj] = v;
        sm.S.G[jj * K + i] = v;
      }
      if (t == 0) sm.S.bad = 0;
      __syncthreads();
      if (t < K * K && !__builtin_isfinite(sm.S.G[t])) sm.S.bad = 1;
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
        // lane i < K holds task i's weight and variable; lanes r <
        // kFlagCopies store record r, then the outputs follow
        float wk[K];
        double xk[K];
#pragma unroll
        for (int i = 0; i < K; ++i) {
          wk[i] = (float)__shfl(wt, i, kWave);
          xk[i] = __shfl(ax, i, kWave);
        }
        publish_point();  // nothing of this bucket in flight when its weights appear
        if (t < kFlagCopies) {
          uint32_t *rec = a.recs + ((int64_t)t * a.B + b) * kSyncStride;
#pragma unroll
          for (int i = 0; i < K; ++i) store_agent(rec + i, __float_as_uint(wk[i]));
        }
        if (t == 0) {
#pragma unroll
          for (int i = 0; i < K; ++i) {
            a.weights[(int64_t)b * K + i] = wk[i];
            if (a.aux) a.aux[(int64_t)b * K + i] = xk[i];
          }
        }
        for (int e = t; e < K * K; e += kWave) a.gram[(int64_t)b * K * K + e] = sm.S.G[e];
      }
      __syncthreads();
    }
  }
};

template <int K, int DT, int ODT>
__global__ __launch_bounds__(kRefThreads, 2) void refill_kernel(Rows<K> rows, RefArgs a) {
  using R = Refill<K, DT, ODT>;
  __shared__ typename R::Smem sm;
  // the solvers are the lowest block indices: dispatched first, they are the
  // older workgroup on their CU, which the wave arbiter favours
  const int w = (int)blockIdx.x - a.nsolv;
  if (*a.err & kErrOffsets) {
    // the schedule rejected the offsets: NaN Gram and weights, no update
    if (w == 0) {
      const double nan = __builtin_nan("");
      for (int64_t i = threadIdx.x; i < (int64_t)a.B * K * K; i += kRefThreads) a.gram[i] = nan;
      for (int64_t i = threadIdx.x; i < (int64_t)a.B * K; i += kRefThreads) {
        a.weights[i] = (float)nan;
        if (a.aux) a.aux[i] = nan;
      }
    }
    return;
  }
  if (w < 0) {
    R::solve(a, sm, (int)blockIdx.x);
    return;
  }
  R::data(rows, a, sm, w);
}

// Zero arrival counters, pending marks in the weight records.
__global__ void refill_init_kernel(uint32_t *arrive, int64_t narrive, uint32_t *recs, int64_t nrec) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < narrive; i += stride) arrive[i] = 0u;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nrec; i += stride)
    recs[i] = kWeightPending;
}

template <int K, int DT, int ODT>
hipError_t launch_refill_t(const void *const *row_ptrs, const RefArgs &a, int grid, hipStream_t s) {
  Rows<K> rows;
  for (int i = 0; i < K; ++i) rows.p[i] = row_ptrs[i];
  RefArgs args = a;
  void *kargs[] = {&rows, &args};
  return hipLaunchCooperativeKernel(reinterpret_cast<const void *>(&refill_kernel<K, DT, ODT>),
                                    dim3((unsigned)grid), dim3(kRefThreads), kargs, 0, s);
}

template <int K, int DT, int ODT>
int refill_grid_t() {
  int occ = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, refill_kernel<K, DT, ODT>, kRefThreads, 0) !=
      hipSuccess)
    return 0;
  const int g = (occ < 2 ? occ : 2) * device_cu_count();
  return g > 2 * kRefMaxGroups && g - kHybridSolvers <= kRefMaxSlots ? g : 0;
}

}  // namespace

int refill_grid(int K, int dt, int out_dt) {
#define BKMOO_REF_CASE(k)                                                                           \
  case k:                                                                                           \
    if (dt == F32) return out_dt == F32 ? refill_grid_t<k, F32, F32>() : refill_grid_t<k, F32, BF16>(); \
    return out_dt == F32 ? refill_grid_t<k, BF16, F32>() : refill_grid_t<k, BF16, BF16>();
  switch (K) {
    BKMOO_REF_CASE(2)
    BKMOO_REF_CASE(3)
    BKMOO_REF_CASE(4)
    BKMOO_REF_CASE(5)
    BKMOO_REF_CASE(6)
    BKMOO_REF_CASE(7)
    BKMOO_REF_CASE(8)
    BKMOO_REF_CASE(9)
    BKMOO_REF_CASE(10)
    default: return 0;
  }
#undef BKMOO_REF_CASE
}

int refill_stream_min() { return kRefStreamMin; }

// The streamed part a round of the groups' buckets leaves in the last-level
// cache for its second read: at most kRefTemporalMiB over all data
// workgroups (one round's is re-read while the next round's is read).
int refill_temporal_slots(int K, int dt, int grid, int groups) {
  const int nsolv = refill_solvers(groups);
  const double per_slot = (double)(grid - nsolv) * kRefThreads * 16.0 * K;  // one vector per row and thread
  const int t = (int)(kRefTemporalMiB * (1 << 20) / per_slot);
  return t < 0 ? 0 : t;
}

// One solver per group, at least four: solver j takes the buckets of group
// j (more groups than solvers would queue one group's ready bucket behind
// another's unfinished one).
int refill_solvers(int groups) { return groups < kHybridSolvers ? kHybridSolvers : groups; }

int64_t refill_held_elems(int K, int dt, int out_dt) {
  return (int64_t)kRefThreads * (ref_regs(K, dt, out_dt) + ref_lds(K)) * vec_elems(dt);
}

hipError_t launch_refill(int K, int dt, int out_dt, const void *const *rows, const int64_t *offs, int B,
                         int shift, int method, int iters, double c, const int8_t *order, double *gram,
                         float *weights, double *aux, void *out, double *partials, uint32_t *arrive,
                         uint32_t *recs, uint32_t *err, uint32_t spin_limit, int grid, int groups,
                         int tslots, hipStream_t s) {
  const int nsolv = refill_solvers(groups);
  if (groups < 1 || grid - nsolv < groups) return hipErrorInvalidValue;
  const HybLayout lay{(grid - nsolv) / groups, 0, 0, 0};
  const RefArgs a{offs, B, shift, method, iters, c, order, gram, weights, aux, out, partials, arrive, recs,
                  err, spin_limit, lay, nsolv, groups, tslots};
  hipLaunchKernelGGL(refill_init_kernel, dim3(64), dim3(256), 0, s, arrive, (int64_t)B * kSyncStride, recs,
                     (int64_t)kFlagCopies * B * kSyncStride);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
#define BKMOO_REF_CASE(k)                                                                        \
  case k:                                                                                        \
    if (dt == F32)                                                                               \
      return out_dt == F32 ? launch_refill_t<k, F32, F32>(rows, a, grid, s)                      \
                           : launch_refill_t<k, F32, BF16>(rows, a, grid, s);                    \
    return out_dt == F32 ? launch_refill_t<k, BF16, F32>(rows, a, grid, s)                       \
                         : launch_refill_t<k, BF16, BF16>(rows, a, grid, s);
  switch (K) {
    BKMOO_REF_CASE(2)
    BKMOO_REF_CASE(3)
    BKMOO_REF_CASE(4)
    BKMOO_REF_CASE(5)
    BKMOO_REF_CASE(6)
    BKMOO_REF_CASE(7)
    BKMOO_REF_CASE(8)
    BKMOO_REF_CASE(9)
    BKMOO_REF_CASE(10)
    default: return hipErrorInvalidValue;
  }
#undef BKMOO_REF_CASE
}

}  // namespace bkmoo
