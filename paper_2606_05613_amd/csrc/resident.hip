// Single-read resolve: Gram, solve and combine of every bucket in one
// cooperative persistent kernel, with each bucket's data held on chip
// between its Gram pass and its combine pass.
//
// Why.  The two-pass path reads every gradient element twice (Gram, then
// combine): (2K+1)*s*N bytes.  The combine of a bucket needs that bucket's
// weights, which need its whole Gram matrix, so a fused pass must keep the
// whole bucket resident until its weights exist.  MI355X has 256 CUs with
// 512 KiB of VGPRs and 160 KiB of LDS each; a 25 MiB-per-task bucket of
// K=4 bf16 gradients (105 MB) fits in about 60% of that.  Holding it there
// cuts HBM traffic to the (K+1)*s*N floor.
//
// How.  One workgroup of 512 threads per CU (LDS-bound), all co-resident.
// A bucket is cut into segments of SEG elements (NR register vectors and NL
// LDS vectors per task row and thread); segment s of bucket b goes to
// workgroup s mod G.  Each workgroup loads its segment, accumulates the
// K(K+1)/2 products in fp32 (same arithmetic as the streaming Gram pass),
// reduces them in a fixed order and stores them in the segment's own slot.
// It then arrives at the bucket's counter; the last to arrive adds the
// segment slots in a fixed order (independent of the grid and of arrival
// order), solves the bucket, and publishes the weights with a flag that the
// others wait for (bounded wait).  Every workgroup then combines straight
// from the registers/LDS it loaded.  A workgroup with more than one segment
// in a bucket (a bucket larger than the chip holds) re-reads its segments
// for the combine: correct, just two reads.
//
// Cross-workgroup data (segment slots, counters, flags, weights) crosses
// XCDs, whose L2 caches are not coherent with each other.  All of it moves
// through agent-scope atomic loads and stores, which the hardware performs
// device-coherently (the sc1 policy), so no L2 writeback or invalidate is
// needed: a writer waits until its stores are acknowledged (vmcnt = 0)
// before it bumps the counter or sets the flag, and a reader issues its
// loads only after observing them (control dependency).  Agent-scope fences
// would instead write back or invalidate a whole XCD's L2 per workgroup and
// bucket.
#include "combine_impl.h"
#include "coop_common.h"
#include "solve_impl.h"

namespace bkmoo {

namespace {

constexpr int kResThreads = 512;
constexpr int kResWaves = kResThreads / kWave;

// Vectors per task row and thread held in registers (NR) and LDS (NL):
// 36 register vectors (144 VGPRs) and 128 KiB of LDS per workgroup.
constexpr int res_regs(int K) { return K <= 2 ? 18 : K == 3 ? 12 : 9; }
constexpr int res_lds(int K) { return K <= 2 ? 8 : K == 3 ? 5 : 4; }

}  // namespace

int64_t resident_segment_elems(int K, int dt) {
  return (int64_t)kResThreads * (res_regs(K) + res_lds(K)) * vec_elems(dt);
}

namespace {

struct ResArgs {
  const int64_t *offs;       // [B+1]
  const int64_t *seg_start;  // [B+1] prefix sum of segments per bucket
  int B;
  int shift;
  int method, iters;
  double c;
  const int8_t *order;
  double *gram;              // [B][K][K]
  float *weights;            // [B][K]
  double *aux;               // [B][K] or null
  void *out;
  double *partials;          // [segments][P]
  uint32_t *arrive;          // [B] at stride kSyncStride, zero at launch
  uint32_t *flags;           // [B] at stride kSyncStride, zero at launch
  uint32_t *err;
  uint32_t spin_limit;
};

template <int K, int DT, int ODT>
__global__ __launch_bounds__(kResThreads, 1) void resident_kernel(Rows<K> rows, ResArgs a) {
  constexpr int V = vec_elems(DT);
  constexpr int NR = res_regs(K);
  constexpr int NL = res_lds(K);
  constexpr int P = pairs(K);
  constexpr int EB = elem_bytes(DT);
  constexpr int T = kResThreads;
  constexpr int64_t SEG = (int64_t)T * (NR + NL) * V;
  constexpr int NG = T / P;  // reduction groups per Gram entry

  __shared__ u32x4 lds[NL][K][T];
  __shared__ double red[kResWaves][P];
  __shared__ double red2[P][NG];
  __shared__ Shared S;
  __shared__ float wsh[K];
  __shared__ int last_sh;

  const int t = threadIdx.x, lane = t & (kWave - 1), wave = t / kWave;
  const int G = gridDim.x, w = blockIdx.x;

  if (*a.err & kErrOffsets) {
    // the schedule rejected the offsets: NaN Gram and weights, no update
    if (w == 0) {
      const double nan = __builtin_nan("");
      for (int64_t i = t; i < (int64_t)a.B * K * K; i += T) a.gram[i] = nan;
      for (int64_t i = t; i < (int64_t)a.B * K; i += T) {
        a.weights[i] = (float)nan;
        if (a.aux) a.aux[i] = nan;
      }
    }
    return;
  }

  u32x4 reg[NR][K];
  float hs[K];  // this thread's head/tail element (threads < nh + nt)

  for (int b = 0; b < a.B; ++b) {
    const int64_t lo_b = a.offs[b], hi_b = a.offs[b + 1];
    const int64_t s0 = a.seg_start[b];
    const int64_t nseg = a.seg_start[b + 1] - s0;
    const bool resident = nseg <= G;  // at most one segment per workgroup

    // ---- Gram pass over this workgroup's segments -------------------------
    for (int64_t s = w; s < nseg; s += G) {
      const int64_t lo = lo_b + s * SEG;
      const int64_t hi = lo + SEG < hi_b ? lo + SEG : hi_b;
      const Split<V> sp(lo, hi, a.shift);
      float acc[P];
#pragma unroll
      for (int p = 0; p < P; ++p) acc[p] = 0.0f;
      if (t < sp.nh + sp.nt) {
        const int64_t n = t < sp.nh ? lo + t : sp.hi_a + (t - sp.nh);
#pragma unroll
        for (int i = 0; i < K; ++i) hs[i] = load_elem<DT>(rows.p[i], n);
        accumulate<K>(acc, hs);
      }
      // Whole vectors through range-checked buffer loads (lanes past the
      // segment's last vector read zeros, which add nothing).  LDS slots
      // first, staged through a few VGPRs, then the register slots, then
      // the products.
      Rsrc rs[K];
#pragma unroll
      for (int i = 0; i < K; ++i)
        rs[i] = make_rsrc(static_cast<const char *>(rows.p[i]) + sp.lo_a * EB, (uint32_t)sp.nv * 16u);
      const uint32_t voff = (uint32_t)t * 16u;
      // all loads in flight together: register slots land in their final
      // registers, LDS slots are staged and written once they arrive
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
          for (int i = 0; i < K; ++i) lds[j][i][t] = stage[j][i];
        }
      }
#pragma unroll
      for (int j = 0; j < NR + NL; ++j) {
        float x[K][V];
#pragma unroll
        for (int i = 0; i < K; ++i)
          decode<DT>(j < NR ? reg[j < NR ? j : 0][i] : lds[j < NR ? 0 : j - NR][i][t], x[i]);
#pragma unroll
        for (int e = 0; e < V; ++e) {
          float xe[K];
#pragma unroll
          for (int i = 0; i < K; ++i) xe[i] = x[i][e];
          accumulate<K>(acc, xe);
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
        for (int p = 0; p < P; ++p) red[wave][p] = (double)acc[p];
      }
      __syncthreads();
      if (t < P) {
        double v = red[0][t];
#pragma unroll
        for (int q = 1; q < kResWaves; ++q) v += red[q][t];
        store_agent(&a.partials[(s0 + s) * P + t], v);
      }
      __syncthreads();
    }

    // ---- arrive; the last workgroup reduces, solves and publishes ---------
    if (t == 0) {
      wait_vm_complete();  // this workgroup's segment slots (written by wave 0) are out
      const uint32_t old =
          __hip_atomic_fetch_add(&a.arrive[(int64_t)b * kSyncStride], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      last_sh = old == (uint32_t)G - 1;
    }
    __syncthreads();
    if (last_sh) {
      // segment slots in a fixed order: group g of entry p sums segments
      // g, g+NG, ... ascending, then entry p sums its groups ascending
      if (t < P * NG) {
        const int p = t / NG, g = t % NG;
        double v = 0.0;
        for (int64_t s = g; s < nseg; s += 8 * NG) {  // 8 device-coherent loads in flight
          double q[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            const int64_t ss = s + (int64_t)u * NG;
            q[u] = ss < nseg ? load_agent(&a.partials[(s0 + ss) * P + p]) : 0.0;
          }
#pragma unroll
          for (int u = 0; u < 8; ++u) v += q[u];
        }
        red2[p][g] = v;
      }
      if (t == 0) S.bad = 0;
      __syncthreads();
      if (t < P) {
        double v = 0.0;
        for (int g = 0; g < NG; ++g) v += red2[t][g];
        int i = 0, rem = t;
        while (rem >= K - i) {
          rem -= K - i;
          ++i;
        }
        const int j = i + rem;
        S.G[i * K + j] = v;
        S.G[j * K + i] = v;
        a.gram[((int64_t)b * K + i) * K + j] = v;
        a.gram[((int64_t)b * K + j) * K + i] = v;
        if (!__builtin_isfinite(v)) S.bad = 1;
      }
      __syncthreads();
      if (wave == 0) {  // one wavefront solves; the others wait at the barrier
        double wt = 0.0, ax = 0.0;
        if (a.method == PCGRAD || S.bad) {
          solver_run<WaveSync>(S, K, a.method, a.iters, a.c, a.order, b, t, &wt, &ax);
        } else {
          // MGDA / CAGrad / mean entirely in registers (every lane the same)
          double Gr[K][K], wr[K], xr[K];
#pragma unroll
          for (int i = 0; i < K; ++i)
#pragma unroll
            for (int j = 0; j < K; ++j) Gr[i][j] = S.G[i * K + j];
          if (a.method == MGDA) {
            reg_solve_mgda<K>(Gr, a.iters, xr);
#pragma unroll
            for (int i = 0; i < K; ++i) wr[i] = xr[i];
          } else if (a.method == CAGRAD) {
            reg_solve_cagrad<K>(Gr, a.iters, a.c, wr, xr);
          } else {
#pragma unroll
            for (int i = 0; i < K; ++i) wr[i] = xr[i] = 1.0 / (double)K;
          }
#pragma unroll
          for (int i = 0; i < K; ++i)
            if (t == i) {
              wt = wr[i];
              ax = xr[i];
            }
        }
        if (t < K) {
          wsh[t] = (float)wt;
          store_agent(&a.weights[(int64_t)b * K + t], (float)wt);
          if (a.aux) a.aux[(int64_t)b * K + t] = ax;
        }
        if (t == 0) {
          wait_vm_complete();  // weights (written by this wavefront) are out
          store_agent(&a.flags[(int64_t)b * kSyncStride], 1u);
        }
      }
      __syncthreads();
    } else {
      if (t == 0) {
        uint32_t spins = 0;
        while (load_agent(&a.flags[(int64_t)b * kSyncStride]) == 0u) {
          __builtin_amdgcn_s_sleep(1);
          if (++spins >= a.spin_limit) {
            __hip_atomic_fetch_or(a.err, kErrTimeout, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            break;
          }
        }
#pragma unroll
        for (int i = 0; i < K; ++i) wsh[i] = load_agent(&a.weights[(int64_t)b * K + i]);
      }
      __syncthreads();
    }
    float wv[K];
#pragma unroll
    for (int i = 0; i < K; ++i) wv[i] = wsh[i];

    // ---- combine from the resident data (re-read if not resident) --------
    for (int64_t s = w; s < nseg; s += G) {
      const int64_t lo = lo_b + s * SEG;
      const int64_t hi = lo + SEG < hi_b ? lo + SEG : hi_b;
      const Split<V> sp(lo, hi, a.shift);
      if (t < sp.nh + sp.nt) {
        const int64_t n = t < sp.nh ? lo + t : sp.hi_a + (t - sp.nh);
        if (!resident) {
#pragma unroll
          for (int i = 0; i < K; ++i) hs[i] = load_elem<DT>(rows.p[i], n);
        }
        store_elem<ODT>(a.out, n, wsum<K, ODT>(wv, hs));
      }
      Rsrc rs[K];
#pragma unroll
      for (int i = 0; i < K; ++i)
        rs[i] = make_rsrc(static_cast<const char *>(rows.p[i]) + sp.lo_a * EB, (uint32_t)sp.nv * 16u);
#pragma unroll
      for (int j = 0; j < NR + NL; ++j) {
        u32x4 q[K];
#pragma unroll
        for (int i = 0; i < K; ++i) {
          if (!resident) q[i] = buf_load16(rs[i], (uint32_t)t * 16u, (uint32_t)(j * T * 16));
          else if (j < NR) q[i] = reg[j < NR ? j : 0][i];
          else q[i] = lds[j < NR ? 0 : j - NR][i][t];
        }
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
        // one 16-byte non-temporal global store per vector: the lanes of a
        // wavefront write 1 KiB contiguously
        if (j * T + t < sp.nv) store_vec<ODT, V>(a.out, sp.lo_a + (int64_t)(j * T + t) * V, y);
      }
    }
    __syncthreads();  // LDS slots and shared scratch are reused by the next bucket
  }
}

template <int K, int DT, int ODT>
hipError_t launch_resident_t(const void *const *row_ptrs, const ResArgs &a, int grid, hipStream_t s) {
  Rows<K> rows;
  for (int i = 0; i < K; ++i) rows.p[i] = row_ptrs[i];
  ResArgs args = a;
  void *kargs[] = {&rows, &args};
  return hipLaunchCooperativeKernel(reinterpret_cast<const void *>(&resident_kernel<K, DT, ODT>),
                                    dim3((unsigned)grid), dim3(kResThreads), kargs, 0, s);
}

template <int K, int DT, int ODT>
int resident_grid_t() {
  int occ = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, resident_kernel<K, DT, ODT>, kResThreads, 0) !=
      hipSuccess)
    return 0;
  return occ * device_cu_count();
}

}  // namespace

// Workgroups the cooperative launch uses (0: this combination cannot run
// resident on this device).
int resident_grid(int K, int dt, int out_dt) {
#define BKMOO_RES_CASE(k)                                                                   \
  case k:                                                                                   \
    if (dt == F32) return out_dt == F32 ? resident_grid_t<k, F32, F32>() : resident_grid_t<k, F32, BF16>(); \
    return out_dt == F32 ? resident_grid_t<k, BF16, F32>() : resident_grid_t<k, BF16, BF16>();
  switch (K) {
    BKMOO_RES_CASE(2)
    BKMOO_RES_CASE(3)
    BKMOO_RES_CASE(4)
    default: return 0;
  }
#undef BKMOO_RES_CASE
}

hipError_t launch_resident(int K, int dt, int out_dt, const void *const *rows, const int64_t *offs,
                           const int64_t *seg_start, int B, int shift, int method, int iters, double c,
                           const int8_t *order, double *gram, float *weights, double *aux, void *out,
                           double *partials, uint32_t *arrive, uint32_t *flags, uint32_t *err,
                           uint32_t spin_limit, int grid, hipStream_t s) {
  const ResArgs a{offs, seg_start, B, shift, method, iters, c, order, gram, weights, aux, out,
                  partials, arrive, flags, err, spin_limit};
#define BKMOO_RES_CASE(k)                                                                          \
  case k:                                                                                          \
    if (dt == F32)                                                                                 \
      return out_dt == F32 ? launch_resident_t<k, F32, F32>(rows, a, grid, s)                      \
                           : launch_resident_t<k, F32, BF16>(rows, a, grid, s);                    \
    return out_dt == F32 ? launch_resident_t<k, BF16, F32>(rows, a, grid, s)                       \
                         : launch_resident_t<k, BF16, BF16>(rows, a, grid, s);
  switch (K) {
    BKMOO_RES_CASE(2)
    BKMOO_RES_CASE(3)
    BKMOO_RES_CASE(4)
    default: return hipErrorInvalidValue;
  }
#undef BKMOO_RES_CASE
}

}  // namespace bkmoo
