// Pass 1: per-bucket Gram matrices G_b[i][j] = <x_i, x_j> over the bucket.
//
// The bucket-level problems (Eq. shard-mgda, the local CAGrad problem and
// PCGrad's local conflict test, Section 3.2) depend on the local gradients
// only through these inner products, so this pass is the only one that
// needs all K rows at once.  It is HBM-bound: K*N*s bytes read, K(K+1)
// flops per element position, far below the fp32 vector ridge point, so
// it uses plain fp32 FMAs and no matrix cores.
//
// Design (gfx950): persistent workgroups of 4 wavefronts own contiguous
// runs of chunks.  Every thread issues K*R independent 128-bit
// non-temporal loads per iteration and accumulates all K(K+1)/2 products
// in fp32 registers over the chunk's iterations.  Lane sums are combined by
// a fixed xor butterfly across the wavefront, then in fp64 across the 4
// wavefronts through LDS in wave order, and land in a per-chunk slot.  Two
// finalize kernels add a bucket's chunk slots in fp64 in an order fixed by
// the bucket's chunk count (groups of consecutive chunks, then the groups in
// order).  No atomics: the result is bitwise independent of the grid and of
// scheduling.
#include "stream_common.h"

namespace bkmoo {

namespace {

template <int K, int DT>
__global__ __launch_bounds__(kThreads) void gram_partial_kernel(
    Rows<K> rows, const int64_t *__restrict__ offs, const int64_t *__restrict__ cs, int B,
    int shift, int vec, double *__restrict__ partials) {
  constexpr int V = vec_elems(DT);
  constexpr int R = gram_shape(K).R;
  constexpr int U = gram_shape(K).U;
  constexpr int64_t C = gram_chunk_elems(K, DT);
  constexpr int P = pairs(K);
  constexpr int EB = elem_bytes(DT);
  __shared__ double red[kThreads / kWave][P];

  int64_t c, cend;
  my_chunks(cs[B], c, cend);
  if (c >= cend) return;
  int b = find_bucket(cs, B, c);
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;

  for (; c < cend; ++c) {
    while (cs[b + 1] <= c) ++b;
    const int64_t lo = offs[b] + (c - cs[b]) * C;
    const int64_t hi = lo + C < offs[b + 1] ? lo + C : offs[b + 1];

    float acc[P];
#pragma unroll
    for (int p = 0; p < P; ++p) acc[p] = 0.0f;

    if (vec) {
      const Split<V> sp(lo, hi, shift);
      if (tid < sp.nh + sp.nt) {
        const int64_t n = tid < sp.nh ? lo + tid : sp.hi_a + (tid - sp.nh);
        float x[K];
#pragma unroll
        for (int i = 0; i < K; ++i) x[i] = load_elem<DT>(rows.p[i], n);
        accumulate<K>(acc, x);
      }
#pragma unroll 2
      for (int u = 0; u < U; ++u) {
        const int vb = u * kThreads * R + tid;
        u32x4 buf[R][K];
#pragma unroll
        for (int r = 0; r < R; ++r) {
          const int v = vb + r * kThreads;
          if (v < sp.nv) {
#pragma unroll
            for (int i = 0; i < K; ++i)
              buf[r][i] = stream_load(static_cast<const char *>(rows.p[i]) + sp.lo_a * EB, v);
          }
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
          const int v = vb + r * kThreads;
          if (v < sp.nv) {
            float x[K][V];
#pragma unroll
            for (int i = 0; i < K; ++i) decode<DT>(buf[r][i], x[i]);
#pragma unroll
            for (int e = 0; e < V; ++e) {
              float xe[K];
#pragma unroll
              for (int i = 0; i < K; ++i) xe[i] = x[i][e];
              accumulate<K>(acc, xe);
            }
          }
        }
      }
    } else {
      for (int64_t n = lo + tid; n < hi; n += kThreads) {
        float x[K];
#pragma unroll
        for (int i = 0; i < K; ++i) x[i] = load_elem<DT>(rows.p[i], n);
        accumulate<K>(acc, x);
      }
    }

    // fixed-order reduction: xor butterfly across the wavefront (fp32),
    // then the 4 wavefronts in order in fp64
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
    for (int p = tid; p < P; p += kThreads) {
      double s = red[0][p];
#pragma unroll
      for (int w = 1; w < kThreads / kWave; ++w) s += red[w][p];
      partials[c * P + p] = s;
    }
    __syncthreads();
  }
}

// Finalize, level 1: one workgroup per group of up to kFinalizeGroup
// consecutive chunks of one bucket (grid-stride over the groups).  Wavefront
// w handles the pairs p = w, w + 4, ...; lane l adds the group's chunks l,
// l + 64, l + 128, ... in that order in fp64, then a fixed xor butterfly adds
// the 64 lane sums.  The order depends only on the group's chunk count.
__global__ __launch_bounds__(kThreads) void gram_group_kernel(
    int K, int B, const int64_t *__restrict__ cs, const int64_t *__restrict__ gs,
    const double *__restrict__ partials, double *__restrict__ groups) {
  const int P = K * (K + 1) / 2;
  const int64_t total = gs[B];
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  for (int64_t v = blockIdx.x; v < total; v += gridDim.x) {
    const int b = find_bucket(gs, B, v);
    const int64_t c_lo = cs[b] + (v - gs[b]) * kFinalizeGroup;
    const int64_t c_end = c_lo + kFinalizeGroup < cs[b + 1] ? c_lo + kFinalizeGroup : cs[b + 1];
    for (int p = wave; p < P; p += kThreads / kWave) {
      double s = 0.0;
      for (int64_t c = c_lo + lane; c < c_end; c += kWave) s += partials[c * P + p];
#pragma unroll
      for (int off = kWave / 2; off >= 1; off >>= 1) s += __shfl_xor(s, off, kWave);
      if (lane == 0) groups[v * P + p] = s;
    }
  }
}

// Finalize, level 2: one wavefront per bucket adds the bucket's group sums in
// group order and writes the symmetric K x K matrix (NaN everywhere when the
// offsets were rejected by the schedule).
__global__ __launch_bounds__(kWave) void gram_finalize_kernel(
    int K, const int64_t *__restrict__ gs, const double *__restrict__ groups,
    const uint32_t *__restrict__ err, double *__restrict__ gram) {
  const int b = blockIdx.x;
  const int P = K * (K + 1) / 2;
  const bool bad = (*err & kErrOffsets) != 0u;
  const int64_t g0 = gs[b], g1 = gs[b + 1];
  for (int p = threadIdx.x; p < P; p += kWave) {
    double s = 0.0;
    for (int64_t g = g0; g < g1; ++g) s += groups[g * P + p];
    if (bad) s = __builtin_nan("");
    int i = 0, rem = p;
    while (rem >= K - i) {
      rem -= K - i;
      ++i;
    }
    const int j = i + rem;
    gram[((int64_t)b * K + i) * K + j] = s;
    gram[((int64_t)b * K + j) * K + i] = s;
  }
}

template <int K, int DT>
hipError_t launch_gram_t(const StreamArgs &a, double *partials, hipStream_t s) {
  Rows<K> rows;
  for (int i = 0; i < K; ++i) rows.p[i] = a.rows[i];
  auto kern = gram_partial_kernel<K, DT>;
  const int64_t C = gram_chunk_elems(K, DT);
  const int64_t cap = (a.N + C - 1) / C + a.B;
  static const int occ = occupancy(kern);
  int64_t grid = a.grid > 0 ? a.grid : (int64_t)device_cu_count() * occ;
  if (grid > cap) grid = cap;
  if (grid < 1) grid = 1;
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(kThreads), 0, s, rows, a.offsets,
                     a.chunk_start, a.B, a.shift, a.vec ? 1 : 0, partials);
  return hipGetLastError();
}

template <int DT>
hipError_t dispatch_gram(const StreamArgs &a, double *partials, hipStream_t s) {
  switch (a.K) {
    case 2: return launch_gram_t<2, DT>(a, partials, s);
    case 3: return launch_gram_t<3, DT>(a, partials, s);
    case 4: return launch_gram_t<4, DT>(a, partials, s);
    case 5: return launch_gram_t<5, DT>(a, partials, s);
    case 6: return launch_gram_t<6, DT>(a, partials, s);
    case 7: return launch_gram_t<7, DT>(a, partials, s);
    case 8: return launch_gram_t<8, DT>(a, partials, s);
    case 9: return launch_gram_t<9, DT>(a, partials, s);
    case 10: return launch_gram_t<10, DT>(a, partials, s);
    case 11: return launch_gram_t<11, DT>(a, partials, s);
    case 12: return launch_gram_t<12, DT>(a, partials, s);
    case 13: return launch_gram_t<13, DT>(a, partials, s);
    case 14: return launch_gram_t<14, DT>(a, partials, s);
    case 15: return launch_gram_t<15, DT>(a, partials, s);
    case 16: return launch_gram_t<16, DT>(a, partials, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_gram(const StreamArgs &a, double *partials, double *groups, int64_t cap_groups,
                       double *gram, hipStream_t s) {
  hipError_t e = a.dt == F32 ? dispatch_gram<F32>(a, partials, s) : dispatch_gram<BF16>(a, partials, s);
  if (e != hipSuccess) return e;
  const int64_t limit = (int64_t)device_cu_count() * 8;
  const int64_t ggrid = cap_groups < limit ? cap_groups : limit;
  hipLaunchKernelGGL(gram_group_kernel, dim3((unsigned)(ggrid > 0 ? ggrid : 1)), dim3(kThreads), 0, s,
                     a.K, a.B, a.chunk_start, a.group_start, partials, groups);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(gram_finalize_kernel, dim3((unsigned)a.B), dim3(kWave), 0, s, a.K,
                     a.group_start, groups, a.err, gram);
  return hipGetLastError();
}

}  // namespace bkmoo
