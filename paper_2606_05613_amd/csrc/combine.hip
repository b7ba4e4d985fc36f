// Pass 2: the resolved bucket updates d[o_b:o_{b+1}] = sum_i w_{b,i} x_i,
// concatenated over buckets (Algorithm 1: the per-strategy d_(k), then
// d = [d_(1), ..., d_(K)]).
//
// Bandwidth-bound: K*N*s bytes read, N*s_out written, 2K flops per
// element.  Same chunks and 128-bit non-temporal loads as the Gram pass;
// the K weights of a chunk's bucket are wave-uniform scalars.  Unlike the
// Gram pass, chunks are dealt round-robin (chunk c to workgroup c mod grid),
// so the whole grid sweeps the vector together: measured 1-2.5% faster
// than one contiguous run per workgroup on every workload shape here, in
// fast and slow buffer placements alike (the Gram pass gains nothing).
//
// Arithmetic.  For an fp32 output the sum is an fp32 FMA chain in task
// order.  For a bf16 output that is not enough: with bf16 inputs the exact
// sum of w_i x_i often lies within an fp32 rounding error of a bf16 tie
// (e.g. weights of 1/K), and an fp32 chain then rounds the wrong way on a
// few percent of elements.  So the bf16 path accumulates in fp64, where
// every product of an fp32 weight and an fp32/bf16 input is exact, and
// rounds once: fp64 -> fp32 with round-to-odd, then RNE to bf16.  Rounding
// to odd into a format with at least two more significand bits than the
// target makes the second rounding the correct single rounding.
#include "combine_impl.h"

namespace bkmoo {

namespace {

template <int K, int DT, int ODT>
__global__ __launch_bounds__(kThreads) void combine_kernel(
    Rows<K> rows, const int64_t *__restrict__ offs, const int64_t *__restrict__ cs, int B,
    int shift, int vec, const float *__restrict__ weights, void *out) {
  constexpr int V = vec_elems(DT);
  constexpr int R = combine_shape(K).R;
  constexpr int U = combine_shape(K).U;
  constexpr int64_t C = combine_chunk_elems(K, DT);
  constexpr int EB = elem_bytes(DT);

  const int64_t total = cs[B];
  const int tid = threadIdx.x;

  for (int64_t c = blockIdx.x; c < total; c += gridDim.x) {
    const int b = find_bucket(cs, B, c);
    const int64_t lo = offs[b] + (c - cs[b]) * C;
    const int64_t hi = lo + C < offs[b + 1] ? lo + C : offs[b + 1];
    float w[K];
#pragma unroll
    for (int i = 0; i < K; ++i) w[i] = weights[(int64_t)b * K + i];

    if (vec) {
      const Split<V> sp(lo, hi, shift);
      if (tid < sp.nh + sp.nt) {
        const int64_t n = tid < sp.nh ? lo + tid : sp.hi_a + (tid - sp.nh);
        float x[K];
#pragma unroll
        for (int i = 0; i < K; ++i) x[i] = load_elem<DT>(rows.p[i], n);
        store_elem<ODT>(out, n, wsum<K, ODT>(w, x));
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
            float y[V];
#pragma unroll
            for (int e = 0; e < V; ++e) {
              float xe[K];
#pragma unroll
              for (int i = 0; i < K; ++i) xe[i] = x[i][e];
              y[e] = wsum<K, ODT>(w, xe);
            }
            store_vec<ODT, V>(out, sp.lo_a + (int64_t)v * V, y);
          }
        }
      }
    } else {
      for (int64_t n = lo + tid; n < hi; n += kThreads) {
        float x[K];
#pragma unroll
        for (int i = 0; i < K; ++i) x[i] = load_elem<DT>(rows.p[i], n);
        store_elem<ODT>(out, n, wsum<K, ODT>(w, x));
      }
    }
  }
}

template <int K, int DT, int ODT>
hipError_t launch_combine_t(const StreamArgs &a, const float *weights, void *out, hipStream_t s) {
  Rows<K> rows;
  for (int i = 0; i < K; ++i) rows.p[i] = a.rows[i];
  auto kern = combine_kernel<K, DT, ODT>;
  const int64_t C = combine_chunk_elems(K, DT);
  const int64_t cap = (a.N + C - 1) / C + a.B;
  static const int occ = occupancy(kern);
  int64_t grid = a.grid > 0 ? a.grid : (int64_t)device_cu_count() * occ;
  if (grid > cap) grid = cap;
  if (grid < 1) grid = 1;
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(kThreads), 0, s, rows, a.offsets,
                     a.chunk_start, a.B, a.shift, a.vec ? 1 : 0, weights, out);
  return hipGetLastError();
}

template <int DT, int ODT>
hipError_t dispatch_combine(const StreamArgs &a, const float *w, void *out, hipStream_t s) {
  switch (a.K) {
    case 2: return launch_combine_t<2, DT, ODT>(a, w, out, s);
    case 3: return launch_combine_t<3, DT, ODT>(a, w, out, s);
    case 4: return launch_combine_t<4, DT, ODT>(a, w, out, s);
    case 5: return launch_combine_t<5, DT, ODT>(a, w, out, s);
    case 6: return launch_combine_t<6, DT, ODT>(a, w, out, s);
    case 7: return launch_combine_t<7, DT, ODT>(a, w, out, s);
    case 8: return launch_combine_t<8, DT, ODT>(a, w, out, s);
    case 9: return launch_combine_t<9, DT, ODT>(a, w, out, s);
    case 10: return launch_combine_t<10, DT, ODT>(a, w, out, s);
    case 11: return launch_combine_t<11, DT, ODT>(a, w, out, s);
    case 12: return launch_combine_t<12, DT, ODT>(a, w, out, s);
    case 13: return launch_combine_t<13, DT, ODT>(a, w, out, s);
    case 14: return launch_combine_t<14, DT, ODT>(a, w, out, s);
    case 15: return launch_combine_t<15, DT, ODT>(a, w, out, s);
    case 16: return launch_combine_t<16, DT, ODT>(a, w, out, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_combine(const StreamArgs &a, const float *weights, void *out, int out_dt,
                          hipStream_t s) {
  if (a.dt == F32)
    return out_dt == F32 ? dispatch_combine<F32, F32>(a, weights, out, s)
                         : dispatch_combine<F32, BF16>(a, weights, out, s);
  return out_dt == F32 ? dispatch_combine<BF16, F32>(a, weights, out, s)
                       : dispatch_combine<BF16, BF16>(a, weights, out, s);
}

}  // namespace bkmoo
