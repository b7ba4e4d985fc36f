// Device helpers for the two streaming passes (Gram and combine).
#pragma once

#include "internal.h"

namespace bkmoo {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Element n of a row, converted exactly to fp32.
template <int DT>
__device__ __forceinline__ float load_elem(const void *row, int64_t n) {
  if constexpr (DT == F32) {
    return static_cast<const float *>(row)[n];
  } else {
    const uint32_t u = static_cast<const uint16_t *>(row)[n];
    return __uint_as_float(u << 16);
  }
}

// The 4 (fp32) or 8 (bf16) elements of a 16-byte vector, in memory order.
template <int DT>
__device__ __forceinline__ void decode(const u32x4 &v, float *x) {
  if constexpr (DT == F32) {
    x[0] = __uint_as_float(v.x);
    x[1] = __uint_as_float(v.y);
    x[2] = __uint_as_float(v.z);
    x[3] = __uint_as_float(v.w);
  } else {
    // little endian: the lower-addressed bf16 is the low half of each word
    x[0] = __uint_as_float(v.x << 16);
    x[1] = __uint_as_float(v.x & 0xffff0000u);
    x[2] = __uint_as_float(v.y << 16);
    x[3] = __uint_as_float(v.y & 0xffff0000u);
    x[4] = __uint_as_float(v.z << 16);
    x[5] = __uint_as_float(v.z & 0xffff0000u);
    x[6] = __uint_as_float(v.w << 16);
    x[7] = __uint_as_float(v.w & 0xffff0000u);
  }
}

__device__ __forceinline__ u32x4 stream_load(const void *base, int64_t vec_index) {
  return __builtin_nontemporal_load(static_cast<const u32x4 *>(base) + vec_index);
}

// Raw buffer loads: address = descriptor base (scalar) + per-lane byte
// offset + scalar byte offset, range-checked against the descriptor's size
// (loads beyond it return 0).  Keeps address arithmetic out of vector
// registers when a thread touches many vectors.  (Outputs are written with
// 16-byte global stores: a wavefront's lanes then cover 1 KiB contiguously,
// and a buffer store wider than 64 bits with a register scalar offset has a
// data hazard on gfx950 that the compiler does not model.)
typedef __amdgpu_buffer_rsrc_t Rsrc;
constexpr int kRawBufferDword3 = 0x00020000;  // untyped buffer view on gfx9-family parts
constexpr int kNonTemporal = 2;               // cache policy: streaming (nt)

__device__ __forceinline__ Rsrc make_rsrc(const void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes,
                                           kRawBufferDword3);
}
__device__ __forceinline__ u32x4 buf_load16(Rsrc r, uint32_t voff, uint32_t soff) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, kNonTemporal);
}

// acc[p] += x_i x_j for the K(K+1)/2 pairs i <= j (row-major upper
// triangle), fp32 FMAs in pair order.
template <int K>
__device__ __forceinline__ void accumulate(float *acc, const float *x) {
  int p = 0;
#pragma unroll
  for (int i = 0; i < K; ++i)
#pragma unroll
    for (int j = i; j < K; ++j) {
      acc[p] = __builtin_fmaf(x[i], x[j], acc[p]);
      ++p;
    }
}

// Bucket of chunk c: the b with chunk_start[b] <= c < chunk_start[b+1].
// chunk_start is non-decreasing (empty buckets repeat a value).
__device__ __forceinline__ int find_bucket(const int64_t *__restrict__ cs, int B, int64_t c) {
  int lo = 0, hi = B;  // invariant: cs[lo] <= c < cs[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (cs[mid] <= c) lo = mid; else hi = mid;
  }
  return lo;
}

// The contiguous range of chunks workgroup `blockIdx.x` owns.
__device__ __forceinline__ void my_chunks(int64_t total, int64_t &c0, int64_t &c1) {
  const int64_t per = (total + gridDim.x - 1) / gridDim.x;
  c0 = (int64_t)blockIdx.x * per;
  c1 = c0 + per < total ? c0 + per : total;
}

// Split [lo, hi) into a scalar head, a run of whole 16-byte vectors starting
// at an element index congruent to `shift` (mod V), and a scalar tail.
template <int V>
struct Split {
  int64_t lo_a;  // first vector element
  int nv;        // whole vectors
  int nh, nt;    // head and tail element counts (< V each)
  int64_t hi_a;
  __device__ __forceinline__ Split(int64_t lo, int64_t hi, int shift) {
    lo_a = lo + ((shift - lo) & (V - 1));
    if (lo_a > hi) lo_a = hi;
    nv = (int)((hi - lo_a) / V);
    hi_a = lo_a + (int64_t)nv * V;
    nh = (int)(lo_a - lo);
    nt = (int)(hi - hi_a);
  }
};

}  // namespace bkmoo
