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
