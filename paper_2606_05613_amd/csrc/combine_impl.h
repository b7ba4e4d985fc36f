// Output helpers shared by the combine kernel and the pipelined resolve
// kernel: the weighted sum for each output type and the vector stores.
#pragma once

#include "stream_common.h"

namespace bkmoo {

namespace {

template <int ODT>
__device__ __forceinline__ void store_elem(void *out, int64_t n, float y) {
  if constexpr (ODT == F32) {
    static_cast<float *>(out)[n] = y;
  } else {
    static_cast<__bf16 *>(out)[n] = (__bf16)y;
  }
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  bf16x2 v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

// Store V results (V = 4 or 8) at out + first*s_out, 16-byte or 8-byte wide.
template <int ODT, int V>
__device__ __forceinline__ void store_vec(void *out, int64_t first, const float *y) {
  if constexpr (ODT == F32) {
    u32x4 *p = reinterpret_cast<u32x4 *>(static_cast<float *>(out) + first);
#pragma unroll
    for (int q = 0; q < V / 4; ++q) {
      u32x4 v = {__float_as_uint(y[4 * q]), __float_as_uint(y[4 * q + 1]),
                 __float_as_uint(y[4 * q + 2]), __float_as_uint(y[4 * q + 3])};
      __builtin_nontemporal_store(v, p + q);
    }
  } else if constexpr (V == 8) {
    u32x4 v = {pack_bf16x2(y[0], y[1]), pack_bf16x2(y[2], y[3]), pack_bf16x2(y[4], y[5]),
               pack_bf16x2(y[6], y[7])};
    __builtin_nontemporal_store(v, reinterpret_cast<u32x4 *>(static_cast<__bf16 *>(out) + first));
  } else {
    u32x2 v = {pack_bf16x2(y[0], y[1]), pack_bf16x2(y[2], y[3])};
    __builtin_nontemporal_store(v, reinterpret_cast<u32x2 *>(static_cast<__bf16 *>(out) + first));
  }
}

// fp64 -> fp32 rounding to odd: truncate toward zero and, if anything was
// dropped, set the last significand bit.  NaN stays NaN; values beyond the
// fp32 range become +-FLT_MAX with the odd bit set (which a bf16 RNE then
// sends to infinity, as the exact value would).
__device__ __forceinline__ float f32_round_odd(double d) {
  float f = (float)d;
  const double back = (double)f;
  if (back != d) {
    uint32_t u = __float_as_uint(f);
    if (fabs(back) > fabs(d)) u -= 1u;
    f = __uint_as_float(u | 1u);
  }
  return f;
}

// sum_i w_i x_i for the output type ODT: an fp32 FMA chain for fp32
// outputs; for bf16 outputs an fp64 chain rounded to odd into fp32 (the
// store then rounds to nearest even).
template <int K, int ODT>
__device__ __forceinline__ float wsum(const float *w, const float *x) {
  if constexpr (ODT == F32) {
    float y = w[0] * x[0];
#pragma unroll
    for (int i = 1; i < K; ++i) y = __builtin_fmaf(w[i], x[i], y);
    return y;
  } else {
    double y = (double)w[0] * (double)x[0];
#pragma unroll
    for (int i = 1; i < K; ++i) y = __builtin_fma((double)w[i], (double)x[i], y);
    return f32_round_odd(y);
  }
}

}  // namespace

}  // namespace bkmoo
