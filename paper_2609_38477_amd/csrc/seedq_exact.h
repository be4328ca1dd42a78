// Exact evaluation of one search candidate (block, seed), shared by the
// search engines.
#pragma once

#include "seedq_internal.h"

namespace seedq {

// Quantised error of seed s for block w (fp64, exact reconstruction).
// A: pinv(U(s)), P x 8 row-major (fp64).
template <int P>
__device__ __forceinline__ double exact_eval(const float (&w)[kC], const double* __restrict__ A,
                                             uint32_t s, int K, uint32_t mask, int& e_out,
                                             int (&q)[P]) {
#pragma clang fp contract(off)
  double t[P];
#pragma unroll
  for (int p = 0; p < P; ++p) {
    double acc = 0.0;
#pragma unroll
    for (int i = 0; i < kC; ++i) acc = acc + A[p * kC + i] * double(w[i]);
    t[p] = acc;
  }
  // largest e in [0, 15] at which every rne(t_p 2^e) lies in [-8, 7]
  int e = 15;
  for (; e >= 0; --e) {
    bool fits = true;
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const double r = rint(ldexp(t[p], e));
      fits = fits && (r <= 7.0) && (r >= -8.0);
    }
    if (fits) break;
  }
  if (e < 0) e = 0;
#pragma unroll
  for (int p = 0; p < P; ++p) {
    const double r = fmin(fmax(rint(ldexp(t[p], e)), -8.0), 7.0);
    q[p] = int(r);
  }
  const int32_t half = int32_t(1) << (K - 1);
  int32_t acc[kC];
#pragma unroll
  for (int i = 0; i < kC; ++i) acc[i] = 0;
  uint32_t x = s;
#pragma unroll
  for (int j = 0; j < P; ++j) {
#pragma unroll
    for (int i = 0; i < kC; ++i) {
      acc[i] += (int32_t(x) - half) * q[j];
      x = lfsr_step(x, mask);
    }
  }
  const int sh = -(K - 1 + e);
  double err = 0.0;
#pragma unroll
  for (int i = 0; i < kC; ++i) {
    const double d = double(w[i]) - ldexp(double(acc[i]), sh);
    err = err + d * d;
  }
  e_out = e;
  return err;
}

// Ordering key of a candidate: the fp64 error with its low 24 mantissa bits
// replaced by the seed. Keys order candidates by error to 2^-28 relative and,
// among errors equal to that resolution, by seed; err >= 0, so the unsigned
// order of the bits is the numeric order.
__device__ __forceinline__ uint64_t candidate_key(double err, uint32_t seed) {
  return (uint64_t(__double_as_longlong(err)) & ~uint64_t(0xFFFFFF)) | uint64_t(seed);
}

__device__ __forceinline__ double key_error(uint64_t key) {
  return __longlong_as_double((long long)(key & ~uint64_t(0xFFFFFF)));
}

}  // namespace seedq
