// Exact evaluation of one search candidate (block, seed): the search kernels'
// fp64 refinement of the candidates that pass the matrix-core screen.
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
  int e = 15;
#pragma unroll
  for (int p = 0; p < P; ++p) {
    double acc = 0.0;
#pragma unroll
    for (int i = 0; i < kC; ++i) acc = acc + A[p * kC + i] * double(w[i]);
    t[p] = acc;
    // The largest e in [0, 15] at which every rne(t_p 2^e) lies in [-8, 7], in
    // closed form, folded into the coefficient loop. A positive t = f 2^E
    // (f in [0.5, 1)) fits while t 2^e < 7.5: up to e = 3 - E when f < 15/16,
    // else 2 - E. A negative one fits while |t| 2^e <= 8.5 (rne(-8.5) = -8):
    // up to e = 4 - E when f <= 17/32, else 3 - E. Fitting is monotone in e, so
    // the answer is the smallest limit and 15; below 0 no scale fits and e = 0
    // with clamping.
    if (acc != 0.0) {
      const double f = __builtin_amdgcn_frexp_mant(acc < 0.0 ? -acc : acc);
      const int E = __builtin_amdgcn_frexp_exp(acc);
      const int lim = acc > 0.0 ? (f < 0.9375 ? 3 - E : 2 - E) : (f <= 0.53125 ? 4 - E : 3 - E);
      e = lim < e ? lim : e;
    }
  }
  if (e < 0) e = 0;
#pragma unroll
  for (int p = 0; p < P; ++p) {
    const double r = fmin(fmax(rint(ldexp(t[p], e)), -8.0), 7.0);
    q[p] = int(r);
  }
  // x - 2^(K-1) lies in [-2^23, 2^23) for K <= 24, so each product is one
  // signed 24-bit multiply-add.
  const int32_t half = int32_t(1) << (K - 1);
  int32_t acc[kC];
#pragma unroll
  for (int i = 0; i < kC; ++i) acc[i] = 0;
  uint32_t x = s;
#pragma unroll
  for (int j = 0; j < P; ++j) {
#pragma unroll
    for (int i = 0; i < kC; ++i) {
      acc[i] += __mul24(int32_t(x) - half, q[j]);
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

}  // namespace seedq
