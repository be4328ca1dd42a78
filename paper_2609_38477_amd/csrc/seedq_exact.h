// Exact evaluation of one search candidate (block, seed): the search kernels'
// fp64 refinement of the candidates that pass the matrix-core screen.
#pragma once

#include "seedq_internal.h"

namespace seedq {

typedef short seedq_short2 __attribute__((ext_vector_type(2)));

// Quantised error of seed s for block w (fp64, exact reconstruction).
// A:  pinv(U(s)), P x 8 row-major (fp64).
// kTable and K <= kPackedMaxK: read the states from the table Ub, else step
// the LFSR (mask) from s. Ub: the seed's integer basis from the basis stack
// (see BasesLayout), (P+1)/2 x 8 words, word (j, i) = the centred states
// u[2j][i] (low half) and u[2j+1][i] (high half) as int16, u[j][i] =
// x_{8j+i} - 2^(K-1), x_0 = s.
template <int P, bool kTable>
__device__ __forceinline__ double exact_eval(const float (&w)[kC], const double* __restrict__ A,
                                             const uint32_t* __restrict__ Ub, uint32_t s, int K,
                                             uint32_t mask, int& e_out, int (&q)[P]) {
#pragma clang fp contract(off)
  double t[P];
  int e = 15;
#pragma unroll
  for (int p = 0; p < P; ++p) {
    double acc = 0.0;
#pragma unroll
    for (int i = 0; i < kC; ++i) acc = fma(A[p * kC + i], double(w[i]), acc);
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
  // acc_i = sum_j u[j][i] q_j, exact in int32 (|u| < 2^23, |q| <= 8, P <= 6).
  // From the table the basis address is made to depend on e (a zero offset
  // the compiler cannot see through), so that its loads are issued after the
  // coefficient loads are consumed and the two sets of registers are not live
  // at once; the pointer itself keeps its global address space.
  auto after = [](int dep) {
    uint32_t z = 0u;
    asm volatile("" : "+v"(z) : "v"(dep));
    return z;
  };
  int32_t acc[kC];
  if (kTable && K <= kPackedMaxK) {
    // two coefficients per dot2 (v_dot2_i32_i16)
    constexpr int PW = (P + 1) / 2;
    const uint4* src = reinterpret_cast<const uint4*>(Ub) + after(e);
#pragma unroll
    for (int i = 0; i < kC; ++i) acc[i] = 0;
#pragma unroll
    for (int j = 0; j < PW; ++j) {
      const uint32_t qp = uint32_t(uint16_t(int16_t(q[2 * j]))) |
                          (2 * j + 1 < P ? uint32_t(uint16_t(int16_t(q[2 * j + 1]))) << 16 : 0u);
      const seedq_short2 qv = __builtin_bit_cast(seedq_short2, qp);
      const uint4 lo = src[2 * j], hi = src[2 * j + 1];
      const uint32_t u[kC] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
#pragma unroll
      for (int i = 0; i < kC; ++i)
        acc[i] = __builtin_amdgcn_sdot2(__builtin_bit_cast(seedq_short2, u[i]), qv, acc[i], false);
    }
  } else {
    // the states by LFSR steps from the seed (x - 2^(K-1) lies in [-2^23,
    // 2^23) for K <= 24: one 24-bit multiply-add each)
    const int32_t half = int32_t(1) << (K - 1);
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
  }
  // the definition's error: index order, no fused multiply-add
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
