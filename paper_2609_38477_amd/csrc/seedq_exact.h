// Exact evaluation of one search candidate (block, seed): the search kernels'
// fp64 refinement of the candidates that pass the matrix-core screen.
#pragma once

#include "seedq_internal.h"

namespace seedq {

typedef short seedq_short2 __attribute__((ext_vector_type(2)));

// The exponent e and mantissas q of seed s for block w, decided in fp64:
// t = pinv(U(s)) w with A = pinv(U(s)), P x 8 row-major (fp64), then the
// largest e in [0, 15] at which every rne(t_p 2^e) lies in [-8, 7] (0 when
// none does) and q_p = clamp(rne(t_p 2^e), -8, 7).
template <int P>
__device__ __forceinline__ void decide_f64(const float (&w)[kC], const double* __restrict__ A,
                                           int& e_out, int (&q)[P]) {
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
  e_out = e;
}

// The same decision from the fp32 copy A32 of pinv(U(s)), when it is provably
// the one decide_f64 takes; false when it may not be (then the caller decides
// in fp64). t32_p is an fp32 chain of 8 fused multiply-adds of fp32(A) and w,
// so |t32_p - t64_p| <= (8 + 1 + 8 2^-29) 2^-24 S_p with S_p = sum_i |A_pi w_i|
// (the rounding of A to fp32, the fp32 chain and the fp64 chain of decide_f64)
// plus underflow terms below 2^-140; d_p = 2^-19 S'_p + 2^-120, S'_p the fp32
// sum from fp32(A), covers that and the roundings of t32_p +- d_p. Then every
// t in the box [t32 - d, t32 + d] takes the same exponent and the same
// mantissas (so the fp64 t does): exponent e is kept when it fits for every t
// in the box and e + 1 fits for none (for e = 0 only the latter; for e = 15
// only the former), because fitting is monotone in e; each mantissa when rint
// gives the same integer at both ends of its interval, because rint is
// monotone.
template <int P>
__device__ __forceinline__ bool decide_f32(const float (&w)[kC], const float* __restrict__ A32,
                                           int& e_out, int (&q)[P]) {
  float lo[P], hi[P];
  int e = 15;
#pragma unroll
  for (int p = 0; p < P; ++p) {
    float acc = 0.0f, s = 0.0f;
#pragma unroll
    for (int i = 0; i < kC; ++i) {
      const float a = A32[p * kC + i];
      acc = fmaf(a, w[i], acc);
      s = fmaf(fabsf(a), fabsf(w[i]), s);
    }
    const float d = fmaf(s, 0x1p-19f, 0x1p-120f);
    lo[p] = acc - d;
    hi[p] = acc + d;
    if (acc != 0.0f) {
      const float f = __builtin_amdgcn_frexp_mantf(fabsf(acc));
      const int E = __builtin_amdgcn_frexp_expf(acc);
      const int lim = acc > 0.0f ? (f < 0.9375f ? 3 - E : 2 - E) : (f <= 0.53125f ? 4 - E : 3 - E);
      e = lim < e ? lim : e;
    }
  }
  if (e < 0) e = 0;
  bool fits = true, next_fails = false;
#pragma unroll
  for (int p = 0; p < P; ++p) {
    fits = fits && ldexpf(lo[p], e) >= -8.5f && ldexpf(hi[p], e) < 7.5f;
    next_fails = next_fails || ldexpf(hi[p], e + 1) < -8.5f || ldexpf(lo[p], e + 1) >= 7.5f;
  }
  bool ok = (e == 0 || fits) && (e == 15 || next_fails);
#pragma unroll
  for (int p = 0; p < P; ++p) {
    const float r0 = rintf(ldexpf(lo[p], e)), r1 = rintf(ldexpf(hi[p], e));
    ok = ok && r0 == r1;
    q[p] = int(fminf(fmaxf(r0, -8.0f), 7.0f));
  }
  e_out = e;
  return ok;
}

// Quantised error of seed s for block w at exponent e and mantissas q (fp64,
// exact reconstruction). kTable and K <= kPackedMaxK: read the states from the
// table Ub, else step the LFSR (mask) from s. Ub: the seed's integer basis
// from the basis stack (see BasesLayout), (P+1)/2 x 8 words, word (j, i) =
// the centred states u[2j][i] (low half) and u[2j+1][i] (high half) as int16,
// u[j][i] = x_{8j+i} - 2^(K-1), x_0 = s.
template <int P, bool kTable, bool kLate = true>
__device__ __forceinline__ double quant_error(const float (&w)[kC],
                                              const uint32_t* __restrict__ Ub, uint32_t s, int K,
                                              uint32_t mask, int e, const int (&q)[P]) {
#pragma clang fp contract(off)
  // acc_i = sum_j u[j][i] q_j, exact in int32 (|u| < 2^23, |q| <= 8, P <= 6).
  // With kLate the table address is made to depend on e (a zero offset the
  // compiler cannot see through), so that its loads are issued after the
  // coefficient loads are consumed and the two sets of registers are not live
  // at once; without it they may be issued with the coefficient loads, one
  // memory round trip fewer. The pointer itself keeps its global address
  // space.
  auto after = [](int dep) {
    uint32_t z = 0u;
    asm volatile("" : "+v"(z) : "v"(dep));
    return z;
  };
  int32_t acc[kC];
  if (kTable && K <= kPackedMaxK) {
    // two coefficients per dot2 (v_dot2_i32_i16)
    constexpr int PW = (P + 1) / 2;
    const uint4* src = reinterpret_cast<const uint4*>(Ub) + (kLate ? after(e) : 0u);
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
  return err;
}

// Quantised error of seed s for block w (fp64, exact reconstruction), its
// exponent and mantissas decided in fp64. A: pinv(U(s)), P x 8 row-major.
template <int P, bool kTable>
__device__ __forceinline__ double exact_eval(const float (&w)[kC], const double* __restrict__ A,
                                             const uint32_t* __restrict__ Ub, uint32_t s, int K,
                                             uint32_t mask, int& e_out, int (&q)[P]) {
  decide_f64<P>(w, A, e_out, q);
  return quant_error<P, kTable>(w, Ub, s, K, mask, e_out, q);
}

// The same result, the decision taken from the fp32 copy A32 of pinv(U(s))
// whenever that is provably the fp64 decision (A64 is read only otherwise):
// half the bytes per candidate for the rungs whose evaluations are many.
template <int P>
__device__ __forceinline__ double exact_eval_f32(const float (&w)[kC],
                                                 const float* __restrict__ A32,
                                                 const double* __restrict__ A64,
                                                 const uint32_t* __restrict__ Ub, uint32_t s,
                                                 int K, uint32_t mask, int& e_out, int (&q)[P]) {
  if (!decide_f32<P>(w, A32, e_out, q)) decide_f64<P>(w, A64, e_out, q);
  return quant_error<P, true, false>(w, Ub, s, K, mask, e_out, q);
}

}  // namespace seedq
