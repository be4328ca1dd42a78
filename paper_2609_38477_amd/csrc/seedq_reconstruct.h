// Exact reconstruction of one block from its code (section 3.1 eq. (codec),
// Algorithm 2): regenerate the 8P LFSR states of seed s, form the integer
// products acc_i = sum_j U_int[i][j] q_j (|acc| < 2^29) and scale by
// 2^-(K-1+e) after one rounding to fp32. Shared by the decoders.
#pragma once

#include "seedq_internal.h"

namespace seedq {

// Rung constants for per-lane lookups, kept in LDS: entry r = (K, P, LFSR
// feedback mask, code length l = K + 4 + 4P) of rung r < n, and entry n (n =
// rt.n <= SEEDQ_MAX_RUNGS) stands for every rung byte >= n: an invalid code of
// length 0 (K = SEEDQ_MIN_K, P = 1 keep its arithmetic in range). Threads
// 0..SEEDQ_MAX_RUNGS fill it; the caller synchronises before reading.
constexpr int kRungTable = SEEDQ_MAX_RUNGS + 1;

__device__ __forceinline__ void fill_rung_table(uint4* tab, const RungTable& rt) {
  if (threadIdx.x < kRungTable) {
    const int t = int(threadIdx.x);
    const bool v = t < rt.n;
    const int K = v ? rt.K[t] : SEEDQ_MIN_K;
    const int P = v ? rt.P[t] : 1;
    tab[t] = make_uint4(uint32_t(K), uint32_t(P), lfsr_mask(K), v ? uint32_t(K + 4 + 4 * P) : 0u);
  }
}

__device__ __forceinline__ uint32_t table_index(uint32_t r, uint32_t n) { return r < n ? r : n; }

// acc_i = sum_j (x_{8j+i} - 2^(K-1)) q_j, with q_j = qat(j) in [-8, 7], P >= 1
// and the LFSR feedback mask of K. It is formed as sum_j x q_j - 2^(K-1)
// sum_j q_j: for K <= 23 every state fits a signed 24-bit operand, so each
// product is one full-rate 24-bit multiply-add (|x q| < 2^26, every partial
// sum < 2^29). The first coefficient is peeled so that acc needs no clearing.
template <typename QAt>
__device__ __forceinline__ void block_acc_q(uint32_t s, int K, int P, uint32_t mask, QAt qat,
                                            int32_t (&acc)[kC]) {
  const int32_t half = int32_t(1) << (K - 1);
  uint32_t x = s;
  if (__builtin_expect(K <= 23, 1)) {
    const int32_t q0 = qat(0);
    int32_t qsum = q0;
#pragma unroll
    for (int i = 0; i < kC; ++i) {
      acc[i] = __mul24(int32_t(x), q0);
      x = lfsr_step(x, mask);
    }
    for (int j = 1; j < P; ++j) {
      const int32_t qj = qat(j);
      qsum += qj;
#pragma unroll
      for (int i = 0; i < kC; ++i) {
        acc[i] += __mul24(int32_t(x), qj);
        x = lfsr_step(x, mask);
      }
    }
    const int32_t c = half * qsum;
#pragma unroll
    for (int i = 0; i < kC; ++i) acc[i] -= c;
  } else {
    const int32_t q0 = qat(0);
#pragma unroll
    for (int i = 0; i < kC; ++i) {
      acc[i] = __mul24(int32_t(x) - half, q0);   // x - 2^23 fits 24 bits
      x = lfsr_step(x, mask);
    }
    for (int j = 1; j < P; ++j) {
      const int32_t qj = qat(j);
#pragma unroll
      for (int i = 0; i < kC; ++i) {
        acc[i] += __mul24(int32_t(x) - half, qj);
        x = lfsr_step(x, mask);
      }
    }
  }
}

// q_j is the signed byte j of qw (bytes 0-3 in qw.x, 4-7 in qw.y).
__device__ __forceinline__ void block_acc(uint32_t s, int K, int P, uint2 qw, int32_t (&acc)[kC]) {
  block_acc_q(s, K, P, lfsr_mask(K), [&](int j) {
    const uint32_t word = (j < 4) ? qw.x : qw.y;
    return int32_t(int8_t(uint8_t(word >> (8 * (j & 3)))));
  }, acc);
}

// w_hat_i = acc_i 2^-(K-1+e), NaN for an invalid code.
__device__ __forceinline__ void block_weights(const int32_t (&acc)[kC], int K, int e, bool ok,
                                              float (&o)[kC]) {
  const int sh = -(K - 1 + e);
#pragma unroll
  for (int i = 0; i < kC; ++i)
    o[i] = ok ? ldexpf(__int2float_rn(acc[i]), sh) : __int_as_float(0x7fc00000);
}

}  // namespace seedq
