/*
 * Seed-Q CPU oracle (test infrastructure, fp64).
 *
 * Only the test-suite, the package smoke check and the benchmark's CPU-baseline
 * leg load this library. It shares no code with the HIP path.
 *
 * It computes, plainly and slowly, what the block codec of Seed-Q (section 3.1,
 * eq. (codec) and eq. (rate)) defines:
 *   - U(s): the basis from a full-period K-bit LFSR whose initial state is the seed s
 *     (section 3.1; the appendix on the hardware says the states are centred and
 *     the feedback taps depend on the width). Reading: Galois right-shift LFSR
 *     x <- (x >> 1) ^ (x & 1 ? mask_K : 0); basis column j holds the states
 *     x_{8j}, ..., x_{8j+7}, each centred as x - 2^(K-1), scaled by 2^-(K-1).
 *   - t*: the least-squares coefficients of the block on U(s). The pseudo-inverse
 *     per seed is an input here (computed by LAPACK in the Python half).
 *   - the quantiser: P signed 4-bit mantissas under one shared 4-bit exponent,
 *     t_hat = q * 2^-e, e in [0, 15] the finest exponent at which every
 *     round-half-even mantissa fits [-8, 7] (e = 0 with clamping if none fits).
 *   - the quantised error ||w - U(s) t_hat||^2, evaluated exactly: the integer
 *     reconstruction acc_i = sum_j U_int[i][j] q_j is exact, w_hat_i =
 *     acc_i * 2^-(K-1+e) is exact in fp64, and the sum of squares is taken in
 *     fp64 in index order without fused multiply-add.
 *   - the search: the seed in [1, 2^K - 1] with the smallest quantised error,
 *     ties to the smallest seed (section 3.1: all 2^S - 1 seeds are searched).
 *
 * Compiled with -ffp-contract=off so that every product is rounded on its own.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define OQ_C 8

/* Feedback masks of maximal-length Galois LFSRs, one per width K in [8, 24].
 * Each mask has bit K-1 set; maximal length (period 2^K - 1) is checked by
 * oq_period in the test-suite. */
static uint32_t oq_mask(int K) {
  switch (K) {
    case 8: return 0xB8u;
    case 9: return 0x110u;
    case 10: return 0x240u;
    case 11: return 0x500u;
    case 12: return 0x829u;
    case 13: return 0x100Du;
    case 14: return 0x2015u;
    case 15: return 0x6000u;
    case 16: return 0xD008u;
    case 17: return 0x12000u;
    case 18: return 0x20400u;
    case 19: return 0x40023u;
    case 20: return 0x90000u;
    case 21: return 0x140000u;
    case 22: return 0x300000u;
    case 23: return 0x420000u;
    case 24: return 0xE10000u;
    default: return 0u;
  }
}

static uint32_t oq_step(uint32_t x, uint32_t mask) {
  if (x & 1u) return (x >> 1) ^ mask;
  return x >> 1;
}

uint32_t oq_lfsr_mask(int K) { return oq_mask(K); }

/* Number of steps until the state started at 1 returns to 1 (0 if K is
 * unsupported or the state never returns within 2^K steps). */
uint64_t oq_period(int K) {
  uint32_t mask = oq_mask(K);
  if (!mask) return 0;
  uint32_t x = 1u;
  uint64_t n = 0, cap = (uint64_t)1 << K;
  do {
    x = oq_step(x, mask);
    n++;
  } while (x != 1u && n <= cap);
  return x == 1u ? n : 0;
}

/* Centred states u_n = x_n - 2^(K-1), n = 0..n_states-1, x_0 = seed. */
int oq_states(int K, uint32_t seed, int n_states, int32_t* out) {
  uint32_t mask = oq_mask(K);
  if (!mask || seed == 0 || seed >= (1u << K)) return -1;
  uint32_t x = seed;
  int32_t half = (int32_t)1 << (K - 1);
  for (int n = 0; n < n_states; n++) {
    out[n] = (int32_t)x - half;
    x = oq_step(x, mask);
  }
  return 0;
}

/* Shared-exponent quantiser, by its definition: the largest e in [0, 15] such
 * that every t_j * 2^e rounds (half to even) into [-8, 7]; e = 0 when none does. */
void oq_quantize(const double* t, int P, int32_t* e_out, int32_t* q) {
  int e;
  for (e = 15; e >= 0; e--) {
    int fits = 1;
    for (int j = 0; j < P; j++) {
      double r = nearbyint(ldexp(t[j], e));
      if (r > 7.0 || r < -8.0) fits = 0;
    }
    if (fits) break;
  }
  if (e < 0) e = 0;
  for (int j = 0; j < P; j++) {
    double r = nearbyint(ldexp(t[j], e));
    if (r > 7.0) r = 7.0;
    if (r < -8.0) r = -8.0;
    q[j] = (int32_t)r;
  }
  *e_out = e;
}

/* Exact quantised error of the code (e, q) on basis states u (column-major:
 * u[j*8 + i] is row i of column j). */
static double oq_code_error_u(const float* w, const int32_t* u, int K, int P, int e,
                              const int32_t* q) {
  double err = 0.0;
  for (int i = 0; i < OQ_C; i++) {
    int64_t acc = 0;
    for (int j = 0; j < P; j++) acc += (int64_t)u[j * OQ_C + i] * (int64_t)q[j];
    double w_hat = ldexp((double)acc, -(K - 1 + e));
    double d = (double)w[i] - w_hat;
    err = err + d * d;
  }
  return err;
}

/* Exact error of one given code (seed, e, q) on block w. */
int oq_code_error(const float* w, int K, int P, uint32_t seed, int32_t e, const int32_t* q,
                  double* err) {
  int32_t u[OQ_C * 8];
  if (P < 1 || P > 8) return -1;
  if (oq_states(K, seed, OQ_C * P, u)) return -1;
  *err = oq_code_error_u(w, u, K, P, e, q);
  return 0;
}

/* Exhaustive search over every seed for each of nb blocks.
 * blocks: nb x 8 fp32 weights; pinv: (2^K - 1) x P x 8 fp64, pinv[s-1] the
 * Moore-Penrose pseudo-inverse of U(s); outputs per block: seed, e, q[P], err,
 * and the least-squares residual bound of the chosen seed is not reported. */
int oq_search(const float* blocks, int64_t nb, int K, int P, const double* pinv, int nthreads,
              uint32_t* seed_out, int32_t* e_out, int32_t* q_out, double* err_out) {
  uint32_t mask = oq_mask(K);
  if (!mask || P < 1 || P > 8) return -1;
  const int64_t nseeds = ((int64_t)1 << K) - 1;
  const int ns = OQ_C * P;
  int32_t* states = (int32_t*)malloc(sizeof(int32_t) * (size_t)nseeds * (size_t)ns);
  if (!states) return -2;
  for (int64_t s = 1; s <= nseeds; s++) oq_states(K, (uint32_t)s, ns, states + (s - 1) * ns);
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1)
#endif
  for (int64_t b = 0; b < nb; b++) {
    const float* w = blocks + b * OQ_C;
    double best = INFINITY;
    uint32_t best_s = 0;
    int32_t best_e = 0, best_q[8] = {0};
    for (int64_t s = 1; s <= nseeds; s++) {
      const double* A = pinv + (s - 1) * (int64_t)P * OQ_C;
      double t[8];
      for (int j = 0; j < P; j++) {
        double acc = 0.0;
        for (int i = 0; i < OQ_C; i++) acc = acc + A[j * OQ_C + i] * (double)w[i];
        t[j] = acc;
      }
      int32_t e, q[8];
      oq_quantize(t, P, &e, q);
      double err = oq_code_error_u(w, states + (s - 1) * ns, K, P, e, q);
      if (err < best) {
        best = err;
        best_s = (uint32_t)s;
        best_e = e;
        memcpy(best_q, q, sizeof(int32_t) * (size_t)P);
      }
    }
    seed_out[b] = best_s;
    e_out[b] = best_e;
    for (int j = 0; j < P; j++) q_out[b * P + j] = best_q[j];
    err_out[b] = best;
  }
  free(states);
  return 0;
}

/* Decoder reconstruction (section 3.6, Algorithm 2): w_hat = U(s) t_hat for
 * every block. rung_K/rung_P give the rung of each block; q has stride qstride.
 * Writes the exact integers acc (nullable) and w_hat rounded once to fp32. */
int oq_decompress(int64_t nb, const uint32_t* seed, const uint8_t* e, const int8_t* q,
                  int qstride, const int32_t* rung_K, const int32_t* rung_P, float* w_hat,
                  int32_t* acc_out) {
  for (int64_t b = 0; b < nb; b++) {
    int K = rung_K[b], P = rung_P[b];
    int32_t u[OQ_C * 8];
    if (P < 1 || P > 8 || oq_states(K, seed[b], OQ_C * P, u)) return -1;
    for (int i = 0; i < OQ_C; i++) {
      int64_t acc = 0;
      for (int j = 0; j < P; j++) acc += (int64_t)u[j * OQ_C + i] * (int64_t)q[b * qstride + j];
      if (acc_out) acc_out[b * OQ_C + i] = (int32_t)acc;
      w_hat[b * OQ_C + i] = (float)ldexp((double)acc, -(K - 1 + (int)e[b]));
    }
  }
  return 0;
}
