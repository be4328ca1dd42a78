// The per-block exhaustive seed search (section 3.1: "the encoder searches all
// 2^S - 1 seeds for the smallest quantized error"; the appendix on cost names
// this search, 2^S least-squares fits per block, the encoder's dominant cost).
//
// Every candidate (block, seed) is screened with an exact lower bound on its
// quantised error: the least-squares residual
//     r_LS(s) = ||w||^2 - ||Q_s^T w||^2 <= ||w - U(s) t_hat||^2   for every t_hat,
// with Q_s an orthonormal basis of range(U(s)). A candidate whose bound exceeds
// the block's best error so far cannot win and is skipped; the screen runs in
// fp32 with a margin that covers its rounding, so it never skips a candidate
// that could win. Survivors are evaluated exactly: t* = pinv(U(s)) w in fp64,
// the shared-exponent quantiser, integer reconstruction from regenerated LFSR
// states, and the fp64 sum of squares in index order. Seeds are visited in
// increasing order and only a strictly smaller error replaces the best, so
// ties go to the smallest seed.
#include <cstdlib>
#include <cstring>

#include "seedq_exact.h"
#include "seedq_internal.h"

namespace seedq {

// ------------------------------------------------------------ VALU search kernel

// One thread per block, every thread of a wave walks the seeds in the same
// order, so the basis rows are wave-uniform loads.
template <int P>
__global__ void __launch_bounds__(256)
search_valu_kernel(const float* __restrict__ W, int64_t nblocks, const int32_t* __restrict__ list,
                   const int32_t* __restrict__ off, int rung, int K, uint32_t mask,
                   const double* __restrict__ pinv64, const float* __restrict__ q32,
                   uint32_t* __restrict__ seed_out, uint8_t* __restrict__ exp_out,
                   int8_t* __restrict__ q_out, float* __restrict__ err_out) {
  int64_t begin = 0, count = nblocks;
  if (list) {
    begin = off[rung];
    count = int64_t(off[rung + 1]) - begin;
  }
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (int64_t(blockIdx.x) * blockDim.x >= count) return;  // uniform over the workgroup
  const bool in_range = i < count;
  const int64_t b = in_range ? (list ? int64_t(list[begin + i]) : i) : 0;

  float w[kC];
  {
    const float4* src = reinterpret_cast<const float4*>(W + b * kC);
    const float4 lo = in_range ? src[0] : make_float4(0.f, 0.f, 0.f, 0.f);
    const float4 hi = in_range ? src[1] : make_float4(0.f, 0.f, 0.f, 0.f);
    w[0] = lo.x; w[1] = lo.y; w[2] = lo.z; w[3] = lo.w;
    w[4] = hi.x; w[5] = hi.y; w[6] = hi.z; w[7] = hi.w;
  }
  // Screen in units where max |w_i| lies in [1, 2): a power-of-two scale, exact.
  float amax = 0.f;
#pragma unroll
  for (int k = 0; k < kC; ++k) amax = fmaxf(amax, fabsf(w[k]));
  const bool zero_block = !(amax > 0.f);
  const int ex = zero_block ? 0 : ilogbf(amax);
  float ws[kC];
  float ww = 0.f;
#pragma unroll
  for (int k = 0; k < kC; ++k) {
    ws[k] = ldexpf(w[k], -ex);
    ww = fmaf(ws[k], ws[k], ww);
  }
  const double scale2 = ldexp(1.0, -2 * ex);  // error scale factor of the screen units
  const float ww_lo = ww * (1.0f - 0x1p-16f);

  const bool search = in_range && !zero_block;
  double best = INFINITY;
  uint32_t best_s = 1;
  int best_e = 15;
  int best_q[P];
#pragma unroll
  for (int p = 0; p < P; ++p) best_q[p] = 0;
  float thr = search ? -INFINITY : INFINITY;

  const int64_t nseeds = (int64_t(1) << K) - 1;
  for (int64_t sm1 = 0; sm1 < nseeds; ++sm1) {
    const float* Qs = q32 + sm1 * (P * kC);
    float ss = 0.f;
#pragma unroll
    for (int p = 0; p < P; ++p) {
      float c = 0.f;
#pragma unroll
      for (int k = 0; k < kC; ++k) c = fmaf(Qs[p * kC + k], ws[k], c);
      ss = fmaf(c, c, ss);
    }
    if (ss >= thr) {
      int e, q[P];
      const double err = exact_eval<P>(w, pinv64 + sm1 * (P * kC), uint32_t(sm1 + 1), K, mask, e, q);
      if (err < best) {
        best = err;
        best_s = uint32_t(sm1 + 1);
        best_e = e;
#pragma unroll
        for (int p = 0; p < P; ++p) best_q[p] = q[p];
        // candidates with r_LS > best (plus margin) can no longer win
        const float bu = __double2float_ru(best * scale2) * (1.0f + 0x1p-20f);
        thr = ww_lo - bu;
      }
    }
  }

  if (in_range) {
    seed_out[b] = best_s;
    exp_out[b] = uint8_t(best_e);
    uint32_t lo = 0, hi = 0;
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const uint32_t byte = uint32_t(uint8_t(int8_t(best_q[p])));
      if (p < 4) lo |= byte << (8 * p);
      else hi |= byte << (8 * (p - 4));
    }
    reinterpret_cast<uint2*>(q_out)[b] = make_uint2(lo, hi);
    if (err_out) err_out[b] = zero_block ? 0.f : float(best);
  }
}

template <int P>
hipError_t launch_search_p(const float* d_W, int64_t nblocks, const int32_t* d_list,
                           const int32_t* d_off, int rung, int K, const void* d_bases,
                           uint32_t* d_seed, uint8_t* d_exp, int8_t* d_q, float* d_err,
                           hipStream_t stream) {
  const BasesLayout L = bases_layout(K, P);
  const char* base = static_cast<const char*>(d_bases);
  const int threads = 256;
  const int64_t blocks = (nblocks + threads - 1) / threads;
  if (blocks == 0) return hipSuccess;
  hipLaunchKernelGGL(search_valu_kernel<P>, dim3(unsigned(blocks)), dim3(threads), 0, stream,
                     d_W, nblocks, d_list, d_off, rung, K, lfsr_mask(K),
                     reinterpret_cast<const double*>(base + L.off_pinv64),
                     reinterpret_cast<const float*>(base + L.off_q32), d_seed, d_exp, d_q, d_err);
  return hipGetLastError();
}

hipError_t launch_search_valu(const float* d_W, int64_t nblocks, const int32_t* d_list,
                              const int32_t* d_off, int rung_index, int K, int P,
                              const void* d_bases, uint32_t* d_seed, uint8_t* d_exp, int8_t* d_q,
                              float* d_err, hipStream_t stream) {
  switch (P) {
#define SEEDQ_CASE(PP)                                                                       \
  case PP:                                                                                   \
    return launch_search_p<PP>(d_W, nblocks, d_list, d_off, rung_index, K, d_bases, d_seed, \
                               d_exp, d_q, d_err, stream);
    SEEDQ_CASE(1)
    SEEDQ_CASE(2)
    SEEDQ_CASE(3)
    SEEDQ_CASE(4)
    SEEDQ_CASE(5)
    SEEDQ_CASE(6)
#undef SEEDQ_CASE
    default: return hipErrorInvalidValue;
  }
}

// Engine selection: the matrix-core engine by default; SEEDQ_ENGINE=valu picks
// the one-thread-per-block vector engine (same results, used to cross-check).
static bool use_valu_engine() {
  static const bool v = [] {
    const char* e = std::getenv("SEEDQ_ENGINE");
    return e && std::strcmp(e, "valu") == 0;
  }();
  return v;
}

hipError_t launch_search(const float* d_W, int64_t nblocks, const int32_t* d_list,
                         const int32_t* d_off, int rung_index, int K, int P, const void* d_bases,
                         uint32_t* d_seed, uint8_t* d_exp, int8_t* d_q, float* d_err,
                         hipStream_t stream) {
  if (use_valu_engine())
    return launch_search_valu(d_W, nblocks, d_list, d_off, rung_index, K, P, d_bases, d_seed,
                              d_exp, d_q, d_err, stream);
  return launch_search_mfma(d_W, nblocks, d_list, d_off, rung_index, K, P, d_bases, d_seed, d_exp,
                            d_q, d_err, stream);
}

}  // namespace seedq
