// LFSR basis generation and per-seed pseudo-inverses (section 3.1: the columns
// of U(s) come from a K-bit LFSR of full period whose initial state is the seed
// s; the encoder needs the least-squares fit on U(s) for every seed).
//
// One thread per seed. The 8P centred states are produced by exact integer
// stepping; U(s) = U_int(s) 2^-(K-1) is then decomposed in fp64 by a one-sided
// (Hestenes) Jacobi SVD: rotations of column pairs until all columns are
// mutually orthogonal, U V = [sigma_j u_j]. From it:
//   pinv(U) = sum over kept j of v_j u_j^T / sigma_j   (Moore-Penrose),
//   range basis rows u_j^T for kept j (zero rows for dropped directions),
// where a direction is kept when sigma_j > 2^-30 sigma_max. Some seeds of some
// rungs are exactly rank deficient (their LFSR states happen to make the
// integer columns linearly dependent), hence the minimum-norm solution.
#include "seedq_internal.h"

namespace seedq {
namespace {

template <int P>
__global__ void __launch_bounds__(128)
build_bases_kernel(int K, uint32_t mask, int64_t nseeds, double* __restrict__ pinv64,
                   float* __restrict__ q32, _Float16* __restrict__ pi16, int32_t* __restrict__ U_out,
                   float* __restrict__ pinv_out) {
  const int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  // fragment address of pair k for this seed (see BasesLayout)
  const int64_t tile = idx / kSeedTile;
  const int m = int(idx % kSeedTile);
  auto pi_at = [&](int k) -> _Float16* {
    const int t = k / 16, kk = k % 16;
    const int lane = m + 32 * (kk / 8);
    return pi16 + tile * (kTileBytes / 2) + t * 512 + lane * 8 + (kk % 8);
  };
  if (idx >= nseeds) {
    // padding seeds of the last tile
    if (tile * kSeedTile < nseeds)
      for (int k = 0; k < kPairsPadded; ++k) *pi_at(k) = _Float16(0.0f);
    return;
  }
  const uint32_t s = uint32_t(idx + 1);
  const int32_t half = int32_t(1) << (K - 1);
  const double scale = ldexp(1.0, -(K - 1));

  double A[kC][P];
  uint32_t x = s;
#pragma unroll
  for (int j = 0; j < P; ++j) {
#pragma unroll
    for (int i = 0; i < kC; ++i) {
      const int32_t u = int32_t(x) - half;
      if (U_out) U_out[idx * (P * kC) + j * kC + i] = u;
      A[i][j] = double(u) * scale;
      x = lfsr_step(x, mask);
    }
  }

  double V[P][P];
#pragma unroll
  for (int a = 0; a < P; ++a)
#pragma unroll
    for (int b = 0; b < P; ++b) V[a][b] = (a == b) ? 1.0 : 0.0;

  for (int sweep = 0; sweep < 40; ++sweep) {
    bool rotated = false;
#pragma unroll
    for (int p = 0; p < P; ++p) {
#pragma unroll
      for (int q = p + 1; q < P; ++q) {
        double alpha = 0.0, beta = 0.0, gamma = 0.0;
#pragma unroll
        for (int i = 0; i < kC; ++i) {
          alpha = fma(A[i][p], A[i][p], alpha);
          beta = fma(A[i][q], A[i][q], beta);
          gamma = fma(A[i][p], A[i][q], gamma);
        }
        if (gamma == 0.0 || fabs(gamma) <= 1e-15 * sqrt(alpha * beta)) continue;
        rotated = true;
        const double zeta = (beta - alpha) / (2.0 * gamma);
        const double t = copysign(1.0, zeta) / (fabs(zeta) + sqrt(fma(zeta, zeta, 1.0)));
        const double c = 1.0 / sqrt(fma(t, t, 1.0));
        const double sn = c * t;
#pragma unroll
        for (int i = 0; i < kC; ++i) {
          const double ap = A[i][p], aq = A[i][q];
          A[i][p] = c * ap - sn * aq;
          A[i][q] = sn * ap + c * aq;
        }
#pragma unroll
        for (int k = 0; k < P; ++k) {
          const double vp = V[k][p], vq = V[k][q];
          V[k][p] = c * vp - sn * vq;
          V[k][q] = sn * vp + c * vq;
        }
      }
    }
    if (!rotated) break;
  }

  double sig2[P], smax = 0.0;
#pragma unroll
  for (int j = 0; j < P; ++j) {
    double a = 0.0;
#pragma unroll
    for (int i = 0; i < kC; ++i) a = fma(A[i][j], A[i][j], a);
    sig2[j] = a;
    smax = fmax(smax, sqrt(a));
  }
  double inv2[P], inv1[P];
#pragma unroll
  for (int j = 0; j < P; ++j) {
    const double sj = sqrt(sig2[j]);
    const bool keep = smax > 0.0 && sj > ldexp(smax, -30);
    inv2[j] = keep ? 1.0 / sig2[j] : 0.0;
    inv1[j] = keep ? 1.0 / sj : 0.0;
  }

  // projector Pi = sum over kept j of u_j u_j^T, 2^12-scaled fp16 fragments
  {
    double Un[kC][P];
#pragma unroll
    for (int i = 0; i < kC; ++i)
#pragma unroll
      for (int j = 0; j < P; ++j) Un[i][j] = A[i][j] * inv1[j];
#pragma unroll
    for (int i = 0; i < kC; ++i) {
#pragma unroll
      for (int j2 = i; j2 < kC; ++j2) {
        double v = 0.0;
#pragma unroll
        for (int j = 0; j < P; ++j) v = fma(Un[i][j], Un[j2][j], v);
        *pi_at(pair_index(i, j2)) = _Float16(float(v * double(kOperandScale)));
      }
    }
    for (int k = kPairs; k < kPairsPadded; ++k) *pi_at(k) = _Float16(0.0f);
  }

  double* P64 = pinv64 + idx * (P * kC);
  float* Q32 = q32 + idx * (P * kC);
#pragma unroll
  for (int p = 0; p < P; ++p) {
#pragma unroll
    for (int i = 0; i < kC; ++i) {
      double v = 0.0;
#pragma unroll
      for (int j = 0; j < P; ++j) v = fma(V[p][j] * inv2[j], A[i][j], v);
      P64[p * kC + i] = v;
      if (pinv_out) pinv_out[(int64_t(p) * nseeds + idx) * kC + i] = float(v);
      Q32[p * kC + i] = float(A[i][p] * inv1[p]);
    }
  }
}

template <int P>
hipError_t launch_p(int K, int64_t nseeds, void* d_bases, int32_t* d_U, float* d_pinv,
                    hipStream_t stream) {
  const BasesLayout L = bases_layout(K, P);
  char* base = static_cast<char*>(d_bases);
  const int threads = 128;
  const int64_t blocks = (L.ntiles * kSeedTile + threads - 1) / threads;
  hipLaunchKernelGGL(build_bases_kernel<P>, dim3(unsigned(blocks)), dim3(threads), 0, stream, K,
                     lfsr_mask(K), nseeds, reinterpret_cast<double*>(base + L.off_pinv64),
                     reinterpret_cast<float*>(base + L.off_q32),
                     reinterpret_cast<_Float16*>(base + L.off_pi16), d_U, d_pinv);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_build_bases(int K, int P, void* d_bases, int32_t* d_U, float* d_pinv,
                              hipStream_t stream) {
  const int64_t nseeds = (int64_t(1) << K) - 1;
  switch (P) {
    case 1: return launch_p<1>(K, nseeds, d_bases, d_U, d_pinv, stream);
    case 2: return launch_p<2>(K, nseeds, d_bases, d_U, d_pinv, stream);
    case 3: return launch_p<3>(K, nseeds, d_bases, d_U, d_pinv, stream);
    case 4: return launch_p<4>(K, nseeds, d_bases, d_U, d_pinv, stream);
    case 5: return launch_p<5>(K, nseeds, d_bases, d_U, d_pinv, stream);
    case 6: return launch_p<6>(K, nseeds, d_bases, d_U, d_pinv, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace seedq
