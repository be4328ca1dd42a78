// LFSR basis generation and per-seed pseudo-inverses (section 3.1: the columns
// of U(s) come from a K-bit LFSR of full period whose initial state is the seed
// s; the encoder needs the least-squares fit on U(s) for every seed).
//
// One thread per seed. The 8P centred states are produced by exact integer
// stepping and stored as the seed's integer basis (what the exact evaluation
// reconstructs from); U(s) = U_int(s) 2^-(K-1) is then decomposed in fp64 by a
// one-sided (Hestenes) Jacobi SVD: rotations of column pairs until all columns
// are mutually orthogonal, U V = [sigma_j u_j]. From it:
//   pinv(U) = sum over kept j of v_j u_j^T / sigma_j   (Moore-Penrose),
//   the projector onto range(U) = sum over kept j of u_j u_j^T,
// where a direction is kept when sigma_j > 2^-30 sigma_max. Some seeds of some
// rungs are exactly rank deficient (their LFSR states happen to make the
// integer columns linearly dependent), hence the minimum-norm solution.
// For P >= kComplementMinP the rung's screen also needs 8 - P orthonormal
// vectors orthogonal to range(U): unit vectors e_k orthogonalised against the
// range basis and the vectors already chosen (twice, in fp64), the one with
// the largest remainder taken each time (at least sqrt(remaining dims / 8)).
// For a rank-deficient seed they span only part of the complement, which
// keeps the screen's bound valid (a partial sum of its squares). These rungs
// also get pinv rounded to fp32 (see BasesLayout).
#include "seedq_internal.h"

namespace seedq {
namespace {

template <int P>
__global__ void __launch_bounds__(128)
build_bases_kernel(int K, uint32_t mask, int64_t nseeds, double* __restrict__ pinv64,
                   uint32_t* __restrict__ ub, _Float16* __restrict__ pi16, _Float16* __restrict__ nc16,
                   float* __restrict__ pinv32, int32_t* __restrict__ U_out,
                   float* __restrict__ pinv_out) {
  constexpr int M = complement_dims(P);
  const int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  // fragment address of pair k for this seed (see BasesLayout)
  const int64_t tile = idx / kSeedTile;
  const int m = int(idx % kSeedTile);
  auto pi_at = [&](int k) -> _Float16* {
    const int t = k / 16, kk = k % 16;
    const int lane = m + 32 * (kk / 8);
    return pi16 + tile * (kTileBytes / 2) + t * 512 + lane * 8 + (kk % 8);
  };
  // fragment address of element e of complement vector c (hi or lo half)
  auto nc_at = [&](int c, int lo, int e) -> _Float16* {
    return nc16 + (tile * M + c) * 512 + (m + 32 * lo) * 8 + e;
  };
  if (idx >= nseeds) {
    // padding seeds of the last tile
    if (tile * kSeedTile < nseeds) {
      if constexpr (M == 0)
        for (int k = 0; k < kPairsPadded; ++k) *pi_at(k) = _Float16(0.0f);
      for (int c = 0; c < M; ++c)
        for (int e = 0; e < kC; ++e) *nc_at(c, 0, e) = *nc_at(c, 1, e) = _Float16(0.0f);
    }
    return;
  }
  const uint32_t s = uint32_t(idx + 1);
  const int32_t half = int32_t(1) << (K - 1);
  const double scale = ldexp(1.0, -(K - 1));

  double A[kC][P];
  uint32_t* Ub = ub + idx * basis_words(K, P);
  const bool packed = K <= kPackedMaxK;
  uint32_t x = s;
#pragma unroll
  for (int j = 0; j < P; ++j) {
#pragma unroll
    for (int i = 0; i < kC; ++i) {
      const int32_t u = int32_t(x) - half;
      if (U_out) U_out[idx * (P * kC) + j * kC + i] = u;
      A[i][j] = double(u) * scale;
      if (packed) {   // no table above kPackedMaxK
        if (j % 2 == 0)
          Ub[(j / 2) * kC + i] = uint32_t(uint16_t(int16_t(u)));   // high half below
        else
          Ub[(j / 2) * kC + i] |= uint32_t(uint16_t(int16_t(u))) << 16;
      }
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
  // (P <= 4; P >= 5 screens with the complement vectors below instead)
  {
    double Un[kC][P];
#pragma unroll
    for (int i = 0; i < kC; ++i)
#pragma unroll
      for (int j = 0; j < P; ++j) Un[i][j] = A[i][j] * inv1[j];
    if constexpr (M == 0) {
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

    if constexpr (M > 0) {
      double N[M][kC];
      bool used[kC];
#pragma unroll
      for (int k = 0; k < kC; ++k) used[k] = false;
#pragma unroll
      for (int c = 0; c < M; ++c) {
        // the unit vector with the largest remainder after two projections
        double best[kC], bnorm = -1.0;
        int bk = 0;
        for (int k = 0; k < kC; ++k) {
          if (used[k]) continue;
          double v[kC];
#pragma unroll
          for (int i = 0; i < kC; ++i) v[i] = i == k ? 1.0 : 0.0;
          for (int pass = 0; pass < 2; ++pass) {
#pragma unroll
            for (int j = 0; j < P; ++j) {
              double d = 0.0;
#pragma unroll
              for (int i = 0; i < kC; ++i) d = fma(Un[i][j], v[i], d);
#pragma unroll
              for (int i = 0; i < kC; ++i) v[i] = fma(-d, Un[i][j], v[i]);
            }
            for (int c2 = 0; c2 < c; ++c2) {
              double d = 0.0;
#pragma unroll
              for (int i = 0; i < kC; ++i) d = fma(N[c2][i], v[i], d);
#pragma unroll
              for (int i = 0; i < kC; ++i) v[i] = fma(-d, N[c2][i], v[i]);
            }
          }
          double nn = 0.0;
#pragma unroll
          for (int i = 0; i < kC; ++i) nn = fma(v[i], v[i], nn);
          if (nn > bnorm) {
            bnorm = nn;
            bk = k;
#pragma unroll
            for (int i = 0; i < kC; ++i) best[i] = v[i];
          }
        }
        used[bk] = true;
        const double inv = 1.0 / sqrt(bnorm);
#pragma unroll
        for (int i = 0; i < kC; ++i) N[c][i] = best[i] * inv;
      }
#pragma unroll
      for (int c = 0; c < M; ++c)
#pragma unroll
        for (int e = 0; e < kC; ++e) {
          const double v = N[c][e] * double(kComplementScale);
          const _Float16 hi = _Float16(float(v));
          *nc_at(c, 0, e) = hi;
          *nc_at(c, 1, e) = _Float16(float(v - double(hi)));
        }
    }
  }

  double* P64 = pinv64 + idx * (P * kC);
#pragma unroll
  for (int p = 0; p < P; ++p) {
#pragma unroll
    for (int i = 0; i < kC; ++i) {
      double v = 0.0;
#pragma unroll
      for (int j = 0; j < P; ++j) v = fma(V[p][j] * inv2[j], A[i][j], v);
      P64[p * kC + i] = v;
      if constexpr (M > 0) pinv32[idx * (P * kC) + p * kC + i] = float(v);
      if (pinv_out) pinv_out[(int64_t(p) * nseeds + idx) * kC + i] = float(v);
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
                     reinterpret_cast<uint32_t*>(base + L.off_ub),
                     reinterpret_cast<_Float16*>(base + L.off_pi16),
                     reinterpret_cast<_Float16*>(base + L.off_nc16),
                     reinterpret_cast<float*>(base + L.off_pinv32), d_U, d_pinv);
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
