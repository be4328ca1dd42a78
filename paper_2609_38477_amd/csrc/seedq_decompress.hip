// Reconstruction w_hat = U(s) q 2^-e (Algorithm 2; per the appendix on cost the
// decoder regenerates the LFSR states and does k_b multiply-adds for each
// weight).
//
// One thread per block: it regenerates the 8P LFSR states of its seed, forms
// the exact integer reconstruction acc_i = sum_j U_int[i][j] q_j (|acc| < 2^29)
// and scales it by 2^-(K-1+e) after a single rounding to fp32. Reads 14 bytes
// of code per block, writes 32 bytes of weights (+32 of acc); neighbouring
// threads touch neighbouring 32-byte blocks, so every access is coalesced.
#include "seedq_reconstruct.h"

namespace seedq {
namespace {

constexpr int kDecompressThreads = 256;

__global__ void __launch_bounds__(kDecompressThreads)
decompress_kernel(const uint32_t* __restrict__ seed, const uint8_t* __restrict__ expo,
                  const int8_t* __restrict__ q, const uint8_t* __restrict__ rung, RungTable rt,
                  int64_t nblocks, float* __restrict__ W_hat, int32_t* __restrict__ acc_out) {
  // rung constants from LDS keep the per-lane lookup off the memory path, so
  // a block's loads all issue at once
  __shared__ uint4 tab[kRungTable];
  fill_rung_table(tab, rt);
  __syncthreads();
  const int64_t b0 = int64_t(blockIdx.x) * kDecompressThreads;
  const int64_t b = b0 + threadIdx.x;
  const bool live = b < nblocks;
  const uint32_t r = live && rung ? uint32_t(rung[b]) : 0u;
  const uint32_t s = live ? seed[b] : 1u;
  const int e = live ? int(expo[b]) : 0;
  const uint2 qw = live ? reinterpret_cast<const uint2*>(q)[b] : make_uint2(0u, 0u);
  const uint4 in = tab[table_index(r, uint32_t(rt.n))];
  const int K = int(in.x), P = int(in.y);
  const bool ok = in.w != 0u && s >= 1u && s < (1u << K) && e <= 15;
  int32_t acc[kC];
  block_acc_q(s, K, P, in.z, [&](int j) {
    const uint32_t word = (j < 4) ? qw.x : qw.y;
    return int32_t(int8_t(uint8_t(word >> (8 * (j & 3)))));
  }, acc);
  float o[kC];
  block_weights(acc, K, e, ok, o);
  // The workgroup's 256 blocks are 8 KB of contiguous output: staged in LDS,
  // every store instruction of a wave then writes 1 KB without gaps.
  __shared__ float4 stage[2 * kDecompressThreads];
  stage[2 * threadIdx.x] = make_float4(o[0], o[1], o[2], o[3]);
  stage[2 * threadIdx.x + 1] = make_float4(o[4], o[5], o[6], o[7]);
  __syncthreads();
  const int64_t nlive = nblocks - b0 < kDecompressThreads ? nblocks - b0 : kDecompressThreads;
  float4* dst = reinterpret_cast<float4*>(W_hat + b0 * kC);
  for (int i = threadIdx.x; i < 2 * nlive; i += kDecompressThreads) dst[i] = stage[i];
  if (acc_out && live) {
    if (!ok) {
#pragma unroll
      for (int i = 0; i < kC; ++i) acc[i] = 0;
    }
    int4* da = reinterpret_cast<int4*>(acc_out + b * kC);
    da[0] = make_int4(acc[0], acc[1], acc[2], acc[3]);
    da[1] = make_int4(acc[4], acc[5], acc[6], acc[7]);
  }
}

}  // namespace

hipError_t launch_decompress(const uint32_t* d_seed, const uint8_t* d_exp, const int8_t* d_q,
                             const uint8_t* d_rung, const RungTable& rt, int64_t nblocks,
                             float* d_W_hat, int32_t* d_acc, hipStream_t stream) {
  if (nblocks == 0) return hipSuccess;
  const int threads = kDecompressThreads;
  const int64_t blocks = (nblocks + threads - 1) / threads;
  hipLaunchKernelGGL(decompress_kernel, dim3(unsigned(blocks)), dim3(threads), 0, stream, d_seed,
                     d_exp, d_q, d_rung, rt, nblocks, d_W_hat, d_acc);
  return hipGetLastError();
}

}  // namespace seedq
