// Fault footprint of a corrupted reconstruction against the clean one (the
// security analysis, eq. (security_metrics)): N_flip = the number of weights that
// differ, and the sums behind eta = ||W_corrupt - W_clean||_F / ||W_clean||_F.
// One pass over both matrices (HBM bound); per-workgroup partials, then one
// workgroup adds them in a fixed order, so the result does not depend on
// scheduling.
#include "seedq_internal.h"

namespace seedq {
namespace {

constexpr int kThreads = 256;
constexpr int kPerThread = 16;  // floats per thread per sweep (four float4)
constexpr int64_t kTile = int64_t(kThreads) * kPerThread;

struct Partial {
  long long n;
  double d2, c2;
};

// The difference of two fp32 values is exact in fp64.
__device__ __forceinline__ void add(Partial& p, float c, float x) {
  const double d = double(x) - double(c);
  p.n += (d != 0.0) ? 1 : 0;  // a NaN difference counts as changed
  p.d2 += d * d;
  p.c2 += double(c) * double(c);
}

__device__ Partial wg_sum(Partial p) {
  __shared__ long long sn[kThreads / 64];
  __shared__ double sd[kThreads / 64], sc[kThreads / 64];
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) {
    p.n += __shfl_xor(p.n, d, 64);
    p.d2 += __shfl_xor(p.d2, d, 64);
    p.c2 += __shfl_xor(p.c2, d, 64);
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) {
    sn[wave] = p.n;
    sd[wave] = p.d2;
    sc[wave] = p.c2;
  }
  __syncthreads();
  Partial t{0, 0.0, 0.0};
  for (int w = 0; w < kThreads / 64; ++w) {
    t.n += sn[w];
    t.d2 += sd[w];
    t.c2 += sc[w];
  }
  return t;
}

__global__ void __launch_bounds__(kThreads)
footprint_kernel(const float* __restrict__ clean, const float* __restrict__ corrupt, int64_t n,
                 Partial* __restrict__ part) {
  Partial p{0, 0.0, 0.0};
  const int64_t stride = int64_t(gridDim.x) * kTile;
  for (int64_t base = int64_t(blockIdx.x) * kTile; base < n; base += stride) {
#pragma unroll
    for (int k = 0; k < kPerThread / 4; ++k) {
      const int64_t i = base + (int64_t(k) * kThreads + threadIdx.x) * 4;
      if (i + 4 <= n) {
        const float4 c = *reinterpret_cast<const float4*>(clean + i);
        const float4 x = *reinterpret_cast<const float4*>(corrupt + i);
        add(p, c.x, x.x);
        add(p, c.y, x.y);
        add(p, c.z, x.z);
        add(p, c.w, x.w);
      } else {
        for (int64_t j = i; j < n && j < i + 4; ++j) add(p, clean[j], corrupt[j]);
      }
    }
  }
  const Partial t = wg_sum(p);
  if (threadIdx.x == 0) part[blockIdx.x] = t;
}

__global__ void __launch_bounds__(kThreads)
footprint_total_kernel(const Partial* __restrict__ part, int nparts, long long* __restrict__ count,
                       double* __restrict__ sums) {
  Partial p{0, 0.0, 0.0};
  // thread t adds parts t, t + 256, ... in order; the tree below is fixed
  for (int i = threadIdx.x; i < nparts; i += kThreads) {
    p.n += part[i].n;
    p.d2 += part[i].d2;
    p.c2 += part[i].c2;
  }
  const Partial t = wg_sum(p);
  if (threadIdx.x == 0) {
    *count = t.n;
    sums[0] = t.d2;
    sums[1] = t.c2;
  }
}

constexpr int kParts = 1024;

}  // namespace

size_t footprint_workspace_bytes() { return align256(sizeof(Partial) * kParts); }

hipError_t launch_footprint(const float* d_clean, const float* d_corrupt, int64_t n, void* d_ws,
                            long long* d_count, double* d_sums, hipStream_t stream) {
  Partial* part = static_cast<Partial*>(d_ws);
  const int64_t tiles = (n + kTile - 1) / kTile;
  const int grid = int(tiles < kParts ? (tiles > 0 ? tiles : 1) : kParts);
  hipLaunchKernelGGL(footprint_kernel, dim3(grid), dim3(kThreads), 0, stream, d_clean, d_corrupt, n,
                     part);
  hipLaunchKernelGGL(footprint_total_kernel, dim3(1), dim3(kThreads), 0, stream, part, grid,
                     d_count, d_sums);
  return hipGetLastError();
}

}  // namespace seedq
