// Data-free importance front end on the GPU (the section on data-free block
// importance, eq. (gamma) and eq. (prop); the output-side rho; the channel sort
// before blocking; the appendix on outlier columns).
//
//   sq_gemv:      out_r = sum_c W_rc^2 v_c        (one wave per row)
//   sq_gemv_t:    out_c = sum_r W_rc^2 v_r        (column tiles x row chunks,
//                 partial sums added in a fixed order)
//   column stats: max_i |W_ij| and the median of |W_ij| over the rows, by a
//                 radix select on the bit patterns of |W| (non-negative floats
//                 order like their bits), 8 bits per pass, per-column
//                 histograms in LDS
//   E[silu(g)^2]: Gauss-Hermite quadrature per channel
//   column permutation (gather or scatter) and fp16 column escape.
// All sums are fp64; every result is independent of scheduling.
#include <algorithm>

#include <hip/hip_fp16.h>

#include "seedq_internal.h"

namespace seedq {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d, 64);
  return v;
}

// One wave per row; lanes take 4 consecutive columns at a time. Row r's sum
// goes to out[(r / hd * group + g) * hd + r % hd] for g < group: group = 1,
// hd = nrows is the plain product; group > 1 repeats each block of hd rows
// (one key-value head) for the group query heads that share it, head-major.
__global__ void __launch_bounds__(kThreads)
sq_gemv_kernel(const float* __restrict__ W, int64_t nrows, int64_t ncols,
               const float* __restrict__ v, int64_t hd, int group, double* __restrict__ out) {
  const int64_t r = int64_t(blockIdx.x) * (kThreads / 64) + (threadIdx.x >> 6);
  if (r >= nrows) return;
  const int lane = threadIdx.x & 63;
  const float4* row = reinterpret_cast<const float4*>(W + r * ncols);
  const float4* vv = reinterpret_cast<const float4*>(v);
  double acc = 0.0;
  for (int64_t k = lane; k < ncols / 4; k += 64) {
    const float4 w = row[k], x = vv[k];
    acc += double(w.x) * double(w.x) * double(x.x);
    acc += double(w.y) * double(w.y) * double(x.y);
    acc += double(w.z) * double(w.z) * double(x.z);
    acc += double(w.w) * double(w.w) * double(x.w);
  }
  acc = wave_sum(acc);
  const int64_t head = r / hd, i = r - head * hd;
  if (lane < group) out[(head * group + lane) * hd + i] = acc;
}

// a_j = gamma_j^2 in fp64 (exact: the square of an fp32 value fits in 48 bits).
__global__ void __launch_bounds__(kThreads)
gamma_sq_kernel(const float* __restrict__ g, int64_t n, double* __restrict__ a) {
  const int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  if (i >= n) return;
  const double x = double(g[i]);
  a[i] = x * x;
}

// Importance factors enter the products in single precision (round to nearest).
__global__ void __launch_bounds__(kThreads)
to_f32_kernel(const double* __restrict__ in, int64_t n, float* __restrict__ out) {
  const int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  if (i < n) out[i] = float(in[i]);
}

constexpr int kRowChunk = 256;

// Column tile (256 columns, one per thread) x row chunk (kRowChunk rows).
__global__ void __launch_bounds__(kThreads)
sq_gemv_t_partial_kernel(const float* __restrict__ W, int64_t nrows, int64_t ncols,
                         const float* __restrict__ v, double* __restrict__ part) {
  const int64_t c = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  const int64_t r0 = int64_t(blockIdx.y) * kRowChunk;
  const int64_t r1 = min(nrows, r0 + kRowChunk);
  if (c >= ncols) return;
  double acc = 0.0;
  for (int64_t r = r0; r < r1; ++r) {
    const double w = double(W[r * ncols + c]);
    acc += w * w * double(v[r]);
  }
  part[int64_t(blockIdx.y) * ncols + c] = acc;
}

__global__ void __launch_bounds__(kThreads)
sq_gemv_t_total_kernel(const double* __restrict__ part, int64_t nchunks, int64_t ncols,
                       double* __restrict__ out) {
  const int64_t c = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  if (c >= ncols) return;
  double acc = 0.0;
  for (int64_t k = 0; k < nchunks; ++k) acc += part[k * ncols + c];
  out[c] = acc;
}

constexpr int kStatCols = 32;  // columns per workgroup

// The k-th smallest |W[:, c]| (0-based) for the 32 columns of this workgroup:
// four passes of an 8-bit radix select over the bit patterns, most significant
// byte first. Returns the key for column threadIdx.x (threads < 32).
__device__ uint32_t select_kth(const float* __restrict__ W, int64_t nrows, int64_t ncols,
                               int64_t c0, int64_t k, uint32_t (*hist)[256], uint32_t* prefix_s,
                               uint32_t* mask_s, int64_t* k_s) {
  const int col = threadIdx.x & (kStatCols - 1);
  const int grp = threadIdx.x / kStatCols;          // 8 row groups
  const int64_t c = c0 + col;
  if (threadIdx.x < kStatCols) {
    prefix_s[col] = 0u;
    mask_s[col] = 0u;
    k_s[col] = k;
  }
  __syncthreads();
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int i = threadIdx.x; i < kStatCols * 256; i += kThreads) hist[i / 256][i % 256] = 0u;
    __syncthreads();
    const uint32_t prefix = prefix_s[col], mask = mask_s[col];
    if (c < ncols) {
      for (int64_t r = grp; r < nrows; r += kThreads / kStatCols) {
        const uint32_t key = __float_as_uint(W[r * ncols + c]) & 0x7FFFFFFFu;
        if ((key & mask) == prefix) atomicAdd(&hist[col][(key >> shift) & 255u], 1u);
      }
    }
    __syncthreads();
    if (threadIdx.x < kStatCols) {
      int64_t kk = k_s[col];
      uint32_t b = 0;
      for (; b < 255u; ++b) {
        const int64_t n = hist[col][b];
        if (kk < n) break;
        kk -= n;
      }
      k_s[col] = kk;
      prefix_s[col] |= b << shift;
      mask_s[col] |= 255u << shift;
    }
    __syncthreads();
  }
  return prefix_s[col];
}

__global__ void __launch_bounds__(kThreads)
column_stats_kernel(const float* __restrict__ W, int64_t nrows, int64_t ncols,
                    double* __restrict__ maxabs, double* __restrict__ median) {
  __shared__ uint32_t hist[kStatCols][256];
  __shared__ uint32_t prefix_s[kStatCols], mask_s[kStatCols], mx_s[kStatCols];
  __shared__ int64_t k_s[kStatCols];
  const int64_t c0 = int64_t(blockIdx.x) * kStatCols;
  const int col = threadIdx.x & (kStatCols - 1);
  const int grp = threadIdx.x / kStatCols;
  const int64_t c = c0 + col;
  if (threadIdx.x < kStatCols) mx_s[col] = 0u;
  __syncthreads();
  if (c < ncols) {
    uint32_t m = 0u;
    for (int64_t r = grp; r < nrows; r += kThreads / kStatCols)
      m = max(m, __float_as_uint(W[r * ncols + c]) & 0x7FFFFFFFu);
    atomicMax(&mx_s[col], m);
  }
  __syncthreads();
  const uint32_t lo = select_kth(W, nrows, ncols, c0, (nrows - 1) / 2, hist, prefix_s, mask_s, k_s);
  uint32_t hi = lo;
  if (nrows % 2 == 0)
    hi = select_kth(W, nrows, ncols, c0, nrows / 2, hist, prefix_s, mask_s, k_s);
  if (threadIdx.x < kStatCols && c < ncols) {
    maxabs[c] = double(__uint_as_float(mx_s[col]));
    // the mean of the two middle values for an even count, as a median of an
    // even number of values is usually defined
    median[c] = (double(__uint_as_float(lo)) + double(__uint_as_float(hi))) / 2.0;
  }
}

struct GaussHermite {
  int n;
  double x[128], w[128];
};

// out[i] = E[silu(g)^2], g ~ N(0, var[i]), times scale[i] when scale is given.
__global__ void __launch_bounds__(kThreads)
expect_silu_sq_kernel(const double* __restrict__ var, int64_t n, GaussHermite gh,
                      const double* __restrict__ scale, double* __restrict__ out) {
  const int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  if (i >= n) return;
  const double s = sqrt(2.0 * var[i]);
  double acc = 0.0;
  for (int k = 0; k < gh.n; ++k) {
    const double g = s * gh.x[k];
    const double silu = g / (1.0 + exp(-g));
    acc += gh.w[k] * silu * silu;
  }
  const double e = acc / sqrt(3.14159265358979323846);
  out[i] = scale ? e * scale[i] : e;
}

// out[r][j] = in[r][perm[j]] (gather) or out[r][perm[j]] = in[r][j] (scatter);
// grid-stride over the elements.
__global__ void __launch_bounds__(kThreads)
permute_columns_kernel(const float* __restrict__ in, int64_t nrows, int64_t ncols,
                       const int32_t* __restrict__ perm, int inverse, float* __restrict__ out) {
  const int64_t n = nrows * ncols;
  for (int64_t e = int64_t(blockIdx.x) * kThreads + threadIdx.x; e < n;
       e += int64_t(gridDim.x) * kThreads) {
    const int64_t r = e / ncols, j = e - r * ncols;
    const int64_t p = perm[j];
    if (p < 0 || p >= ncols) {  // not a permutation entry: nothing read or written there
      if (!inverse) out[e] = __int_as_float(0x7fc00000);
      continue;
    }
    if (inverse) out[r * ncols + p] = in[e];
    else out[e] = in[r * ncols + p];
  }
}

// dst[i][r] = fp16(W[r][cols[i]]) (extract) or W[r][cols[i]] = fp32(src[i][r]) (apply).
__global__ void __launch_bounds__(kThreads)
extract_columns_kernel(const float* __restrict__ W, int64_t nrows, int64_t ncols,
                       const int32_t* __restrict__ cols, __half* __restrict__ dst) {
  const int64_t r = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  const int i = blockIdx.y;
  if (r >= nrows) return;
  const int64_t c = cols[i];
  dst[int64_t(i) * nrows + r] =
      (c >= 0 && c < ncols) ? __float2half_rn(W[r * ncols + c]) : __float2half_rn(__int_as_float(0x7fc00000));
}

__global__ void __launch_bounds__(kThreads)
apply_columns_kernel(float* __restrict__ W, int64_t nrows, int64_t ncols,
                     const int32_t* __restrict__ cols, const __half* __restrict__ src) {
  const int64_t r = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  const int i = blockIdx.y;
  if (r >= nrows) return;
  const int64_t c = cols[i];
  if (c >= 0 && c < ncols) W[r * ncols + c] = __half2float(src[int64_t(i) * nrows + r]);
}

}  // namespace

size_t sq_gemv_workspace_bytes(int64_t nrows, int64_t ncols, int transpose) {
  if (!transpose) return 0;
  const int64_t nchunks = (nrows + kRowChunk - 1) / kRowChunk;
  return align256(sizeof(double) * size_t(nchunks) * size_t(ncols));
}

hipError_t launch_sq_gemv(const float* d_W, int64_t nrows, int64_t ncols, const float* d_v,
                          int transpose, double* d_out, void* d_ws, hipStream_t stream) {
  if (!transpose) {
    const unsigned grid = unsigned((nrows + kThreads / 64 - 1) / (kThreads / 64));
    hipLaunchKernelGGL(sq_gemv_kernel, dim3(grid), dim3(kThreads), 0, stream, d_W, nrows, ncols,
                       d_v, nrows, 1, d_out);
    return hipGetLastError();
  }
  const int64_t nchunks = (nrows + kRowChunk - 1) / kRowChunk;
  const unsigned tiles = unsigned((ncols + kThreads - 1) / kThreads);
  double* part = static_cast<double*>(d_ws);
  hipLaunchKernelGGL(sq_gemv_t_partial_kernel, dim3(tiles, unsigned(nchunks)), dim3(kThreads), 0,
                     stream, d_W, nrows, ncols, d_v, part);
  hipLaunchKernelGGL(sq_gemv_t_total_kernel, dim3(tiles), dim3(kThreads), 0, stream, part, nchunks,
                     ncols, d_out);
  return hipGetLastError();
}

hipError_t launch_column_stats(const float* d_W, int64_t nrows, int64_t ncols, double* d_max,
                               double* d_median, hipStream_t stream) {
  const unsigned grid = unsigned((ncols + kStatCols - 1) / kStatCols);
  hipLaunchKernelGGL(column_stats_kernel, dim3(grid), dim3(kThreads), 0, stream, d_W, nrows, ncols,
                     d_max, d_median);
  return hipGetLastError();
}

hipError_t launch_expect_silu_sq(const double* d_var, int64_t n, int nodes, const double* x,
                                 const double* w, const double* d_scale, double* d_out,
                                 hipStream_t stream) {
  GaussHermite gh;
  gh.n = nodes;
  for (int k = 0; k < nodes; ++k) {
    gh.x[k] = x[k];
    gh.w[k] = w[k];
  }
  const unsigned grid = unsigned((n + kThreads - 1) / kThreads);
  hipLaunchKernelGGL(expect_silu_sq_kernel, dim3(grid), dim3(kThreads), 0, stream, d_var, n, gh,
                     d_scale, d_out);
  return hipGetLastError();
}

hipError_t launch_gamma_importance(const float* d_gamma, int64_t n, double* d_a,
                                   hipStream_t stream) {
  const unsigned grid = unsigned((n + kThreads - 1) / kThreads);
  hipLaunchKernelGGL(gamma_sq_kernel, dim3(grid), dim3(kThreads), 0, stream, d_gamma, n, d_a);
  return hipGetLastError();
}

// Workspace of the propagation calls: a_in in fp32 [ncols] and var(g) [nrows].
size_t propagate_workspace_bytes(int64_t nrows, int64_t ncols) {
  return align256(sizeof(float) * size_t(ncols)) + align256(sizeof(double) * size_t(nrows));
}

hipError_t launch_propagate_o(const float* d_Wv, int64_t nrows, int64_t ncols, int n_heads,
                              int n_kv_heads, const double* d_a_in, double* d_a_o, void* d_ws,
                              hipStream_t stream) {
  float* a32 = static_cast<float*>(d_ws);
  hipLaunchKernelGGL(to_f32_kernel, dim3(unsigned((ncols + kThreads - 1) / kThreads)),
                     dim3(kThreads), 0, stream, d_a_in, ncols, a32);
  const unsigned grid = unsigned((nrows + kThreads / 64 - 1) / (kThreads / 64));
  hipLaunchKernelGGL(sq_gemv_kernel, dim3(grid), dim3(kThreads), 0, stream, d_Wv, nrows, ncols,
                     static_cast<const float*>(a32), nrows / n_kv_heads, n_heads / n_kv_heads,
                     d_a_o);
  return hipGetLastError();
}

hipError_t launch_propagate_down(const float* d_Wgate, const float* d_Wup, int64_t nrows,
                                 int64_t ncols, const double* d_a_in, int nodes, const double* x,
                                 const double* w, double* d_a_down, void* d_ws,
                                 hipStream_t stream) {
  float* a32 = static_cast<float*>(d_ws);
  double* var = reinterpret_cast<double*>(static_cast<char*>(d_ws) +
                                          align256(sizeof(float) * size_t(ncols)));
  hipLaunchKernelGGL(to_f32_kernel, dim3(unsigned((ncols + kThreads - 1) / kThreads)),
                     dim3(kThreads), 0, stream, d_a_in, ncols, a32);
  const unsigned grid = unsigned((nrows + kThreads / 64 - 1) / (kThreads / 64));
  hipLaunchKernelGGL(sq_gemv_kernel, dim3(grid), dim3(kThreads), 0, stream, d_Wgate, nrows, ncols,
                     static_cast<const float*>(a32), nrows, 1, var);
  hipLaunchKernelGGL(sq_gemv_kernel, dim3(grid), dim3(kThreads), 0, stream, d_Wup, nrows, ncols,
                     static_cast<const float*>(a32), nrows, 1, d_a_down);
  // a_down = E[silu(g)^2] * up, with up already in d_a_down (read before written, per element)
  return launch_expect_silu_sq(var, nrows, nodes, x, w, d_a_down, d_a_down, stream);
}

hipError_t launch_permute_columns(const float* d_in, int64_t nrows, int64_t ncols,
                                  const int32_t* d_perm, int inverse, float* d_out,
                                  hipStream_t stream) {
  const int64_t blocks = std::min<int64_t>((nrows * ncols + kThreads - 1) / kThreads, 65536);
  hipLaunchKernelGGL(permute_columns_kernel, dim3(unsigned(blocks)), dim3(kThreads), 0, stream, d_in,
                     nrows, ncols, d_perm, inverse, d_out);
  return hipGetLastError();
}

hipError_t launch_columns_fp16(float* d_W, int64_t nrows, int64_t ncols, int32_t ncol,
                               const int32_t* d_cols, void* d_f16, int apply, hipStream_t stream) {
  const dim3 grid(unsigned((nrows + kThreads - 1) / kThreads), unsigned(ncol));
  if (apply)
    hipLaunchKernelGGL(apply_columns_kernel, grid, dim3(kThreads), 0, stream, d_W, nrows, ncols,
                       d_cols, static_cast<const __half*>(d_f16));
  else
    hipLaunchKernelGGL(extract_columns_kernel, grid, dim3(kThreads), 0, stream,
                       static_cast<const float*>(d_W), nrows, ncols, d_cols,
                       static_cast<__half*>(d_f16));
  return hipGetLastError();
}

}  // namespace seedq
