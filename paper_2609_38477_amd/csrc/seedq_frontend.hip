// Data-free importance front end on the GPU (the section on data-free block
// importance, eq. (gamma) and eq. (prop); the output-side rho; the channel sort
// before blocking; the appendix on outlier columns).
//
//   sq_gemv:      out_r = sum_c W_rc^2 v_c        (one wave per row)
//   sq_gemv_t:    out_c = sum_r W_rc^2 v_r        (column tiles x row chunks,
//                 partial sums added in a fixed order)
//   column stats: max_i |W_ij| and the median of |W_ij| over the rows, by a
//                 radix select on the bit patterns of |W| (non-negative floats
//                 order like their bits), three passes of 11, 10 and 10 bits,
//                 per-column histograms in LDS
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

// Column statistics: three passes of a radix select on the 31-bit patterns of
// |W| (non-negative floats order like their bits), digits of 11, 10 and 10
// bits, with per-column histograms in LDS. 8 columns per workgroup (64 KB of
// histograms, two workgroups per CU), 32 row groups of threads per column.
constexpr int kStatCols = 8;
constexpr int kStatGroups = kThreads / kStatCols;   // 32 threads per column
constexpr int kStatBins = 2048;                     // the first digit's bins
constexpr int kStatSuper = 32;                      // workgroups per XCD-aware super-block

// Finds, for every column of the workgroup, the bin of hist[col][0, nbins)
// that holds the element of rank rank[col] (0-based), and the rank inside it:
// each of the 32 threads of a column sums its run of nbins/32 bins, takes the
// prefix of the runs before it, and the thread whose run holds the rank scans
// it. Results in bin_s / rank_s; the caller synchronises.
__device__ void find_rank(const uint32_t (*hist)[kStatBins], int nbins, const int64_t* rank,
                          uint32_t (*part)[kStatGroups], uint32_t* bin_s, int64_t* rank_s) {
  const int col = threadIdx.x % kStatCols, grp = threadIdx.x / kStatCols;
  const int run = nbins / kStatGroups;
  uint32_t sum = 0u;
  for (int b = grp * run; b < (grp + 1) * run; ++b) sum += hist[col][b];
  part[col][grp] = sum;
  __syncthreads();
  int64_t before = 0;
  for (int g = 0; g < grp; ++g) before += part[col][g];
  const int64_t k = rank[col];
  if (k >= before && k < before + int64_t(sum)) {
    int64_t kk = k - before;
    int b = grp * run;
    for (;; ++b) {
      const int64_t n = hist[col][b];
      if (kk < n) break;
      kk -= n;
    }
    bin_s[col] = uint32_t(b);
    rank_s[col] = kk;
  }
}

__global__ void __launch_bounds__(kThreads)
column_stats_kernel(const float* __restrict__ W, int64_t nrows, int64_t ncols,
                    double* __restrict__ maxabs, double* __restrict__ median) {
  __shared__ uint32_t hist[kStatCols][kStatBins];
  __shared__ uint32_t part[kStatCols][kStatGroups];
  __shared__ uint32_t mx_s[kStatCols], above_s[kStatCols], bin_s[kStatCols], next_s[kStatCols];
  __shared__ int64_t rank_s[kStatCols], k_s[kStatCols];
  // XCD-aware column groups: workgroups are dispatched to the 8 XCDs in turn,
  // so of 32 consecutive workgroups those on one XCD take the 4 neighbouring
  // groups of 8 columns that share 128-byte lines of every row.
  const int64_t b = blockIdx.x, b0 = b - b % kStatSuper;
  const int64_t group = b0 + (b % 8) * 4 + (b % kStatSuper) / 8;
  const int64_t c0 = group * kStatCols;
  if (c0 >= ncols) return;   // the grid is rounded up to whole super-blocks
  const int col = threadIdx.x % kStatCols, grp = threadIdx.x / kStatCols;
  const int64_t c = c0 + col;
  const bool live = c < ncols;
  const float* Wc = W + (live ? c : c0);
  const int64_t klo = (nrows - 1) / 2;

  for (int i = threadIdx.x; i < kStatCols * kStatBins; i += kThreads) hist[i / kStatBins][i % kStatBins] = 0u;
  if (threadIdx.x < kStatCols) {
    mx_s[threadIdx.x] = 0u;
    above_s[threadIdx.x] = 0xFFFFFFFFu;
    next_s[threadIdx.x] = 0xFFFFFFFFu;
    k_s[threadIdx.x] = klo;
    bin_s[threadIdx.x] = 0u;     // columns past ncols find no rank: keep bins in range
    rank_s[threadIdx.x] = 0;
  }
  __syncthreads();

  // pass 1: maximum and the histogram of bits 30..20
  if (live) {
    uint32_t m = 0u;
    for (int64_t r = grp; r < nrows; r += kStatGroups) {
      const uint32_t key = __float_as_uint(Wc[r * ncols]) & 0x7FFFFFFFu;
      m = max(m, key);
      atomicAdd(&hist[col][key >> 20], 1u);
    }
    atomicMax(&mx_s[col], m);
  }
  __syncthreads();
  find_rank(hist, kStatBins, k_s, part, bin_s, rank_s);
  __syncthreads();
  const uint32_t d1 = bin_s[col] & (kStatBins - 1u);
  if (threadIdx.x < kStatCols) k_s[threadIdx.x] = rank_s[threadIdx.x];
  for (int i = threadIdx.x; i < kStatCols * kStatBins; i += kThreads) hist[i / kStatBins][i % kStatBins] = 0u;
  __syncthreads();

  // pass 2: bits 19..10 of the keys in the median's first-digit bin
  if (live) {
    for (int64_t r = grp; r < nrows; r += kStatGroups) {
      const uint32_t key = __float_as_uint(Wc[r * ncols]) & 0x7FFFFFFFu;
      if ((key >> 20) == d1) atomicAdd(&hist[col][(key >> 10) & 1023u], 1u);
    }
  }
  __syncthreads();
  find_rank(hist, 1024, k_s, part, bin_s, rank_s);
  __syncthreads();
  const uint32_t pre = (d1 << 10) | (bin_s[col] & 1023u);   // bits 30..10 of the median
  if (threadIdx.x < kStatCols) k_s[threadIdx.x] = rank_s[threadIdx.x];
  for (int i = threadIdx.x; i < kStatCols * 1024; i += kThreads) hist[i / 1024][i % 1024] = 0u;
  __syncthreads();

  // pass 3: bits 9..0 of the keys with that prefix, and the smallest key
  // above the prefix (the upper middle value when the lower one is the
  // largest key with it)
  if (live) {
    uint32_t above = 0xFFFFFFFFu;
    for (int64_t r = grp; r < nrows; r += kStatGroups) {
      const uint32_t key = __float_as_uint(Wc[r * ncols]) & 0x7FFFFFFFu;
      if ((key >> 10) == pre) atomicAdd(&hist[col][key & 1023u], 1u);
      else if ((key >> 10) > pre) above = min(above, key);
    }
    atomicMin(&above_s[col], above);
  }
  __syncthreads();
  find_rank(hist, 1024, k_s, part, bin_s, rank_s);
  __syncthreads();
  const uint32_t d3 = bin_s[col] & 1023u;
  const uint32_t lo = (pre << 10) | d3;
  // the upper middle value of an even count: lo again if its bin holds the
  // next rank too, else the next non-empty bin above it, else the smallest
  // key above the prefix
  const bool same = rank_s[col] + 1 < int64_t(hist[col][d3]);
  {
    const int run = 1024 / kStatGroups;
    uint32_t nb = 0xFFFFFFFFu;
    for (int bb = grp * run; bb < (grp + 1) * run; ++bb)
      if (uint32_t(bb) > d3 && hist[col][bb] != 0u) { nb = uint32_t(bb); break; }
    if (nb != 0xFFFFFFFFu) atomicMin(&next_s[col], nb);
  }
  __syncthreads();
  if (grp == 0 && live) {
    uint32_t hi = lo;
    if (nrows % 2 == 0 && !same)
      hi = next_s[col] != 0xFFFFFFFFu ? ((pre << 10) | next_s[col]) : above_s[col];
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

// out[r][j] = in[r][perm[j]] (gather) or out[r][perm[j]] = in[r][j] (scatter).
// Rows of up to kPermLdsCols columns go through LDS: a workgroup reads a whole
// row with coalesced loads into LDS (in place for the gather, at perm[j] for
// the scatter), then writes the whole output row with coalesced stores (from
// perm[j] for the gather, in place for the scatter), so both HBM sides stream.
// For the scatter a bit per column marks the positions some valid entry
// targets; the others are left unwritten, as in the direct form. Wider rows
// take the direct form: one thread per element, grid-stride.
constexpr int64_t kPermLdsCols = 16384;   // 64 KB of row plus 2 KB of marks

__global__ void __launch_bounds__(kThreads)
permute_rows_lds_kernel(const float* __restrict__ in, int64_t nrows, int64_t ncols,
                        const int32_t* __restrict__ perm, int inverse, float* __restrict__ out) {
  extern __shared__ uint32_t perm_lds[];
  float* row = reinterpret_cast<float*>(perm_lds);
  uint32_t* mark = perm_lds + ncols;   // (ncols + 31) / 32 words, scatter only
  const int n = int(ncols);
  if (inverse) {
    for (int w = threadIdx.x; w < (n + 31) / 32; w += kThreads) mark[w] = 0u;
    __syncthreads();
    for (int j = threadIdx.x; j < n; j += kThreads) {
      const int32_t p = perm[j];
      if (p >= 0 && p < n) atomicOr(&mark[p / 32], 1u << (p % 32));
    }
  }
  for (int64_t r = blockIdx.x; r < nrows; r += gridDim.x) {
    __syncthreads();   // the previous row's reads of the buffer are done
    const float* src = in + r * ncols;
    float* dst = out + r * ncols;
    for (int j = threadIdx.x; j < n; j += kThreads) {
      if (!inverse) {
        row[j] = src[j];
      } else {
        const int32_t p = perm[j];
        if (p >= 0 && p < n) row[p] = src[j];
      }
    }
    __syncthreads();
    for (int j = threadIdx.x; j < n; j += kThreads) {
      if (!inverse) {
        const int32_t p = perm[j];
        dst[j] = (p >= 0 && p < n) ? row[p] : __int_as_float(0x7fc00000);
      } else if ((mark[j / 32] >> (j % 32)) & 1u) {
        dst[j] = row[j];
      }
    }
  }
}

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
  const int64_t groups = (ncols + kStatCols - 1) / kStatCols;
  const unsigned grid = unsigned((groups + kStatSuper - 1) / kStatSuper * kStatSuper);
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
  if (ncols <= kPermLdsCols) {
    const size_t lds = size_t(ncols) * 4 + size_t((ncols + 31) / 32) * 4;
    // more than 64 KB of dynamic LDS must be allowed for the kernel (set on
    // every call: the attribute belongs to the current device)
    const hipError_t attr = hipFuncSetAttribute(
        reinterpret_cast<const void*>(permute_rows_lds_kernel),
        hipFuncAttributeMaxDynamicSharedMemorySize, int(kPermLdsCols * 4 + kPermLdsCols / 8));
    if (attr != hipSuccess) return attr;
    const int64_t blocks = std::min<int64_t>(nrows, 8192);
    hipLaunchKernelGGL(permute_rows_lds_kernel, dim3(unsigned(blocks)), dim3(kThreads), lds, stream,
                       d_in, nrows, ncols, d_perm, inverse, d_out);
    return hipGetLastError();
  }
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
