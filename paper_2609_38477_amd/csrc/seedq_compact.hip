// Split of the blocks by rung for the search: for every rung r the list of its
// block indices in increasing order, all lists back to back. Three passes
// (count per chunk, exclusive scan, ordered scatter), so the result does not
// depend on scheduling. Blocks whose rung index is out of range are left out
// of every list and get seed 0.
//
// Workspace layout (bytes, 256-aligned sections):
//   lists   int32 [nblocks]
//   counts  int32 [nchunks][nrungs]   blocks of rung r in chunk c
//   coff    int32 [nchunks][nrungs]   list position of chunk c's first block of rung r
//   off     int32 [nrungs + 1]        start of every rung's list, off[nrungs] = total
#include "seedq_internal.h"

namespace seedq {
namespace {

constexpr int kThreads = 256;
constexpr int kPerThread = 8;
constexpr int kChunk = kThreads * kPerThread;

struct WsLayout {
  int64_t nchunks;
  size_t lists, counts, coff, off, total;
};

WsLayout ws_layout(int64_t nblocks, int nrungs) {
  WsLayout L;
  L.nchunks = (nblocks + kChunk - 1) / kChunk;
  L.lists = 0;
  L.counts = align256(L.lists + sizeof(int32_t) * size_t(nblocks));
  L.coff = align256(L.counts + sizeof(int32_t) * size_t(L.nchunks) * nrungs);
  L.off = align256(L.coff + sizeof(int32_t) * size_t(L.nchunks) * nrungs);
  L.total = align256(L.off + sizeof(int32_t) * size_t(nrungs + 1));
  return L;
}

__global__ void __launch_bounds__(kThreads)
count_kernel(const uint8_t* __restrict__ rung, int64_t nblocks, int nrungs,
             int32_t* __restrict__ counts, uint32_t* __restrict__ seed_invalid) {
  __shared__ int32_t c[SEEDQ_MAX_RUNGS];
  if (threadIdx.x < SEEDQ_MAX_RUNGS) c[threadIdx.x] = 0;
  __syncthreads();
  const int64_t base = int64_t(blockIdx.x) * kChunk;
  for (int it = 0; it < kPerThread; ++it) {
    const int64_t b = base + it * kThreads + threadIdx.x;
    if (b < nblocks) {
      const int r = rung[b];
      if (r < nrungs) atomicAdd(&c[r], 1);
      else seed_invalid[b] = 0u;
    }
  }
  __syncthreads();
  if (threadIdx.x < nrungs) counts[blockIdx.x * int64_t(nrungs) + threadIdx.x] = c[threadIdx.x];
}

// One workgroup: exclusive scan over chunks for every rung, then rung offsets.
__global__ void __launch_bounds__(kThreads)
scan_kernel(const int32_t* __restrict__ counts, int64_t nchunks, int nrungs,
            int32_t* __restrict__ coff, int32_t* __restrict__ off) {
  __shared__ int32_t part[kThreads];
  __shared__ int32_t rung_total[SEEDQ_MAX_RUNGS];
  const int64_t per = (nchunks + kThreads - 1) / kThreads;
  const int64_t c0 = threadIdx.x * per;
  const int64_t c1 = min(nchunks, c0 + per);
  for (int r = 0; r < nrungs; ++r) {
    int32_t s = 0;
    for (int64_t c = c0; c < c1; ++c) s += counts[c * nrungs + r];
    part[threadIdx.x] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
      int32_t run = 0;
      for (int t = 0; t < kThreads; ++t) {
        const int32_t v = part[t];
        part[t] = run;
        run += v;
      }
      rung_total[r] = run;
    }
    __syncthreads();
    int32_t run = part[threadIdx.x];
    for (int64_t c = c0; c < c1; ++c) {
      coff[c * nrungs + r] = run;
      run += counts[c * nrungs + r];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    int32_t run = 0;
    for (int r = 0; r < nrungs; ++r) {
      off[r] = run;
      run += rung_total[r];
    }
    off[nrungs] = run;
  }
}

__global__ void __launch_bounds__(kThreads)
scatter_kernel(const uint8_t* __restrict__ rung, int64_t nblocks, int nrungs,
               const int32_t* __restrict__ coff, const int32_t* __restrict__ off,
               int32_t* __restrict__ lists) {
  __shared__ int32_t wave_cnt[kThreads / 64];
  __shared__ int32_t running[SEEDQ_MAX_RUNGS];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  if (threadIdx.x < nrungs)
    running[threadIdx.x] = off[threadIdx.x] + coff[blockIdx.x * int64_t(nrungs) + threadIdx.x];
  __syncthreads();
  const int64_t base = int64_t(blockIdx.x) * kChunk;
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int it = 0; it < kPerThread; ++it) {
    const int64_t b = base + it * kThreads + threadIdx.x;
    const int r_b = (b < nblocks) ? int(rung[b]) : 255;
    for (int r = 0; r < nrungs; ++r) {
      const bool mine = (r_b == r);
      const uint64_t m = __ballot(mine);
      if (lane == 0) wave_cnt[wave] = __popcll(m);
      __syncthreads();
      int32_t before = running[r];
      for (int v = 0; v < wave; ++v) before += wave_cnt[v];
      if (mine) lists[before + __popcll(m & lt)] = int32_t(b);
      __syncthreads();
      if (threadIdx.x == 0) {
        int32_t tot = 0;
        for (int v = 0; v < kThreads / 64; ++v) tot += wave_cnt[v];
        running[r] += tot;
      }
      __syncthreads();
    }
  }
}

}  // namespace

size_t compaction_workspace_bytes(int64_t nblocks, int nrungs) {
  return ws_layout(nblocks, nrungs).total;
}

const int32_t* compaction_list(void* d_ws, int64_t nblocks, int nrungs) {
  return reinterpret_cast<const int32_t*>(static_cast<char*>(d_ws) + ws_layout(nblocks, nrungs).lists);
}

const int32_t* compaction_offsets(void* d_ws, int64_t nblocks, int nrungs) {
  return reinterpret_cast<const int32_t*>(static_cast<char*>(d_ws) + ws_layout(nblocks, nrungs).off);
}

hipError_t launch_compaction(const uint8_t* d_rung, int64_t nblocks, int nrungs, void* d_ws,
                             uint32_t* d_seed_invalid, hipStream_t stream) {
  const WsLayout L = ws_layout(nblocks, nrungs);
  char* ws = static_cast<char*>(d_ws);
  int32_t* lists = reinterpret_cast<int32_t*>(ws + L.lists);
  int32_t* counts = reinterpret_cast<int32_t*>(ws + L.counts);
  int32_t* coff = reinterpret_cast<int32_t*>(ws + L.coff);
  int32_t* off = reinterpret_cast<int32_t*>(ws + L.off);
  if (L.nchunks == 0) {
    hipLaunchKernelGGL(scan_kernel, dim3(1), dim3(kThreads), 0, stream, counts, int64_t(0), nrungs,
                       coff, off);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(count_kernel, dim3(unsigned(L.nchunks)), dim3(kThreads), 0, stream, d_rung,
                     nblocks, nrungs, counts, d_seed_invalid);
  hipLaunchKernelGGL(scan_kernel, dim3(1), dim3(kThreads), 0, stream, counts, L.nchunks, nrungs,
                     coff, off);
  hipLaunchKernelGGL(scatter_kernel, dim3(unsigned(L.nchunks)), dim3(kThreads), 0, stream, d_rung,
                     nblocks, nrungs, coff, off, lists);
  return hipGetLastError();
}

}  // namespace seedq
