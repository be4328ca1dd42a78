// The headerless variable-length code stream of one tensor (Algorithm 1, the
// emit step: every block contributes exactly l(g_b) = K + 4P + 4 bits of
// eq. (rate), with no header; Algorithm 2 and the appendix on encoding and
// decoding: a decoder reads a tensor's blocks in order from its start, the
// length of each known from the allocation alone).
//
// Layout: blocks in row-major order; inside a block the seed (K bits), the
// exponent (4 bits) and the mantissas q_0 .. q_{P-1} (4 bits each, two's
// complement), every field least-significant bit first at increasing stream
// bit positions; stream bit n is bit n % 32 of 32-bit word n / 32; the payload
// is padded with zero bits to a whole word.
//
// Every kernel walks the blocks in chunks of 2048 (one workgroup each): a first
// pass sums the lengths of every chunk, one workgroup turns the sums into the
// bit offset of every chunk, and the chunk's workgroup then finds each block's
// offset with one workgroup prefix sum over the rung lengths of all its eight
// 256-block iterations at once (eight 16-bit fields in two 64-bit words), so
// neighbouring threads handle neighbouring blocks, every global access is
// coalesced and a chunk needs two barriers. Rung constants come from a small
// table in LDS. The packer assembles its chunk in LDS and stores whole words;
// only the two words a chunk may share with its neighbours are merged with
// atomic ORs (they are cleared by the offset pass).
#include <algorithm>

#include "seedq_reconstruct.h"

namespace seedq {
namespace {

constexpr int kThreads = 256;
constexpr int kIters = 8;
constexpr int kChunk = kThreads * kIters;  // blocks per workgroup
constexpr int kMaxBlockBits = SEEDQ_MAX_K + 4 + 4 * SEEDQ_MAX_P;
// bit 31 + every bit of a chunk, plus the two words a code may spill into
constexpr int kStageWords = (31 + kChunk * kMaxBlockBits) / 32 + 3;

// Exclusive prefix sums over the workgroup of eight 16-bit fields at once
// (fields 0-3 in v.x, 4-7 in v.y, field k in bits 16(k mod 4) and up). Every
// field's workgroup total stays below 2^16 (kThreads codes of at most
// kMaxBlockBits bits), so the 64-bit sums never carry from one field into the
// next. *total receives the workgroup totals.
static_assert(kThreads * kMaxBlockBits < 65536, "a 16-bit field holds one iteration's bits");
__device__ ulonglong2 wg_exclusive_scan8(ulonglong2 v, ulonglong2* total) {
  __shared__ unsigned long long wsum[2][kThreads / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  unsigned long long a = v.x, b = v.y;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const unsigned long long ya = __shfl_up(a, d, 64), yb = __shfl_up(b, d, 64);
    if (lane >= d) {
      a += ya;
      b += yb;
    }
  }
  if (lane == 63) {
    wsum[0][wave] = a;
    wsum[1][wave] = b;
  }
  __syncthreads();
  unsigned long long ba = 0, bb = 0, ta = 0, tb = 0;
#pragma unroll
  for (int w = 0; w < kThreads / 64; ++w) {
    const unsigned long long sa = wsum[0][w], sb = wsum[1][w];
    ba += (w < wave) ? sa : 0ull;
    bb += (w < wave) ? sb : 0ull;
    ta += sa;
    tb += sb;
  }
  __syncthreads();
  *total = make_ulonglong2(ta, tb);
  return make_ulonglong2(ba + a - v.x, bb + b - v.y);
}

__device__ __forceinline__ uint32_t field16(ulonglong2 v, int k) {
  return uint32_t(((k < 4 ? v.x : v.y) >> (16 * (k & 3))) & 0xFFFFu);
}

// Lengths of 8 consecutive blocks from their rung bytes (8-byte loads where
// the run is whole and aligned, byte loads at a ragged end).
__device__ __forceinline__ uint32_t bits_of_8(const uint8_t* __restrict__ rung, const uint4* tab,
                                              uint32_t nr, int64_t b0, int64_t nblocks) {
  if (!rung) {
    const int64_t n = min(int64_t(8), nblocks - b0);
    return n > 0 ? uint32_t(n) * tab[0].w : 0u;
  }
  uint32_t sum = 0;
  if (b0 + 8 <= nblocks && (reinterpret_cast<uintptr_t>(rung + b0) & 7u) == 0) {
    const uint2 v = *reinterpret_cast<const uint2*>(rung + b0);
#pragma unroll
    for (int i = 0; i < 4; ++i) sum += tab[table_index((v.x >> (8 * i)) & 0xFFu, nr)].w;
#pragma unroll
    for (int i = 0; i < 4; ++i) sum += tab[table_index((v.y >> (8 * i)) & 0xFFu, nr)].w;
  } else {
    for (int64_t b = b0; b < min(b0 + 8, nblocks); ++b) sum += tab[table_index(rung[b], nr)].w;
  }
  return sum;
}

// The 64 stream bits from bit pos on, as (lo, hi); false when the len bits at
// pos are not all inside the stream (then lo and hi are untouched). Bits past
// len belong to the next block, or are zero past the stream's end.
__device__ __forceinline__ bool read_window(const uint32_t* __restrict__ stream, int64_t nwords,
                                            int64_t pos, uint32_t len, uint32_t& lo, uint32_t& hi) {
  if (len == 0u || pos + int64_t(len) > (nwords << 5)) return false;
  const int64_t wi = pos >> 5;
  const uint32_t* sp = stream + wi;
  uint32_t a, b, c;
  if (wi + 2 < nwords) {
    a = sp[0];
    b = sp[1];
    c = sp[2];
  } else {
    a = sp[0];
    b = wi + 1 < nwords ? sp[1] : 0u;
    c = 0u;
  }
  const uint32_t sh = uint32_t(pos) & 31u;
  lo = __builtin_amdgcn_alignbit(b, a, sh);
  hi = __builtin_amdgcn_alignbit(c, b, sh);
  return true;
}

__global__ void __launch_bounds__(kThreads)
chunk_bits_kernel(const uint8_t* __restrict__ rung, RungTable rt, int64_t nblocks,
                  int64_t* __restrict__ chunk) {
  __shared__ uint4 tab[kRungTable];
  fill_rung_table(tab, rt);
  __syncthreads();
  const int64_t b0 = int64_t(blockIdx.x) * kChunk + int64_t(threadIdx.x) * kIters;
  uint32_t v = bits_of_8(rung, tab, uint32_t(rt.n), b0, nblocks);
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d, 64);
  __shared__ uint32_t wsum[kThreads / 64];
  if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = v;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t tot = 0;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) tot += wsum[w];
    chunk[blockIdx.x] = tot;
  }
}

// One workgroup: chunk[c] (bits of chunk c) -> chunk[c] = bit offset of chunk c,
// chunk[nchunks] = total bits, in place. With a stream, also clears the words
// that hold a chunk boundary, the only words two chunks both write. Each of the
// 1024 threads owns a contiguous run of chunks and reads it 8 values at a time
// with independent loads, so the pass is not one load latency per chunk.
constexpr int kScanThreads = 1024;
constexpr int kScanBatch = 8;

__global__ void __launch_bounds__(kScanThreads)
chunk_offsets_kernel(int64_t* __restrict__ chunk, int64_t nchunks, uint32_t* __restrict__ stream,
                     int64_t nwords) {
  __shared__ int64_t part[kScanThreads / 64];
  const int64_t per = (nchunks + kScanThreads - 1) / kScanThreads;
  const int64_t c0 = min(nchunks, int64_t(threadIdx.x) * per);
  const int64_t c1 = min(nchunks, c0 + per);
  int64_t s = 0;
  for (int64_t c = c0; c < c1; c += kScanBatch) {
    int64_t v[kScanBatch];
#pragma unroll
    for (int k = 0; k < kScanBatch; ++k) v[k] = c + k < c1 ? chunk[c + k] : 0;
#pragma unroll
    for (int k = 0; k < kScanBatch; ++k) s += v[k];
  }
  // exclusive scan of the per-thread sums: within each wave by shuffles, then
  // across the waves
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int64_t x = s;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int64_t y = __shfl_up(x, d, 64);
    if (lane >= d) x += y;
  }
  if (lane == 63) part[wave] = x;
  __syncthreads();
  int64_t run = x - s, tot = 0;
#pragma unroll
  for (int w = 0; w < kScanThreads / 64; ++w) {
    run += w < wave ? part[w] : 0;
    tot += part[w];
  }
  if (threadIdx.x == 0) chunk[nchunks] = tot;
  for (int64_t c = c0; c < c1; c += kScanBatch) {
    int64_t v[kScanBatch];
#pragma unroll
    for (int k = 0; k < kScanBatch; ++k) v[k] = c + k < c1 ? chunk[c + k] : 0;
#pragma unroll
    for (int k = 0; k < kScanBatch; ++k) {
      if (c + k < c1) {
        chunk[c + k] = run;
        if (stream && (run >> 5) < nwords) stream[run >> 5] = 0u;
        run += v[k];
      }
    }
  }
  if (stream && threadIdx.x == 0 && (tot >> 5) < nwords) stream[tot >> 5] = 0u;
}

// Table index of every block of this thread's eight (8 bits each) and their
// code lengths as 16-bit fields for wg_exclusive_scan8; blocks past the end
// take the invalid entry (length 0).
__device__ __forceinline__ void chunk_lengths(const uint8_t* __restrict__ rung, const uint4* tab,
                                              uint32_t nr, int64_t base, int64_t nblocks,
                                              unsigned long long& idx, ulonglong2& len) {
  idx = 0ull;
  len = make_ulonglong2(0ull, 0ull);
#pragma unroll
  for (int it = 0; it < kIters; ++it) {
    const int64_t b = base + it * kThreads + threadIdx.x;
    const uint32_t r = b < nblocks ? table_index(rung ? uint32_t(rung[b]) : 0u, nr) : nr;
    idx |= (unsigned long long)r << (8 * it);
    const unsigned long long l = (unsigned long long)tab[r].w << (16 * (it & 3));
    if (it < 4) len.x |= l;
    else len.y |= l;
  }
}

__global__ void __launch_bounds__(kThreads)
pack_kernel(const uint32_t* __restrict__ seed, const uint8_t* __restrict__ expo,
            const int8_t* __restrict__ q, const uint8_t* __restrict__ rung, RungTable rt,
            int64_t nblocks, const int64_t* __restrict__ chunk, uint32_t* __restrict__ stream,
            int64_t nwords) {
  __shared__ uint32_t stage[kStageWords];
  __shared__ uint4 tab[kRungTable];
  fill_rung_table(tab, rt);
  const int64_t base = int64_t(blockIdx.x) * kChunk;
  const int64_t off0 = chunk[blockIdx.x], off1 = chunk[blockIdx.x + 1];
  const int64_t w0 = off0 >> 5;
  const uint32_t shift = uint32_t(off0 & 31);
  const int nw = int((off1 - (w0 << 5) + 31) >> 5);
  for (int i = threadIdx.x; i < nw; i += kThreads) stage[i] = 0u;
  __syncthreads();
  unsigned long long idx;
  ulonglong2 len;
  chunk_lengths(rung, tab, uint32_t(rt.n), base, nblocks, idx, len);
  ulonglong2 tot;
  const ulonglong2 ex = wg_exclusive_scan8(len, &tot);
  uint32_t run = shift;  // bit position inside stage
#pragma unroll
  for (int it = 0; it < kIters; ++it) {
    const int64_t b = base + it * kThreads + threadIdx.x;
    const uint4 in = tab[(idx >> (8 * it)) & 0xFFu];
    const uint32_t pos = run + field16(ex, it);
    run += field16(tot, it);
    if (in.w) {
      const int K = int(in.x), P = int(in.y);
      uint64_t code = uint64_t(seed[b] & ((1u << K) - 1u)) | (uint64_t(expo[b] & 15u) << K);
      const uint2 qw = reinterpret_cast<const uint2*>(q)[b];
      for (int j = 0; j < P; ++j) {
        const uint32_t word = j < 4 ? qw.x : qw.y;
        code |= uint64_t((word >> (8 * (j & 3))) & 15u) << (K + 4 + 4 * j);
      }
      const int wi = int(pos >> 5), sh = int(pos & 31);
      const uint64_t lo = code << sh;
      const uint32_t hi = sh ? uint32_t(code >> (64 - sh)) : 0u;
      atomicOr(&stage[wi], uint32_t(lo));
      if (uint32_t(lo >> 32)) atomicOr(&stage[wi + 1], uint32_t(lo >> 32));
      if (hi) atomicOr(&stage[wi + 2], hi);
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < nw; i += kThreads) {
    const int64_t gw = w0 + i;
    if (gw < nwords) {
      const bool shared = (i == 0 && shift != 0) || (i == nw - 1 && (off1 & 31) != 0);
      if (shared) atomicOr(&stream[gw], stage[i]);
      else stream[gw] = stage[i];
    }
  }
}

// One-pass parse of a chunk: MODE 0 writes the codes (seed, exponent, the P
// mantissas as bytes), MODE 1 the reconstructed weights. A block whose bits
// are not all inside the stream, or whose rung byte is out of range, decodes
// to seed 0 (MODE 1: NaN weights).
template <int MODE>
__global__ void __launch_bounds__(kThreads)
parse_kernel(const uint32_t* __restrict__ stream, int64_t nwords, const uint8_t* __restrict__ rung,
             RungTable rt, int64_t nblocks, const int64_t* __restrict__ chunk,
             uint32_t* __restrict__ seed_out, uint8_t* __restrict__ exp_out,
             int8_t* __restrict__ q_out, float* __restrict__ W_hat) {
  __shared__ uint4 tab[kRungTable];
  fill_rung_table(tab, rt);
  __syncthreads();
  const int64_t base = int64_t(blockIdx.x) * kChunk;
  unsigned long long idx;
  ulonglong2 len;
  chunk_lengths(rung, tab, uint32_t(rt.n), base, nblocks, idx, len);
  ulonglong2 tot;
  const ulonglong2 ex = wg_exclusive_scan8(len, &tot);
  int64_t run = chunk[blockIdx.x];
  // MODE 1: an iteration's 256 blocks are 8 KB of contiguous weights, staged
  // in LDS (two buffers, so one barrier per iteration) and stored so that
  // every store instruction of a wave writes 1 KB without gaps.
  __shared__ float4 stage[MODE == 1 ? 2 : 1][2 * kThreads];
#pragma unroll
  for (int it = 0; it < kIters; ++it) {
    const int64_t b = base + it * kThreads + threadIdx.x;
    const uint4 in = tab[(idx >> (8 * it)) & 0xFFu];
    const int64_t pos = run + field16(ex, it);
    run += field16(tot, it);
    if (MODE == 1 || b < nblocks) {  // MODE 1: every thread, for the barrier
      const int K = int(in.x), P = int(in.y);
      uint32_t lo = 0u, hi = 0u;
      const bool ok = read_window(stream, nwords, pos, in.w, lo, hi);
      const uint32_t s = ok ? lo & ((1u << K) - 1u) : 0u;
      const int e = ok ? int((lo >> K) & 15u) : 0;
      const uint32_t qb = ok ? __builtin_amdgcn_alignbit(hi, lo, uint32_t(K + 4)) : 0u;
      if constexpr (MODE == 0) {
        uint32_t qx = 0u, qy = 0u;
        for (int j = 0; j < P; ++j) {
          const uint32_t byte = uint32_t(__builtin_amdgcn_sbfe(int32_t(qb), 4 * j, 4)) & 0xFFu;
          if (j < 4) qx |= byte << (8 * j);
          else qy |= byte << (8 * (j - 4));
        }
        seed_out[b] = s;
        exp_out[b] = uint8_t(e);
        reinterpret_cast<uint2*>(q_out)[b] = make_uint2(qx, qy);
      } else {
        int32_t acc[kC];
        block_acc_q(ok ? s : 1u, K, P, in.z,
                    [&](int j) { return __builtin_amdgcn_sbfe(int32_t(qb), 4 * j, 4); }, acc);
        float o[kC];
        block_weights(acc, K, e, ok && s != 0u, o);
        float4* buf = stage[it & 1];
        buf[2 * threadIdx.x] = make_float4(o[0], o[1], o[2], o[3]);
        buf[2 * threadIdx.x + 1] = make_float4(o[4], o[5], o[6], o[7]);
        __syncthreads();
        const int64_t b0 = base + it * kThreads;
        const int64_t nlive = nblocks - b0 < kThreads ? nblocks - b0 : kThreads;
        float4* dst = reinterpret_cast<float4*>(W_hat + b0 * kC);
        for (int i = threadIdx.x; i < 2 * nlive; i += kThreads) dst[i] = buf[i];
      }
    }
  }
}

// ---------------------------------------------------------------- decode-GEMV
// y_v = W_hat x_v for nv right-hand sides, W_hat decoded from the stream on the
// fly and never stored (the bandwidth motivation of the codec: a GEMV reads
// l(g)/8 bytes per block instead of 16 for fp16). One wave per row, 256 blocks
// per wave step as 4 sub-steps of 64 consecutive blocks, one per lane, so the
// loads of x stay coalesced. The offsets of all four sub-steps come from one
// wave prefix sum over 64-bit words holding the four bit counts in 16-bit
// fields (a sub-step holds at most 64 x 52 bits). A block's code is read as
// one 64-bit window (two funnel shifts of three words); its rung constants (K,
// P, feedback mask, length) come from a table in LDS. The lane rebuilds the
// block's integers exactly as seedq_decompress does and forms
// d_v = sum_i fp32(acc_i) x_v[8g + i]; since w_hat_i = fp32(acc_i) 2^-(K-1+e)
// exactly, d_v 2^-(K-1+e) is the block's partial product up to fp32 rounding.
// A wave reduction gives y_v[r].

__device__ __forceinline__ uint64_t wave_exclusive_scan64(uint64_t v, uint64_t* total) {
  const int lane = threadIdx.x & 63;
  uint64_t x = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint64_t y = __shfl_up(x, d, 64);
    if (lane >= d) x += y;
  }
  *total = __shfl(x, 63, 64);
  return x - v;
}

// Bits of every row (one wave per row), then exclusive row offsets.
__global__ void __launch_bounds__(kThreads)
row_bits_kernel(const uint8_t* __restrict__ rung, RungTable rt, int64_t nrows, int64_t G,
                int64_t* __restrict__ row_off) {
  __shared__ uint4 tab[kRungTable];
  fill_rung_table(tab, rt);
  __syncthreads();
  const int64_t r = int64_t(blockIdx.x) * (kThreads / 64) + (threadIdx.x >> 6);
  if (r >= nrows) return;
  const int lane = threadIdx.x & 63;
  const uint32_t nr = uint32_t(rt.n);
  int64_t sum = 0;
  const uint8_t* row = rung ? rung + r * G : nullptr;
  for (int64_t g = 8 * lane; g < G; g += 8 * 64) sum += bits_of_8(row, tab, nr, g, G);
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) sum += __shfl_xor(sum, d, 64);
  if (lane == 0) row_off[r] = sum;
}

constexpr int kGemvNB = 4;  // sub-steps of 64 blocks per wave step

// The kernel is bound by issue latency, not bytes: more resident waves hide
// more of it. One vector fits 64 VGPRs (8 waves per SIMD) and four fit 96 (5
// waves) without spilling; two keep the compiler's choice. (Eight vectors go
// to gemv_stream_tile_kernel below.)
template <int NV>
__global__ void __launch_bounds__(kThreads)
__attribute__((amdgpu_waves_per_eu(NV == 1 ? 8 : (NV == 4 ? 5 : 1))))
gemv_stream_kernel(const uint32_t* __restrict__ stream, int64_t nwords,
                   const uint8_t* __restrict__ rung, RungTable rt, int64_t nrows, int64_t G,
                   const int64_t* __restrict__ row_off, const float* __restrict__ x,
                   int64_t ldx, float* __restrict__ y, int64_t ldy) {
  __shared__ uint4 tab[kRungTable];
  fill_rung_table(tab, rt);
  __syncthreads();
  const int64_t r = int64_t(blockIdx.x) * (kThreads / 64) + (threadIdx.x >> 6);
  if (r >= nrows) return;  // wave-uniform
  const int lane = threadIdx.x & 63;
  const uint32_t nr = uint32_t(rt.n);
  float acc[NV];
#pragma unroll
  for (int v = 0; v < NV; ++v) acc[v] = 0.f;
  const uint8_t* row = rung ? rung + r * G : nullptr;
  int64_t run = row_off[r];
  for (int64_t g0 = 0; g0 < G; g0 += 64 * kGemvNB) {
    uint4 info[kGemvNB];
    uint64_t lbits = 0u;  // bit counts of the lane's blocks, 16 bits per sub-step
#pragma unroll
    for (int k = 0; k < kGemvNB; ++k) {
      const int64_t g = g0 + 64 * k + lane;
      info[k] = tab[g < G ? table_index(row ? uint32_t(row[g]) : 0u, nr) : nr];
      lbits |= uint64_t(info[k].w) << (16 * k);
    }
    uint64_t tot;
    const uint64_t ex = wave_exclusive_scan64(lbits, &tot);
#pragma unroll
    for (int k = 0; k < kGemvNB; ++k) {
      const int64_t g = g0 + 64 * k + lane;
      const int64_t pos = run + int64_t((ex >> (16 * k)) & 0xFFFFu);
      run += int64_t((tot >> (16 * k)) & 0xFFFFu);
      if (g < G) {
        const int K = int(info[k].x), P = int(info[k].y);
        const uint32_t len = info[k].w;
        uint32_t lo = 0u, hi = 0u;
        bool ok = read_window(stream, nwords, pos, len, lo, hi);
        const uint32_t s = lo & ((1u << K) - 1u);
        const int e = int((lo >> K) & 15u);
        const uint32_t qb = __builtin_amdgcn_alignbit(hi, lo, uint32_t(K + 4));
        ok = ok && s != 0u;
        int32_t a8[kC];
        block_acc_q(ok ? s : 1u, K, P, info[k].z,
                    [&](int j) { return __builtin_amdgcn_sbfe(int32_t(qb), 4 * j, 4); }, a8);
        float f[kC];
#pragma unroll
        for (int i = 0; i < kC; ++i) f[i] = __int2float_rn(a8[i]);
        const int sc = -(K - 1 + e);
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          const float4* xv = reinterpret_cast<const float4*>(x + v * ldx + g * kC);
          const float4 x0 = xv[0], x1 = xv[1];
          float d = f[0] * x0.x;
          d = fmaf(f[1], x0.y, d);
          d = fmaf(f[2], x0.z, d);
          d = fmaf(f[3], x0.w, d);
          d = fmaf(f[4], x1.x, d);
          d = fmaf(f[5], x1.y, d);
          d = fmaf(f[6], x1.z, d);
          d = fmaf(f[7], x1.w, d);
          acc[v] += ok ? ldexpf(d, sc) : __int_as_float(0x7fc00000);
        }
      }
    }
  }
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    float t = acc[v];
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) t += __shfl_xor(t, d, 64);
    if (lane == 0) y[v * ldy + r] = t;
  }
}

// Decode-GEMV for eight vectors with the products on the matrix core
// (v_mfma_f32_16x16x4_f32). A workgroup of 16 waves takes 16 rows, one wave
// per row decoding 64 consecutive blocks per step exactly as the one-vector
// kernel does (one block per lane, offsets by a wave prefix sum), into a
// 16-row tile of weights in LDS (two buffers, one barrier per step). Then
// wave w multiplies the tile's blocks 4w .. 4w + 3 by the vectors: product m
// takes A[i][k] = weight m of block 4w + k of row i and B[k][n] = x_n at the
// same column, so that lane (i, k) reads 8 consecutive weights of the tile and
// lane (k, n) 8 consecutive entries of x_n. The 16 waves' partial products are
// summed in a fixed order at the end. Rounding: a product passes through at
// most 8 matrix-core accumulations of a step (5 + 7 x 4 roundings), one
// addition per step and the 16-way sum (15). The decode costs the same as in
// the one-vector kernel, so this pays where that kernel's per-vector
// multiply-adds outweigh the tile's barrier and LDS traffic: on an 8192 x 28672
// layer 0.26 against 0.35 ms at eight vectors, but 0.27 against 0.23 at four.
constexpr int kTlRows = 16;
constexpr int kTlBlocks = 64;                  // blocks per row and step
constexpr int kTlStride = kTlBlocks * kC + 4;  // floats per tile row (padded)
typedef float tl_floatx4 __attribute__((ext_vector_type(4)));

template <int NV>
__global__ void __launch_bounds__(64 * kTlRows)
gemv_stream_tile_kernel(const uint32_t* __restrict__ stream, int64_t nwords,
                        const uint8_t* __restrict__ rung, RungTable rt, int64_t nrows, int64_t G,
                        const int64_t* __restrict__ row_off, const float* __restrict__ x,
                        int64_t ldx, float* __restrict__ y, int64_t ldy) {
  static_assert(NV >= 1 && NV <= 16, "one B column per vector");
  static_assert(kTlRows * 4 == kTlBlocks, "each wave multiplies 4 blocks of the tile");
  __shared__ uint4 tab[kRungTable];
  __shared__ __attribute__((aligned(16))) float tile[2][kTlRows][kTlStride];
  fill_rung_table(tab, rt);
  __syncthreads();
  const int wave = int(threadIdx.x >> 6), lane = int(threadIdx.x & 63);
  const int i = lane & 15, k = lane >> 4;
  const int64_t r = int64_t(blockIdx.x) * kTlRows + wave;   // the row this wave decodes
  const bool row_ok = r < nrows;
  const uint32_t nr = uint32_t(rt.n);
  const uint8_t* row = rung && row_ok ? rung + r * G : nullptr;
  int64_t run = row_ok ? row_off[r] : 0;
  tl_floatx4 sum = {0.f, 0.f, 0.f, 0.f};
  int buf = 0;
  for (int64_t g0 = 0; g0 < G; g0 += kTlBlocks) {   // the same trip count in every wave
    // decode block g0 + lane of row r into the tile
    const int64_t g = g0 + lane;
    const bool in = row_ok && g < G;
    const uint4 info = in ? tab[table_index(row ? uint32_t(row[g]) : 0u, nr)]
                          : make_uint4(0u, 0u, 0u, 0u);
    uint64_t tot;
    const uint64_t ex = wave_exclusive_scan64(uint64_t(info.w), &tot);
    const int64_t pos = run + int64_t(ex);
    run += int64_t(tot);
    float f[kC];
#pragma unroll
    for (int e2 = 0; e2 < kC; ++e2) f[e2] = 0.f;
    if (in) {
      const int K = int(info.x), P = int(info.y);
      uint32_t lo = 0u, hi = 0u;
      bool ok = read_window(stream, nwords, pos, info.w, lo, hi);
      const uint32_t sd = lo & ((1u << K) - 1u);
      const int e = int((lo >> K) & 15u);
      const uint32_t qb = __builtin_amdgcn_alignbit(hi, lo, uint32_t(K + 4));
      ok = ok && sd != 0u;
      int32_t a8[kC];
      block_acc_q(ok ? sd : 1u, K, P, info.z,
                  [&](int j) { return __builtin_amdgcn_sbfe(int32_t(qb), 4 * j, 4); }, a8);
      const int sc = -(K - 1 + e);
#pragma unroll
      for (int e2 = 0; e2 < kC; ++e2)
        f[e2] = ok ? ldexpf(__int2float_rn(a8[e2]), sc) : __int_as_float(0x7fc00000);
    }
    float4* dst = reinterpret_cast<float4*>(&tile[buf][wave][lane * kC]);
    dst[0] = make_float4(f[0], f[1], f[2], f[3]);
    dst[1] = make_float4(f[4], f[5], f[6], f[7]);
    __syncthreads();
    // blocks gb = g0 + 4 wave + k of the 16 rows against the vectors
    const int64_t gb = g0 + 4 * wave + k;
    const float4* src = reinterpret_cast<const float4*>(&tile[buf][i][(4 * wave + k) * kC]);
    const float4 a0 = src[0], a1 = src[1];
    float4 b0 = make_float4(0.f, 0.f, 0.f, 0.f), b1 = b0;
    if (i < NV && gb < G) {
      const float4* xv = reinterpret_cast<const float4*>(x + i * ldx + gb * kC);
      b0 = xv[0];
      b1 = xv[1];
    }
    tl_floatx4 acc = {0.f, 0.f, 0.f, 0.f};
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a0.x, b0.x, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a0.y, b0.y, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a0.z, b0.z, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a0.w, b0.w, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a1.x, b1.x, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a1.y, b1.y, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a1.z, b1.z, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a1.w, b1.w, acc, 0, 0, 0);
    sum += acc;
    buf ^= 1;
  }
  // lane l of wave w holds rows 4 (l / 16) + v, vector l % 16; the 16 waves'
  // sums go through the (no longer read) tile
  __syncthreads();
  float* part = &tile[0][0][0];
#pragma unroll
  for (int v = 0; v < 4; ++v) part[(wave * 4 + v) * 64 + lane] = sum[v];
  __syncthreads();
  if (wave == 0) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      float t = part[v * 64 + lane];
      for (int w = 1; w < kTlRows; ++w) t += part[(w * 4 + v) * 64 + lane];
      const int64_t rr = int64_t(blockIdx.x) * kTlRows + 4 * k + v;
      if (i < NV && rr < nrows) y[i * ldy + rr] = t;
    }
  }
}

}  // namespace

int64_t stream_chunks(int64_t nblocks) { return (nblocks + kChunk - 1) / kChunk; }

size_t stream_workspace_bytes(int64_t nblocks, int64_t nrows) {
  const int64_t n = std::max(stream_chunks(nblocks), nrows) + 1;
  return align256(sizeof(int64_t) * size_t(n));
}

static hipError_t launch_offsets(const uint8_t* d_rung, const RungTable& rt, int64_t nblocks,
                                 int64_t* chunk, uint32_t* zero_stream, int64_t nwords,
                                 hipStream_t stream) {
  const int64_t nchunks = stream_chunks(nblocks);
  if (nchunks > 0)
    hipLaunchKernelGGL(chunk_bits_kernel, dim3(unsigned(nchunks)), dim3(kThreads), 0, stream, d_rung,
                       rt, nblocks, chunk);
  hipLaunchKernelGGL(chunk_offsets_kernel, dim3(1), dim3(kScanThreads), 0, stream, chunk, nchunks,
                     zero_stream, nwords);
  return hipGetLastError();
}

hipError_t launch_pack(const uint32_t* d_seed, const uint8_t* d_exp, const int8_t* d_q,
                       const uint8_t* d_rung, const RungTable& rt, int64_t nblocks,
                       uint32_t* d_stream, int64_t nwords, void* d_ws, hipStream_t stream) {
  int64_t* chunk = static_cast<int64_t*>(d_ws);
  hipError_t err = launch_offsets(d_rung, rt, nblocks, chunk, d_stream, nwords, stream);
  if (err != hipSuccess) return err;
  const int64_t nchunks = stream_chunks(nblocks);
  if (nchunks == 0) return hipSuccess;
  hipLaunchKernelGGL(pack_kernel, dim3(unsigned(nchunks)), dim3(kThreads), 0, stream, d_seed, d_exp,
                     d_q, d_rung, rt, nblocks, chunk, d_stream, nwords);
  return hipGetLastError();
}

hipError_t launch_parse(const uint32_t* d_stream, int64_t nwords, const uint8_t* d_rung,
                        const RungTable& rt, int64_t nblocks, void* d_ws, uint32_t* d_seed,
                        uint8_t* d_exp, int8_t* d_q, float* d_W_hat, hipStream_t stream) {
  int64_t* chunk = static_cast<int64_t*>(d_ws);
  hipError_t err = launch_offsets(d_rung, rt, nblocks, chunk, nullptr, 0, stream);
  if (err != hipSuccess) return err;
  const int64_t nchunks = stream_chunks(nblocks);
  if (nchunks == 0) return hipSuccess;
  if (d_W_hat)
    hipLaunchKernelGGL(parse_kernel<1>, dim3(unsigned(nchunks)), dim3(kThreads), 0, stream, d_stream,
                       nwords, d_rung, rt, nblocks, chunk, nullptr, nullptr, nullptr, d_W_hat);
  else
    hipLaunchKernelGGL(parse_kernel<0>, dim3(unsigned(nchunks)), dim3(kThreads), 0, stream, d_stream,
                       nwords, d_rung, rt, nblocks, chunk, d_seed, d_exp, d_q, nullptr);
  return hipGetLastError();
}

hipError_t launch_gemv_stream(const uint32_t* d_stream, int64_t nwords, const uint8_t* d_rung,
                              const RungTable& rt, int64_t nrows, int64_t ncols, void* d_ws,
                              const float* d_x, int64_t ldx, float* d_y, int64_t ldy, int nv,
                              hipStream_t stream) {
  int64_t* row_off = static_cast<int64_t*>(d_ws);
  const int64_t G = ncols / kC;
  const unsigned grid = unsigned((nrows + kThreads / 64 - 1) / (kThreads / 64));
  hipLaunchKernelGGL(row_bits_kernel, dim3(grid), dim3(kThreads), 0, stream, d_rung, rt, nrows, G,
                     row_off);
  hipLaunchKernelGGL(chunk_offsets_kernel, dim3(1), dim3(kScanThreads), 0, stream, row_off, nrows,
                     nullptr, int64_t(0));
  switch (nv) {
    case 1:
      hipLaunchKernelGGL(gemv_stream_kernel<1>, dim3(grid), dim3(kThreads), 0, stream, d_stream,
                         nwords, d_rung, rt, nrows, G, row_off, d_x, ldx, d_y, ldy);
      break;
    case 2:
      hipLaunchKernelGGL(gemv_stream_kernel<2>, dim3(grid), dim3(kThreads), 0, stream, d_stream,
                         nwords, d_rung, rt, nrows, G, row_off, d_x, ldx, d_y, ldy);
      break;
    case 4:
      hipLaunchKernelGGL(gemv_stream_kernel<4>, dim3(grid), dim3(kThreads), 0, stream, d_stream,
                         nwords, d_rung, rt, nrows, G, row_off, d_x, ldx, d_y, ldy);
      break;
    case 8:
      hipLaunchKernelGGL(gemv_stream_tile_kernel<8>, dim3(unsigned((nrows + kTlRows - 1) / kTlRows)),
                         dim3(64 * kTlRows), 0, stream, d_stream, nwords, d_rung, rt, nrows, G,
                         row_off, d_x, ldx, d_y, ldy);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace seedq
