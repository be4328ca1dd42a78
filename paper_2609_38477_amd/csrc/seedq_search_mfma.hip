// Matrix-core engine of the per-block exhaustive seed search (section 3.1;
// the appendix on cost names this search, one least-squares fit per block and
// seed, as what the encoder spends its time on).
//
// Screen. For block w and seed s the least-squares residual
//     r_LS(s) = ||w||^2 - w^T Pi_s w,        Pi_s = projector onto range(U(s)),
// is a lower bound on every quantised error of that seed. w^T Pi_s w is linear
// in the 36 products z_ij = c_ij w_i w_j (i <= j), so the bounds of 32 seeds x
// 32 blocks are one [32 x 48] x [48 x 32] product: three
// v_mfma_f32_32x32x16_f16 with fp16 operands (2^12-scaled projector entries
// from the basis stack, 2^12-scaled pair products of the block) and fp32
// accumulation. A candidate passes when its bound can be at most the block's
// best error so far; the fp16 rounding of the operands is covered by the
// margin gamma = sqrt(P) 2^-10 (1 + 2^-6) + 2^-14 (relative to ||w||^2), so no
// candidate that could win is ever skipped. That margin is relative to
// ||w||^2, while the bound itself is a difference: at P >= 5, where the best
// errors are small beside ||w||^2, the screen instead computes r_LS directly as
// the squared projections of w on 8 - P orthonormal vectors orthogonal to
// range(U(s)) (complement_screen), whose rounding margin is relative to r_LS.
//
// Survivors. Each wave queues its passing (seed, block) pairs in LDS and
// evaluates them 64 at a time, one per lane, with the exact fp64 evaluation
// (seedq_exact.h). In the first kernel a lane whose fold passes first stores
// its 16 bounds as a record; records are turned into queued seeds 64 at a time
// against the thresholds of that moment. Every block's best is its exact fp64
// error (an atomic minimum on the bit pattern in LDS) and the smallest seed of
// that error (record_best), so the result is the exhaustive search's, ties to
// the smallest seed, whatever the order in which survivors are evaluated. A
// pilot pass over the first seed tile finds, per lane, the seed with the
// smallest bound; their exact errors start every block's best, so that the
// walk does not begin with an infinite threshold. The final codes go through
// the same queue.
//
// Work split. A workgroup is 4 independent waves; a wave owns 4 tiles of 32
// blocks (128 blocks) and walks the seed tiles once, reusing each A fragment
// for its 4 block tiles; its B fragments stay in registers for the whole walk.
// Large rungs walk the seed tiles in sequential chunks (see "seed chunks"
// below).
// Block tiles go to the matrix core in pairs (six products) before the vector
// ALU folds them, with one branch per pair; the fold waits on its own
// products, so it is occupancy (several waves per SIMD) that keeps the matrix
// core busy. At P = 4 the fp64 evaluation needs more registers than the walk
// leaves free, so a second kernel rebuilds the block data and reloads the
// seed-tile fragments after every evaluation batch instead of keeping them
// live across it, and runs at four waves per SIMD. (P >= 5 screens with the
// complement projections below, whose block operand is a single fragment, and
// stays in the first kernel.)
#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <type_traits>

#include "seedq_exact.h"
#include "seedq_internal.h"

namespace seedq {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kWaves = 4;
constexpr int kNB = 4;               // 32-block tiles per wave
constexpr int kSlots = kNB * 32;     // blocks per wave
// Per-wave LDS pool of the rebuilding kernel: its queue (fewer than 64 entries
// wait when a pair of block tiles adds its at most 2 x 1024) or, with the
// record stage, the records, their queue and the per-slot threshold data.
constexpr int kPoolWords = 128 + 2 * 1024;
// P = 4 in the rebuilding kernel keeps walk survivors as records (16 bounds
// and a meta word each) in its per-wave pool: 16 records waiting after a pair
// of block tiles, rounds of 32 records (at most 512 queued seeds each). Only
// from K = 13: with fewer seed tiles the per-wave set-up costs more than the
// records save (measured on 2.1 M blocks: (8..10,4) 4-7 % slower, (11,4)
// even, (12,4) 8 % slower, (13..16,4) 2.5-5 % faster, (20,4) 5 % faster).
constexpr int kRecordP = 4;
constexpr bool kRemTable = false;   // the rebuilding kernel steps the LFSR
constexpr int kRecordMinK = 13;
constexpr int kRecFlushR = 16;
constexpr int kRecCapR = kRecFlushR + 64;
constexpr int kRecRound = 32;
constexpr int kRecQueueWords = 64 + kRecRound * 16;
static_assert(kRecQueueWords % 4 == 0, "records start 16-byte aligned");
static_assert(kRecQueueWords + 17 * kRecCapR + 128 + 64 <= kPoolWords,
              "the record stage fits the per-wave pool");
constexpr int kBlocksPerWG = kWaves * kSlots;

// Row and column of pair k (i <= j, row-major over the upper triangle) for
// k < 36; -1 for the padding pairs 36..47. A compile-time table, so that the
// unrolled prologue indexes it with constants.
struct PairTable {
  int i[kPairsPadded];
  int j[kPairsPadded];
};
constexpr PairTable make_pair_table() {
  PairTable t{};
  int k = 0;
  for (int i = 0; i < kC; ++i)
    for (int j = i; j < kC; ++j) {
      t.i[k] = i;
      t.j[k] = j;
      ++k;
    }
  for (; k < kPairsPadded; ++k) {
    t.i[k] = -1;
    t.j[k] = -1;
  }
  return t;
}
constexpr PairTable kPairTable = make_pair_table();
static_assert(kPairTable.i[35] == 7 && kPairTable.j[35] == 7, "36 pairs");
static_assert(pair_index(2, 5) == 18 && kPairTable.i[18] == 2 && kPairTable.j[18] == 5,
              "pair numbering agrees with the basis builder");

template <int K0>
__device__ __forceinline__ float pair_value(const float (&ws)[kC]) {
  constexpr int i = kPairTable.i[K0], j = kPairTable.j[K0];
  if constexpr (i < 0) {
    return 0.f;
  } else {
    return (i == j ? 1.f : 2.f) * ws[i] * ws[j] * kOperandScale;
  }
}

template <int T, int E>
__device__ __forceinline__ _Float16 b_element(const float (&ws)[kC], int h) {
  const float z0 = pair_value<16 * T + E>(ws);
  const float z1 = pair_value<16 * T + 8 + E>(ws);
  return _Float16(h ? z1 : z0);
}

template <int T>
__device__ __forceinline__ half8 b_fragment(const float (&ws)[kC], int h) {
  half8 v;
  v[0] = b_element<T, 0>(ws, h);
  v[1] = b_element<T, 1>(ws, h);
  v[2] = b_element<T, 2>(ws, h);
  v[3] = b_element<T, 3>(ws, h);
  v[4] = b_element<T, 4>(ws, h);
  v[5] = b_element<T, 5>(ws, h);
  v[6] = b_element<T, 6>(ws, h);
  v[7] = b_element<T, 7>(ws, h);
  return v;
}

struct MfmaArgs {
  const float* W;
  int64_t nblocks;
  const int32_t* list;
  const int32_t* off;
  int rung;
  int K;
  uint32_t mask;
  const uint32_t* ub;
  const float* pinv32;
  const double* pinv64;
  const half8* pi16;
  int64_t ntiles;
  float one_minus_gamma;
  uint32_t* seed_out;
  uint8_t* exp_out;
  int8_t* q_out;
  float* err_out;
};

#define SEEDQ_INLINE __device__ __attribute__((always_inline)) inline

SEEDQ_INLINE void load_block(const float* __restrict__ W, int64_t b, bool ok, float (&w)[kC]) {
  float4 lo = make_float4(0.f, 0.f, 0.f, 0.f), hi = lo;
  if (ok) {
    const float4* src = reinterpret_cast<const float4*>(W + b * kC);
    lo = src[0];
    hi = src[1];
  }
  w[0] = lo.x; w[1] = lo.y; w[2] = lo.z; w[3] = lo.w;
  w[4] = hi.x; w[5] = hi.y; w[6] = hi.z; w[7] = hi.w;
}

// Largest of the 16 bounds of a lane. The bounds are finite (products of
// finite fp16 values), so the NaN-propagating maximum equals the IEEE maxNum
// here; it needs no operand canonicalisation and folds as v_maximum3_f32. The
// compiler inserts the wait states between the matrix-core write and the reads.
SEEDQ_INLINE float fold_max(const floatx16& acc) {
  float m = __builtin_elementwise_maximum(__builtin_elementwise_maximum(acc[0], acc[1]), acc[2]);
#pragma unroll
  for (int j = 3; j < 15; j += 2)
    m = __builtin_elementwise_maximum(__builtin_elementwise_maximum(m, acc[j]), acc[j + 1]);
  return __builtin_elementwise_maximum(m, acc[15]);
}

// Wave-wide vote (a bit per lane whose p is set).
SEEDQ_INLINE uint64_t ballot(bool p) { return __builtin_amdgcn_ballot_w64(p); }

SEEDQ_INLINE floatx16 bounds(const half8& a0, const half8& a1, const half8& a2, const half8 (&b)[3]) {
  floatx16 acc = {};
  acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(a0, b[0], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(a1, b[1], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(a2, b[2], acc, 0, 0, 0);
  return acc;
}

// Complement screen (P >= kComplementMinP): the projections d_c = 2^4 n_c^T w
// of a block on the M complement vectors of 32 seeds are M products with K =
// 16 (the hi and lo parts of 2^4 n_c against the block's fp16 weights, given
// twice), and -sum_c d_c^2 is returned so that the max-fold, the records and
// the pilot treat it like the quadratic form's bound: larger passes.
template <int M>
SEEDQ_INLINE floatx16 complement_screen(const half8 (&a)[M], const half8& b) {
  floatx16 d[M];
#pragma unroll
  for (int c = 0; c < M; ++c) d[c] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a[c], b, floatx16{}, 0, 0, 0);
  floatx16 v;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    float r = -(d[0][j] * d[0][j]);
#pragma unroll
    for (int c = 1; c < M; ++c) r = fmaf(-d[c][j], d[c][j], r);
    v[j] = r;
  }
  return v;
}

// Seed of accumulator j of a lane in half h of the wave, for tile seedbase.
SEEDQ_INLINE uint32_t seed_of(uint32_t seedbase, int j, int h) {
  return seedbase + 8u * uint32_t(j / 4) + 4u * uint32_t(h) + uint32_t(j % 4);
}

// Per-block best of a search: the exact fp64 error of the best code so far,
// as its bit pattern (errors are >= 0, so the bits order like the values), in
// LDS, and its seed, the smallest among the codes of exactly that error, in the
// caller's seed array (12 more bytes of LDS per block cost a workgroup per CU:
// measured 11 % slower at (16,3)). A block is only ever touched by the one wave
// that owns it, so one evaluation batch (a candidate per lane, `mine`) updates
// both in four steps: every lane lowers the error; if any lane tied or
// improved, every lane reads the minimum the batch left; a lane that holds
// that minimum while its block held a larger one before resets the seed with
// an atomic exchange that the wave waits for (vmcnt(0): performed in L2; no
// device-wide fence, which on this GPU writes back and invalidates the L2);
// then every lane that holds the minimum lowers the seed to its own. Ties in
// the exact error go to the smallest seed, and the result does not depend on
// the order in which candidates are evaluated.
SEEDQ_INLINE void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

SEEDQ_INLINE void record_best(unsigned long long* best, uint32_t* seed_best, int slot, int64_t b,
                              double err, uint32_t seed, bool mine) {
  const unsigned long long eb = mine ? (unsigned long long)__double_as_longlong(err) : 0ull;
  unsigned long long old = 0ull;
  if (mine) old = atomicMin(&best[slot], eb);
  const bool cand = mine && eb <= old;
  if (__builtin_amdgcn_ballot_w64(cand) == 0ull) return;
  __threadfence_block();
  const unsigned long long now = cand ? best[slot] : ~0ull;
  const bool holds = cand && eb == now;
  const bool reset = holds && old != now;
  if (__builtin_amdgcn_ballot_w64(reset) != 0ull) {
    if (reset) {
      const uint32_t prev = __hip_atomic_exchange(&seed_best[b], seed, __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_AGENT);
      asm volatile("" ::"v"(prev));   // keep the returning form
    }
    wait_vmem();
  }
  if (holds) __hip_atomic_fetch_min(&seed_best[b], seed, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The same update with the seeds in LDS (sbest, one per slot of the wave),
// for the kernels whose LDS has room for them: no global atomics and no wait
// for them. LDS operations of one wave take effect in program order; the
// fence waits for the reset before the minimum. (At P >= 5, where about one
// batch in two improves some block, this measured (12..16,6) 2-11 % and
// (13..16,5) 2-6 % faster on 2.1 M blocks.)
SEEDQ_INLINE void record_best_lds(unsigned long long* best, uint32_t* sbest, int slot, double err,
                                  uint32_t seed, bool mine) {
  const unsigned long long eb = mine ? (unsigned long long)__double_as_longlong(err) : 0ull;
  unsigned long long old = 0ull;
  if (mine) old = atomicMin(&best[slot], eb);
  const bool cand = mine && eb <= old;
  if (__builtin_amdgcn_ballot_w64(cand) == 0ull) return;
  __threadfence_block();
  const unsigned long long now = cand ? best[slot] : ~0ull;
  const bool holds = cand && eb == now;
  const bool reset = holds && old != now;
  if (__builtin_amdgcn_ballot_w64(reset) != 0ull) {
    if (reset) atomicExch(&sbest[slot], seed);
    __threadfence_block();
  }
  if (holds) atomicMin(&sbest[slot], seed);
}

// The best seed of block b once the wave's updates are performed.
SEEDQ_INLINE uint32_t best_seed(const uint32_t* seed_best, int64_t b) {
  return __hip_atomic_load(&seed_best[b], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Number of lanes below this one whose bit is set in mask.
SEEDQ_INLINE int lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi(uint32_t(mask >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(mask), 0u));
}

// This lane's index, recomputed where it is used (volatile, so that it is not
// hoisted and kept live through the walk, where registers are short).
SEEDQ_INLINE uint32_t lane_now() {
  uint32_t l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}

// Queue entries: seed << 8 | final << 7 | slot (slot < 128). Seed 0 = no-op.
constexpr uint32_t kFinal = 0x80u;
static_assert(kSlots <= 128, "slot must fit 7 bits");

// Walk survivors of this kernel are first kept as records: a lane whose fold
// passes stores its 16 bounds with the seed tile, its half and the block slot
// (one row and one meta word in LDS; meta = tile << 8 | half << 7 | slot).
// Records become candidates 64 at a time, each compared with its block's
// threshold of that moment, so the per-seed ballots run once per 64 records
// instead of once per passing block tile, and records whose block has
// meanwhile found a better code drop out before the exact evaluation.
// At P >= 5, where several hundred seeds per block survive the screen, the
// records wait until 64 of them fill a round (kRecRoundMin; the rest wait for
// the next call) and a round's passing bounds are compacted by a prefix sum
// over the lanes instead of one ballot and branch per seed row (measured on
// 2.1 M blocks: (16,6) 9-10 % and (13..16,5) 6-10 % faster than per-row
// ballots over rounds of 32-64).
template <int P>
constexpr int kRecFlush = complement_dims(P) > 0 ? 64 : 32;   // records waiting after a pair
template <int P>
constexpr int kRecCap = kRecFlush<P> + 64;   // one block tile adds at most 64
template <int P>
constexpr int kRecRoundMin = complement_dims(P) > 0 ? 64 : 1;
constexpr int kQCapRec = 64 + 64 * 16;        // < 64 waiting + one round of 64 records
// At P >= 5 (complement screen) records hold their bounds as fp16 (16 x 2
// bytes: two float4 of storage instead of four), which keeps the kernel's LDS
// at 44 KB with 128 records per wave, three workgroups per CU. The values
// -sum d^2 lie in fp16's range (sum d^2 <= 2^8 ||w||^2 < 2^13: the complement
// operand carries 2^4 and the block's power-of-two scaling leaves every |w_i|
// below 2) and are rounded toward zero, i.e. up, so that a stored bound is
// never below the computed one.
__host__ __device__ constexpr bool half_records(int P) { return complement_dims(P) > 0; }
template <int P>
constexpr int kRecVecs = half_records(P) ? 2 : 4;
typedef __fp16 fp16x2 __attribute__((ext_vector_type(2)));

template <int P>
__global__ void __launch_bounds__(kWaves * 64)
__attribute__((amdgpu_waves_per_eu(3)))
search_mfma_kernel(const float* __restrict__ W, int64_t nblocks, const int32_t* __restrict__ list,
                   const int32_t* __restrict__ off, int rung, int K, uint32_t mask,
                   const uint32_t* __restrict__ ub, const float* __restrict__ pinv32,
                   const double* __restrict__ pinv64, const half8* __restrict__ pi16,
                   int64_t ntiles, float one_minus_gamma, uint32_t* __restrict__ seed_out,
                   uint8_t* __restrict__ exp_out, int8_t* __restrict__ q_out,
                   float* __restrict__ err_out, int nchunks, int chunk,
                   unsigned long long* __restrict__ carry) {
  __shared__ unsigned long long best_all[kWaves][kSlots];
  __shared__ int32_t blk_all[kWaves][kSlots];
  __shared__ float thr_base_all[kWaves][kSlots];   // ||w||^2 (1 - gamma) in accumulator units
  // power-of-two scaling of the block: ilogb of its largest |w_i|, down to -149
  // for fp32 subnormals, so 16 bits
  __shared__ int16_t ex_all[kWaves][kSlots];
  // 16 bounds per record: fp32, or fp16 at P >= 5 (see half_records)
  __shared__ float4 rec_all[kWaves][kRecCap<P>][kRecVecs<P>];
  __shared__ uint32_t meta_all[kWaves][kRecCap<P>];
  __shared__ uint32_t queue_all[kWaves][kQCapRec];
  // at P >= 5 the best seed of every slot lives in LDS (2 KB per workgroup;
  // the quadratic-form kernels keep it in seed_out: three of their workgroups
  // per CU leave no room for it) and goes to seed_out when the launch ends
  constexpr bool kSeedsInLds = complement_dims(P) > 0;
  __shared__ uint32_t sbest_all[kWaves][kSeedsInLds ? kSlots : 1];

  const int lane = threadIdx.x & 63;
  // wave-uniform, so that the per-wave LDS addresses are scalar
  const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
  const int n = lane & 31;   // block column of the MFMA tile
  const int h = lane >> 5;   // which half of the rows / reduction this lane holds
  unsigned long long* best = best_all[wave];
  int32_t* blk = blk_all[wave];
  float* slot_thr = thr_base_all[wave];
  int16_t* slot_ex = ex_all[wave];
  float4 (*rec)[kRecVecs<P>] = rec_all[wave];
  uint32_t* meta = meta_all[wave];
  uint32_t* queue = queue_all[wave];
  uint32_t* sbest = sbest_all[wave];

  int64_t begin = 0, count = nblocks;
  if (list) {
    begin = off[rung];
    count = int64_t(off[rung + 1]) - begin;
  }
  const int64_t wave_base = (int64_t(blockIdx.x) * kWaves + wave) * kSlots;
  if (wave_base >= count) return;  // wave-uniform; waves never synchronise
  const uint32_t nseeds = uint32_t((int64_t(1) << K) - 1);
  // quadratic form: 3 A and 3 B fragments per tile; complement screen: M A
  // fragments (one per complement vector) and one B fragment (the weights)
  constexpr int M = complement_dims(P);
  constexpr int NA = M > 0 ? M : 3;
  constexpr int NB = M > 0 ? 1 : 3;
  constexpr int64_t kTileFrags = NA * 64;   // half8 per seed tile of A fragments
  auto screen = [&](const half8 (&a)[NA], const half8 (&b)[NB]) __attribute__((always_inline)) {
    if constexpr (M > 0) return complement_screen<M>(a, b[0]);
    else return bounds(a[0], a[1], a[2], b);
  };

  // ---------------------------------------------------------------- prologue
  half8 bop[kNB][NB];
  float thr[kNB];
  bool active[kNB], valid[kNB];
#pragma unroll
  for (int nt = 0; nt < kNB; ++nt) {
    const int64_t idx = wave_base + nt * 32 + n;
    valid[nt] = idx < count;
    const int64_t b = valid[nt] ? (list ? int64_t(list[begin + idx]) : idx) : 0;
    float w[kC];
    load_block(W, b, valid[nt], w);
    float amax = 0.f;
#pragma unroll
    for (int i = 0; i < kC; ++i) amax = fmaxf(amax, fabsf(w[i]));
    active[nt] = valid[nt] && amax > 0.f;
    const int ex = active[nt] ? ilogbf(amax) : 0;
    float ws[kC], ww = 0.f;
#pragma unroll
    for (int i = 0; i < kC; ++i) {
      ws[i] = ldexpf(w[i], -ex);
      ww = fmaf(ws[i], ws[i], ww);
    }
    thr[nt] = active[nt] ? -INFINITY : INFINITY;
    if constexpr (M > 0) {
#pragma unroll
      for (int e = 0; e < kC; ++e) bop[nt][0][e] = _Float16(ws[e]);
    } else {
      bop[nt][0] = b_fragment<0>(ws, h);
      bop[nt][1] = b_fragment<1>(ws, h);
      bop[nt][2] = b_fragment<2>(ws, h);
    }
    if (h == 0) {
      // a later chunk starts from the best so far (error in carry, seed in
      // seed_out); the first one from none
      best[nt * 32 + n] = chunk > 0 && valid[nt] ? carry[b] : ~0ull;
      if constexpr (kSeedsInLds)
        sbest[nt * 32 + n] = chunk > 0 && valid[nt] ? seed_out[b] : ~0u;
      else if (chunk == 0 && valid[nt])
        seed_out[b] = ~0u;
      blk[nt * 32 + n] = int32_t(b);
      if constexpr (M > 0) {
        // sqrt(M) times the bound on the error of each computed projection,
        // in accumulator units (kComplementScale): fp16 rounding of the
        // weights (2^-11 relative each, Cauchy-Schwarz with |n_c| = 1) plus
        // that of the hi/lo complement vector (2^-22 relative; below fp16's
        // normal range 2^-25 absolute in the 2^4-scaled entries, 2^-29 of
        // n_c) and the fp32 accumulation of 16 exact products,
        // all under 2^-11 (1 + 2^-7) |w| + 2^-20; |w| <= sqrt(ww) (1 + 2^-20)
        const float norm = sqrtf(ww) * (1.0f + 0x1p-20f);
        slot_thr[nt * 32 + n] = sqrtf(float(M)) * (1.0f + 0x1p-20f) * kComplementScale *
                                (0x1p-11f * (1.0f + 0x1p-7f) * norm + 0x1p-20f);
      } else {
        // thresholds live in accumulator units (both operands carry 2^12)
        slot_thr[nt * 32 + n] = ww * one_minus_gamma * (kOperandScale * kOperandScale);
      }
      slot_ex[nt * 32 + n] = int16_t(ex);
    }
  }
  __threadfence_block();
  wait_vmem();   // the seed resets are performed before any update of them

  // Screening threshold of slot s from its best: a bound passes when it can
  // reach the block's best exact error so far (-inf before the first one).
  auto slot_threshold = [&](int s) __attribute__((always_inline)) {
    const unsigned long long key = best[s];
    if (key == ~0ull) return -INFINITY;
    if constexpr (M > 0) {
      // a seed whose residual r_LS(w) is at most the best error b has computed
      // projections of norm <= 2^4 sqrt(b 2^-2ex) + slot_thr (triangle
      // inequality over the M of them), so their fp32 sum of squares (within
      // 2^-20 of its value) is at most T = (2^4 sqrt(b 2^-2ex) + slot_thr)^2
      // (1 + 2^-19). Evaluated in fp32 and rounded up by the factors below:
      // the nearest-rounded conversion (2^-24 relative, 2^-150 absolute below
      // the normal range), sqrtf (1 ulp) and each later rounding (2^-24).
      const float bs = float(ldexp(__longlong_as_double((long long)key), -2 * int(slot_ex[s])));
      const float rb = fmaf(sqrtf(bs), 1.0f + 0x1p-21f, 0x1p-62f);
      const float t = fmaf(rb, kComplementScale, slot_thr[s]) * (1.0f + 0x1p-22f);
      return -(t * t * (1.0f + 0x1p-18f));
    } else {
      return slot_thr[s] - __double2float_ru(ldexp(__longlong_as_double((long long)key),
                                                   24 - 2 * int(slot_ex[s])));
    }
  };
  auto refresh = [&]() __attribute__((always_inline)) {
    __threadfence_block();
#pragma unroll
    for (int nt = 0; nt < kNB; ++nt)
      if (active[nt]) thr[nt] = slot_threshold(nt * 32 + n);
  };

  int qcount = 0;  // wave-uniform
  // Evaluate the top min(64, qcount) candidates, one per lane, until fewer
  // than min_batch remain.
  auto evaluate = [&](int min_batch) __attribute__((always_inline)) {
    __threadfence_block();
    while (qcount >= min_batch && qcount > 0) {
      const int e = qcount < 64 ? qcount : 64;
      const int base = qcount - e;
      bool mine = false;
      uint32_t seed = 0u;
      int slot = 0;
      int64_t b = 0;
      double err = 0.0;
      if (lane < e) {
        const uint32_t ent = queue[base + lane];
        seed = ent >> 8;
        slot = int(ent & 0x7Fu);
        if (seed != 0u) {
          b = blk[slot];
          float w[kC];
          load_block(W, b, true, w);
          int qe, q[P];
          if constexpr (M > 0)
            err = exact_eval_f32<P>(w, pinv32 + int64_t(seed - 1) * (P * kC),
                                    pinv64 + int64_t(seed - 1) * (P * kC),
                                    ub + int64_t(seed - 1) * basis_words(K, P), seed, K, mask, qe,
                                    q);
          else
            err = exact_eval<P, false>(w, pinv64 + int64_t(seed - 1) * (P * kC),
                                       ub + int64_t(seed - 1) * basis_words(K, P), seed, K, mask,
                                       qe, q);
          if (ent & kFinal) {
            seed_out[b] = seed;
            exp_out[b] = uint8_t(qe);
            uint32_t lo = 0, hi = 0;
#pragma unroll
            for (int p = 0; p < P; ++p) {
              const uint32_t byte = uint32_t(uint8_t(int8_t(q[p])));
              if (p < 4) lo |= byte << (8 * p);
              else hi |= byte << (8 * (p - 4));
            }
            reinterpret_cast<uint2*>(q_out)[b] = make_uint2(lo, hi);
            if (err_out) err_out[b] = float(err);
          } else {
            mine = true;
          }
        }
      }
      if constexpr (kSeedsInLds) record_best_lds(best, sbest, slot, err, seed, mine);
      else record_best(best, seed_out, slot, b, err, seed, mine);
      qcount = base;
    }
    __threadfence_block();
  };

  int nrec = 0;  // wave-uniform
  // Records -> candidates: lane l takes record base + l of the top 64 and
  // compares its 16 bounds with the block's current threshold; the passing
  // seeds are queued. Rounds run while at least min_round records wait. Full
  // batches are evaluated after each round of records; the walk's thresholds
  // are refreshed at the end.
  auto process = [&](int min_round) __attribute__((always_inline)) {
    __threadfence_block();
    while (nrec >= min_round && nrec > 0) {
      const int e = nrec < 64 ? nrec : 64;
      const int base = nrec - e;
      const bool live = lane < e;
      uint32_t m = 0u;
      float t = INFINITY;
      float bnd[16];
      if constexpr (half_records(P)) {
        float4 r0 = make_float4(0.f, 0.f, 0.f, 0.f), r1 = r0;
        if (live) {
          m = meta[base + lane];
          t = slot_threshold(int(m & 0x7Fu));
          r0 = rec[base + lane][0];
          r1 = rec[base + lane][1];
        }
        const float r[8] = {r0.x, r0.y, r0.z, r0.w, r1.x, r1.y, r1.z, r1.w};
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const fp16x2 v = __builtin_bit_cast(fp16x2, r[k]);
          bnd[2 * k] = float(v[0]);
          bnd[2 * k + 1] = float(v[1]);
        }
      } else {
        float4 r0 = make_float4(0.f, 0.f, 0.f, 0.f), r1 = r0, r2 = r0, r3 = r0;
        if (live) {
          m = meta[base + lane];
          t = slot_threshold(int(m & 0x7Fu));
          r0 = rec[base + lane][0];
          r1 = rec[base + lane][1];
          r2 = rec[base + lane][2];
          r3 = rec[base + lane][3];
        }
        const float r[16] = {r0.x, r0.y, r0.z, r0.w, r1.x, r1.y, r1.z, r1.w,
                             r2.x, r2.y, r2.z, r2.w, r3.x, r3.y, r3.z, r3.w};
#pragma unroll
        for (int k = 0; k < 16; ++k) bnd[k] = r[k];
      }
      const uint32_t seedbase = (m >> 8) * 32u + 1u;
      const int hh = int((m >> 7) & 1u);
      const uint32_t slot = m & 0x7Fu;
      if constexpr (M > 0) {
        // the lane's passing bounds as a mask (t = +inf on lanes without a
        // record), the exclusive prefix sum of their counts over the wave (by
        // the counts' five bit planes), then one queued seed per lane and step
        uint32_t pm = 0u;
#pragma unroll
        for (int j = 0; j < 16; ++j) pm |= (bnd[j] >= t ? 1u : 0u) << j;
        const uint32_t cnt = uint32_t(__builtin_popcount(pm));
        uint32_t off = uint32_t(qcount);
        int total = 0;
#pragma unroll
        for (int k = 0; k < 5; ++k) {
          const uint64_t mk = ballot(((cnt >> k) & 1u) != 0u);
          off += uint32_t(lanes_below(mk)) << k;
          total += __popcll(mk) << k;
        }
        while (ballot(pm != 0u) != 0ull) {
          if (pm != 0u) {
            // seed_of for the lowest set row j
            const uint32_t j = uint32_t(__builtin_ctz(pm));
            const uint32_t seed = seedbase + 8u * (j >> 2) + 4u * uint32_t(hh) + (j & 3u);
            queue[off] = ((seed <= nseeds ? seed : 0u) << 8) | slot;
            ++off;
            pm &= pm - 1u;
          }
        }
        qcount += total;
      } else {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const bool pass = bnd[j] >= t;   // t = +inf on lanes without a record
          const uint64_t mk = ballot(pass);
          if (mk != 0ull) {
            if (pass) {
              const uint32_t seed = seed_of(seedbase, j, hh);
              queue[qcount + lanes_below(mk)] = ((seed <= nseeds ? seed : 0u) << 8) | slot;
            }
            qcount += __popcll(mk);
          }
        }
      }
      nrec = base;
      if (qcount >= 64) evaluate(64);
    }
    refresh();
  };

  const half8* A = pi16;

  // ---------------------------------------------------------------- pilot
  // Over the first tile each lane tracks its seed of smallest bound; their
  // exact errors start every block's best. (Longer pilots cost more matrix
  // time than the survivors they save.) Later chunks start from the best so far
  // instead.
  if (chunk > 0) {
    refresh();
  } else {
    half8 a[NA];
#pragma unroll
    for (int t = 0; t < NA; ++t) a[t] = A[64 * t + lane];
#pragma unroll
    for (int nt = 0; nt < kNB; ++nt) {
      const floatx16 acc = screen(a, bop[nt]);
      const float mx = fold_max(acc);
      int jb = 15;
#pragma unroll
      for (int j = 14; j >= 0; --j)
        if (acc[j] == mx) jb = j;
      // seeds 1..32 all exist (K >= 8)
      const uint32_t sd = seed_of(1u, jb, h);
      const bool put = active[nt];
      const uint64_t mk = ballot(put);
      if (put) queue[qcount + lanes_below(mk)] = (sd << 8) | uint32_t(nt * 32 + n);
      qcount += __popcll(mk);
      if (qcount >= 64) evaluate(64);
    }
    evaluate(1);
    refresh();
  }

  // ---------------------------------------------------------------- seed walk
  // Lanes of block tile nt whose fold passed store their 16 bounds as records.
  // mk = ballot(pass), taken once by the caller.
  auto record = [&](int nt, const floatx16& acc, bool pass, uint64_t mk, uint32_t T)
                    __attribute__((always_inline)) {
    if (mk == 0ull) return;
    if (pass) {
      const int r = nrec + lanes_below(mk);
      if constexpr (half_records(P)) {
        float pk[8];
#pragma unroll
        for (int k = 0; k < 8; ++k)
          pk[k] = __builtin_bit_cast(float, __builtin_amdgcn_cvt_pkrtz(acc[2 * k], acc[2 * k + 1]));
        rec[r][0] = make_float4(pk[0], pk[1], pk[2], pk[3]);
        rec[r][1] = make_float4(pk[4], pk[5], pk[6], pk[7]);
      } else {
        rec[r][0] = make_float4(acc[0], acc[1], acc[2], acc[3]);
        rec[r][1] = make_float4(acc[4], acc[5], acc[6], acc[7]);
        rec[r][2] = make_float4(acc[8], acc[9], acc[10], acc[11]);
        rec[r][3] = make_float4(acc[12], acc[13], acc[14], acc[15]);
      }
      meta[r] = (T << 8) | (uint32_t(h) << 7) | uint32_t(nt * 32 + n);
    }
    nrec += __popcll(mk);
  };
  static_assert(kNB == 4, "the walk below unrolls four block tiles");

  // One seed tile against the four block tiles: two block tiles at a time,
  // six products to the matrix core, then the folds, one branch per pair.
  // Before each block tile's records at most kRecCap - 64 are waiting.
  auto tile = [&](const half8 (&a)[NA], int64_t T) __attribute__((always_inline)) {
    const uint32_t t32 = uint32_t(T);
#pragma unroll
    for (int pr = 0; pr < 2; ++pr) {
      // raised issue priority while this wave feeds the matrix core, so that
      // its products start ahead of the other waves' folds (measured +0.5 to
      // +1.1 % at (16,3); the rebuilding kernel measured slower with it)
      __builtin_amdgcn_s_setprio(1);
      const floatx16 acc0 = screen(a, bop[2 * pr]);
      const floatx16 acc1 = screen(a, bop[2 * pr + 1]);
      __builtin_amdgcn_s_setprio(0);
      const bool p0 = fold_max(acc0) >= thr[2 * pr];
      const bool p1 = fold_max(acc1) >= thr[2 * pr + 1];
      const uint64_t m0 = ballot(p0), m1 = ballot(p1);
      if ((m0 | m1) != 0ull) {
        record(2 * pr, acc0, p0, m0, t32);
        if (nrec > kRecCap<P> - 64) process(kRecRoundMin<P>);
        record(2 * pr + 1, acc1, p1, m1, t32);
        if (nrec >= kRecFlush<P>) process(kRecRoundMin<P>);
      }
    }
  };
  // Two register sets of seed-tile fragments in turn: the set of one tile is
  // loaded while the other tile is screened. The loads are unconditional (the
  // index is clamped to the last tile) so that the wait before each tile
  // covers only that tile's own loads.
  // Chunk `chunk` walks tiles [T0, T1) (at least 8 of them).
  const int64_t T0 = int64_t(chunk) * ntiles / nchunks, T1 = int64_t(chunk + 1) * ntiles / nchunks;
  const int64_t last = T1 - 1;
  half8 x[NA], y[NA];
#pragma unroll
  for (int t = 0; t < NA; ++t) x[t] = A[T0 * kTileFrags + 64 * t + lane];
  for (int64_t T = T0; T < T1; T += 2) {
    {
      const half8* An = A + (T + 1 < last ? T + 1 : last) * kTileFrags;
#pragma unroll
      for (int t = 0; t < NA; ++t) y[t] = An[64 * t + lane];
    }
    tile(x, T);
    {
      const half8* An = A + (T + 2 < last ? T + 2 : last) * kTileFrags;
#pragma unroll
      for (int t = 0; t < NA; ++t) x[t] = An[64 * t + lane];
    }
    if (T + 1 < T1) tile(y, T + 1);
  }
  process(1);
  evaluate(1);

  // ---------------------------------------------------------------- results
  // A chunk before the last hands its best errors on to the next launch (the
  // seeds are in seed_out already); the last one emits the codes.
  if (chunk + 1 < nchunks) {
#pragma unroll
    for (int nt = 0; nt < kNB; ++nt)
      if (h == 0 && valid[nt]) {
        carry[blk[nt * 32 + n]] = best[nt * 32 + n];
        if constexpr (kSeedsInLds) seed_out[blk[nt * 32 + n]] = sbest[nt * 32 + n];
      }
    return;
  }
  wait_vmem();   // every seed update of this wave is performed
  // the winning seed of every block, evaluated once more to emit its code
#pragma unroll
  for (int nt = 0; nt < kNB; ++nt) {
    const bool put = h == 0 && active[nt];
    const uint64_t mk = ballot(put);
    if (put) {
      // every active block has a best after the pilot; seed 1 is a guard
      uint32_t seed = 1u;
      if (best[nt * 32 + n] != ~0ull) {
        if constexpr (kSeedsInLds) seed = sbest[nt * 32 + n];
        else seed = best_seed(seed_out, blk[nt * 32 + n]);
      }
      queue[qcount + lanes_below(mk)] = (seed << 8) | kFinal | uint32_t(nt * 32 + n);
    }
    qcount += __popcll(mk);
    if (h == 0 && valid[nt] && !active[nt]) {
      // all-zero block: every seed ties, the smallest one wins
      const int64_t b = blk[nt * 32 + n];
      seed_out[b] = 1u;
      exp_out[b] = 15;
      reinterpret_cast<uint2*>(q_out)[b] = make_uint2(0u, 0u);
      if (err_out) err_out[b] = 0.f;
    }
  }
  evaluate(1);
}

// The same search at P = 4, where the fp64 evaluation needs more registers:
// the block data (B fragments and thresholds) and the seed-tile fragments are
// rebuilt from W, the keys and the projector stack after every evaluation
// batch, so none of it is live across that code and the kernel fits four waves
// per SIMD.
template <int P, bool kRec>
__global__ void __launch_bounds__(kWaves * 64) __attribute__((amdgpu_waves_per_eu(4)))
search_mfma_remat_kernel(const float* __restrict__ W, int64_t nblocks, const int32_t* __restrict__ list,
                   const int32_t* __restrict__ off, int rung, int K, uint32_t mask,
                   const uint32_t* __restrict__ ub,
                   const double* __restrict__ pinv64, const half8* __restrict__ pi16,
                   int64_t ntiles, float one_minus_gamma,
                   uint32_t* __restrict__ seed_out, uint8_t* __restrict__ exp_out,
                   int8_t* __restrict__ q_out, float* __restrict__ err_out, int nchunks,
                   int chunk, unsigned long long* __restrict__ carry) {
  // With the record stage (kRec, P = 4 only) the per-wave pool holds the
  // candidate queue, the records (16 bounds and a meta word each) and the
  // per-slot threshold data; otherwise it is the queue alone.
  static_assert(!kRec || P == kRecordP, "records only at P = 4");
  __shared__ unsigned long long best_all[kWaves][kSlots];
  __shared__ int32_t blk_all[kWaves][kSlots];
  __shared__ __attribute__((aligned(16))) uint32_t pool_all[kWaves][kPoolWords];

  const int lane = threadIdx.x & 63;
  // wave-uniform, so that the per-wave LDS addresses are scalar
  // (the other variants measured faster without it)
  const int wave = kRec ? __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6)) : int(threadIdx.x >> 6);
  const int n = lane & 31;   // block column of the MFMA tile
  const int h = lane >> 5;   // which half of the rows / reduction this lane holds
  unsigned long long* best = best_all[wave];
  int32_t* blk = blk_all[wave];
  uint32_t* pool = pool_all[wave];
  uint32_t* queue = pool;
  float4 (*rec)[4] = reinterpret_cast<float4 (*)[4]>(pool + kRecQueueWords);
  uint32_t* meta = pool + kRecQueueWords + 16 * kRecCapR;
  float* slot_thr = reinterpret_cast<float*>(meta + kRecCapR);
  int16_t* slot_ex = reinterpret_cast<int16_t*>(slot_thr + kSlots);   // ilogb, down to -149

  int64_t begin = 0, count = nblocks;
  if (list) {
    begin = off[rung];
    count = int64_t(off[rung + 1]) - begin;
  }
  const int64_t wave_base = (int64_t(blockIdx.x) * kWaves + wave) * kSlots;
  if (wave_base >= count) return;  // wave-uniform; waves never synchronise
  const uint32_t nseeds = uint32_t((int64_t(1) << K) - 1);

  // ---------------------------------------------------------------- prologue
#pragma unroll
  for (int nt = 0; nt < kNB; ++nt) {
    const int64_t idx = wave_base + nt * 32 + n;
    const int64_t b = idx < count ? (list ? int64_t(list[begin + idx]) : idx) : 0;
    if (h == 0) {
      // a later chunk starts from the best so far (its seed is already in
      // seed_out); the first one from none
      best[nt * 32 + n] = chunk > 0 && idx < count ? carry[b] : ~0ull;
      if (chunk == 0 && idx < count) seed_out[b] = ~0u;
      blk[nt * 32 + n] = int32_t(b);
    }
    if constexpr (kRec) {
      if (h == 0) {
        const bool valid = idx < count;
        float w[kC];
        load_block(W, b, valid, w);
        float amax = 0.f;
#pragma unroll
        for (int i = 0; i < kC; ++i) amax = fmaxf(amax, fabsf(w[i]));
        const int ex = valid && amax > 0.f ? ilogbf(amax) : 0;
        float ww = 0.f;
#pragma unroll
        for (int i = 0; i < kC; ++i) {
          const float ws = ldexpf(w[i], -ex);
          ww = fmaf(ws, ws, ww);
        }
        slot_thr[nt * 32 + n] = ww * one_minus_gamma * (kOperandScale * kOperandScale);
        slot_ex[nt * 32 + n] = int16_t(ex);
      }
    }
  }
  __threadfence_block();
  wait_vmem();   // the seed resets are performed before any update of them

  // Per-lane block data: the B fragments (2^12-scaled pair products of the
  // block scaled by a power of two so that max |w_i| lies in [1, 2)) and the
  // screening threshold in accumulator units. Rebuilt from W and the keys after
  // every exact evaluation, so that none of it is live across that code.
  half8 bop[kNB][3];
  float thr[kNB];
  auto setup = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int nt = 0; nt < kNB; ++nt) {
      const bool valid = wave_base + nt * 32 + n < count;
      float w[kC];
      load_block(W, blk[nt * 32 + n], valid, w);
      float amax = 0.f;
#pragma unroll
      for (int i = 0; i < kC; ++i) amax = fmaxf(amax, fabsf(w[i]));
      const bool active = valid && amax > 0.f;
      const int ex = active ? ilogbf(amax) : 0;
      float ws[kC], ww = 0.f;
#pragma unroll
      for (int i = 0; i < kC; ++i) {
        ws[i] = ldexpf(w[i], -ex);
        ww = fmaf(ws[i], ws[i], ww);
      }
      bop[nt][0] = b_fragment<0>(ws, h);
      bop[nt][1] = b_fragment<1>(ws, h);
      bop[nt][2] = b_fragment<2>(ws, h);
      // -inf before a block's first exact error, +inf for blocks not searched
      const unsigned long long key = best[nt * 32 + n];
      const float thr_base = ww * one_minus_gamma * (kOperandScale * kOperandScale);
      thr[nt] = !active ? INFINITY
                : key == ~0ull ? -INFINITY
                : thr_base - __double2float_ru(ldexp(__longlong_as_double((long long)key),
                                                     24 - 2 * ex));
    }
  };

  int qcount = 0;  // wave-uniform
  // Evaluate the top min(64, qcount) queued entries, one per lane, until fewer
  // than min_batch remain; after any evaluation rebuild the block data and
  // thresholds. Returns whether it evaluated (wave-uniform).
  auto exact_with = [&](int min_batch, auto&& rebuild) __attribute__((always_inline)) {
    bool ran = false;
    while (qcount >= min_batch && qcount > 0) {
      const int e = qcount < 64 ? qcount : 64;
      const int base = qcount - e;
      bool mine = false;
      uint32_t seed = 0u;
      int slot = 0;
      int64_t b = 0;
      double err = 0.0;
      if (lane < e) {
        const uint32_t ent = queue[base + lane];
        seed = ent >> 8;
        slot = int(ent & 0x7Fu);
        if (seed != 0u) {
          b = blk[slot];
          float w[kC];
          load_block(W, b, true, w);
          int qe, q[P];
          err = exact_eval<P, kRemTable>(w, pinv64 + int64_t(seed - 1) * (P * kC),
                                         ub + int64_t(seed - 1) * basis_words(K, P), seed, K,
                                         mask, qe, q);
          if (ent & kFinal) {
            seed_out[b] = seed;
            exp_out[b] = uint8_t(qe);
            uint32_t lo = 0, hi = 0;
#pragma unroll
            for (int p = 0; p < P; ++p) {
              const uint32_t byte = uint32_t(uint8_t(int8_t(q[p])));
              if (p < 4) lo |= byte << (8 * p);
              else hi |= byte << (8 * (p - 4));
            }
            reinterpret_cast<uint2*>(q_out)[b] = make_uint2(lo, hi);
            if (err_out) err_out[b] = float(err);
          } else {
            mine = true;
          }
        }
      }
      record_best(best, seed_out, slot, b, err, seed, mine);
      qcount = base;
      ran = true;
    }
    if (ran) {
      __threadfence_block();
      rebuild();
    }
    return ran;
  };
  auto exact = [&](int min_batch) __attribute__((always_inline)) { return exact_with(min_batch, setup); };

  // Records -> queued seeds (P = 4): lane l < 32 takes record base + l of the
  // top 32 and compares its 16 bounds with the block's current threshold; one
  // ballot per seed row queues the passing seeds, and full batches are
  // evaluated after each round, each evaluation followed at once by rebuild()
  // (block data and the fragments the walk still needs), so that none of the
  // walk's state is live across the evaluation.
  int nrec = 0;  // wave-uniform
  auto process = [&](auto&& rebuild) __attribute__((always_inline)) {
    __threadfence_block();
    while (nrec > 0) {
      const int e = nrec < kRecRound ? nrec : kRecRound;
      const int base = nrec - e;
      uint32_t m = 0u;
      float t = INFINITY;
      float4 r0 = make_float4(0.f, 0.f, 0.f, 0.f), r1 = r0, r2 = r0, r3 = r0;
      if (lane < e) {
        m = meta[base + lane];
        const int sl = int(m & 0x7Fu);
        const unsigned long long key = best[sl];
        t = -INFINITY;
        if (key != ~0ull)
          t = slot_thr[sl] - __double2float_ru(ldexp(__longlong_as_double((long long)key),
                                                     24 - 2 * int(slot_ex[sl])));
        r0 = rec[base + lane][0];
        r1 = rec[base + lane][1];
        r2 = rec[base + lane][2];
        r3 = rec[base + lane][3];
      }
      const float bnd[16] = {r0.x, r0.y, r0.z, r0.w, r1.x, r1.y, r1.z, r1.w,
                             r2.x, r2.y, r2.z, r2.w, r3.x, r3.y, r3.z, r3.w};
      const uint32_t seedbase = (m >> 8) * 32u + 1u;
      const int hh = int((m >> 7) & 1u);
      const uint32_t slot = m & 0x7Fu;
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const bool pass = bnd[j] >= t;   // t = +inf on lanes without a record
        const uint64_t mk = ballot(pass);
        if (mk != 0ull) {
          if (pass) {
            const uint32_t seed = seed_of(seedbase, j, hh);
            queue[qcount + lanes_below(mk)] = ((seed <= nseeds ? seed : 0u) << 8) | slot;
          }
          qcount += __popcll(mk);
        }
      }
      nrec = base;
      if (qcount >= 64) exact_with(64, rebuild);
    }
  };
  // Lanes of block tile nt whose fold passed store their 16 bounds as records.
  // mk = ballot(pass), taken once by the caller.
  auto record = [&](int nt, const floatx16& acc, bool pass, uint64_t mk, uint32_t T)
                    __attribute__((always_inline)) {
    if (mk == 0ull) return;
    if (pass) {
      const int r = nrec + lanes_below(mk);
      rec[r][0] = make_float4(acc[0], acc[1], acc[2], acc[3]);
      rec[r][1] = make_float4(acc[4], acc[5], acc[6], acc[7]);
      rec[r][2] = make_float4(acc[8], acc[9], acc[10], acc[11]);
      rec[r][3] = make_float4(acc[12], acc[13], acc[14], acc[15]);
      const uint32_t l = lane_now();   // = lane
      meta[r] = (T << 8) | ((l >> 5) << 7) | (uint32_t(nt * 32) + (l & 31u));
    }
    nrec += __popcll(mk);
  };

  const half8* A = pi16;
  setup();

  // ---------------------------------------------------------------- pilot
  // Over the first tile each lane takes its seed of smallest bound; their exact
  // errors start every block's best. (Longer pilots cost more matrix time than
  // the survivors they save.) Later chunks start from the best so far (setup()
  // above has turned it into thresholds).
  if (chunk == 0) {
    const half8 a0 = A[lane], a1 = A[64 + lane], a2 = A[128 + lane];
#pragma unroll
    for (int nt = 0; nt < kNB; ++nt) {
      const floatx16 acc = bounds(a0, a1, a2, bop[nt]);
      const float m = fold_max(acc);
      int jb = 15;
#pragma unroll
      for (int j = 14; j >= 0; --j)
        if (acc[j] == m) jb = j;
      // seeds 1..32 all exist (K >= 8)
      const uint32_t sd = seed_of(1u, jb, h);
      const bool put = thr[nt] != INFINITY;
      const uint64_t mk = ballot(put);
      if (put) queue[qcount + lanes_below(mk)] = (sd << 8) | uint32_t(nt * 32 + n);
      qcount += __popcll(mk);
    }
    exact(1);
  }

  // ---------------------------------------------------------------- seed walk
  // Queue the candidates of block tile nt whose bound passes, one ballot per
  // seed. At most 1024 per block tile; fewer than 64 are queued before a pair
  // of block tiles, so the 2 x 1024 of one pair always fit.
  auto check = [&](auto ntc, const floatx16& acc, bool any, uint32_t seedbase)
                   __attribute__((always_inline)) {
    constexpr int nt = decltype(ntc)::value;
    if (ballot(any) == 0ull) return;
    // half and slot recomputed here, so that the 16 seed offsets and the slot
    // are not hoisted out of the walk and kept live (or spilled) across it
    const uint32_t l = lane_now();
    const int hh = int(l >> 5);
    const uint32_t slot = uint32_t(nt * 32) + (l & 31u);
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const bool pass = acc[j] >= thr[nt];
      const uint64_t mk = ballot(pass);
      if (mk != 0ull) {
        if (pass) {
          const uint32_t seed = seed_of(seedbase, j, hh);
          queue[qcount + lanes_below(mk)] = ((seed <= nseeds ? seed : 0u) << 8) | slot;
        }
        qcount += __popcll(mk);
      }
    }
  };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I3 = std::integral_constant<int, 3>;
  static_assert(kNB == 4, "the walk below unrolls four block tiles");

  // Seed-tile fragments; the index is clamped to the last tile so that every
  // load is unconditional and each wait covers only the tile it is for.
  // Chunk `chunk` walks tiles [T0, T1) (at least 8 of them).
  const int T0 = int(int64_t(chunk) * ntiles / nchunks), T1 = int(int64_t(chunk + 1) * ntiles / nchunks);
  const int last = T1 - 1;   // 32-bit tile indices (ntiles < 2^19), kept scalar
  auto load_tile = [&](int T, half8 (&f)[3]) __attribute__((always_inline)) {
    // without records the lane's offset is recomputed here, so that no 64-bit
    // per-lane address stays live (or spilled) across the walk (with records
    // the same change makes the allocator spill elsewhere)
    const half8* At = A + (T < last ? T : last) * 192;
    const uint32_t l = kRec ? uint32_t(lane) : lane_now();
    f[0] = At[l];
    f[1] = At[64 + l];
    f[2] = At[128 + l];
  };

  // Seed tile T (fragments c) against the four block tiles, two block tiles
  // at a time: six products to the matrix core, then the folds, one branch per
  // pair. An exact evaluation rebuilds the block data and reloads both this
  // tile's fragments and those of the other set (tile To, in o).
  auto tile = [&](half8 (&c)[3], int T, half8 (&o)[3], int To)
                  __attribute__((always_inline)) {
    const uint32_t seedbase = uint32_t(T) * 32u + 1u;
    {
      const floatx16 acc0 = bounds(c[0], c[1], c[2], bop[0]);
      const floatx16 acc1 = bounds(c[0], c[1], c[2], bop[1]);
      const bool p0 = fold_max(acc0) >= thr[0];
      const bool p1 = fold_max(acc1) >= thr[1];
      const uint64_t m0 = ballot(p0), m1 = ballot(p1);
      if ((m0 | m1) != 0ull) {
        if constexpr (kRec) {
          auto rebuild = [&]() __attribute__((always_inline)) {
            setup();
            load_tile(T, c);
            load_tile(To, o);
          };
          record(0, acc0, p0, m0, uint32_t(T));
          if (nrec > kRecCapR - 64) process(rebuild);
          record(1, acc1, p1, m1, uint32_t(T));
          if (nrec >= kRecFlushR) process(rebuild);
        } else {
          check(I0{}, acc0, p0, seedbase);
          check(I1{}, acc1, p1, seedbase);
          if (qcount >= 64 && exact(64)) {
            load_tile(T, c);
            load_tile(To, o);
          }
        }
      }
    }
    {
      const floatx16 acc2 = bounds(c[0], c[1], c[2], bop[2]);
      const floatx16 acc3 = bounds(c[0], c[1], c[2], bop[3]);
      const bool p2 = fold_max(acc2) >= thr[2];
      const bool p3 = fold_max(acc3) >= thr[3];
      const uint64_t m2 = ballot(p2), m3 = ballot(p3);
      if ((m2 | m3) != 0ull) {
        if constexpr (kRec) {
          auto rebuild = [&]() __attribute__((always_inline)) {
            setup();
            load_tile(To, o);
          };
          record(2, acc2, p2, m2, uint32_t(T));
          if (nrec > kRecCapR - 64) process(rebuild);
          record(3, acc3, p3, m3, uint32_t(T));
          if (nrec >= kRecFlushR) process(rebuild);
        } else {
          check(I2{}, acc2, p2, seedbase);
          check(I3{}, acc3, p3, seedbase);
          if (qcount >= 64 && exact(64)) load_tile(To, o);
        }
      }
    }
  };

  // Two fragment sets in turn: one tile is loaded while the other is screened.
  half8 x[3], y[3];
  load_tile(T0, x);
  for (int T = T0; T < T1; T += 2) {
    load_tile(T + 1, y);
    tile(x, T, y, T + 1);
    load_tile(T + 2, x);
    if (T + 1 < T1) tile(y, T + 1, x, T + 2);
  }
  if constexpr (kRec) process(setup);
  exact(1);

  // ---------------------------------------------------------------- results
  // A chunk before the last hands its best errors on to the next launch (the
  // seeds are in seed_out already); the last one emits the codes.
  if (chunk + 1 < nchunks) {
#pragma unroll
    for (int nt = 0; nt < kNB; ++nt)
      if (h == 0 && wave_base + nt * 32 + n < count) carry[blk[nt * 32 + n]] = best[nt * 32 + n];
    return;
  }
  wait_vmem();   // every seed update of this wave is performed
  // The winning seed of every block, evaluated once more to emit its code.
  // Every searched block holds a best after the pilot; a valid block without
  // one is all zero, where every seed ties and the smallest wins.
#pragma unroll
  for (int nt = 0; nt < kNB; ++nt) {
    const bool valid = wave_base + nt * 32 + n < count;
    const unsigned long long key = best[nt * 32 + n];
    const bool put = h == 0 && valid && key != ~0ull;
    const uint64_t mk = ballot(put);
    if (put)
      queue[qcount + lanes_below(mk)] =
          (best_seed(seed_out, blk[nt * 32 + n]) << 8) | kFinal | uint32_t(nt * 32 + n);
    qcount += __popcll(mk);
    if (h == 0 && valid && key == ~0ull) {
      const int64_t b = blk[nt * 32 + n];
      seed_out[b] = 1u;
      exp_out[b] = 15;
      reinterpret_cast<uint2*>(q_out)[b] = make_uint2(0u, 0u);
      if (err_out) err_out[b] = 0.f;
    }
  }
  exact(1);
}

// ---------------------------------------------------------------- seed chunks
// The seed tiles of a large rung are walked in sequential chunks, one launch
// per chunk of kChunkTiles tiles, so that every wave walks the same 6 MB of
// projector fragments at about the same time and they stay in L2 (one walk
// over a 101 MB stack at K = 20 missed L2 on most requests). Each block stays
// with the same wave position in every launch; a chunk before the last leaves
// the block's best exact error in the caller's mantissa output (8 bytes per
// block, 8-byte aligned) and its seed in the seed output, and the next launch
// starts from them, so only the first runs the pilot and the thresholds are as
// tight as in one walk. The last chunk emits the codes.
constexpr int64_t kChunkTiles = 2048;

int64_t env_int(const char* name, int64_t fallback) {
  if (const char* env = std::getenv(name)) {
    char* end = nullptr;
    const long long v = std::strtoll(env, &end, 10);
    if (end != env && v >= 0) return v;
  }
  return fallback;
}

template <int P>
hipError_t launch_mfma_p(const float* d_W, int64_t nblocks, const int32_t* d_list,
                         const int32_t* d_off, int rung, int K, const void* d_bases,
                         uint32_t* d_seed, uint8_t* d_exp, int8_t* d_q, float* d_err,
                         hipStream_t stream) {
  const BasesLayout L = bases_layout(K, P);
  const char* base = static_cast<const char*>(d_bases);
  const int64_t blocks = (nblocks + kBlocksPerWG - 1) / kBlocksPerWG;
  if (blocks == 0) return hipSuccess;
  MfmaArgs a;
  a.W = d_W;
  a.nblocks = nblocks;
  a.list = d_list;
  a.off = d_off;
  a.rung = rung;
  a.K = K;
  a.mask = lfsr_mask(K);
  a.ub = reinterpret_cast<const uint32_t*>(base + L.off_ub);
  a.pinv64 = reinterpret_cast<const double*>(base + L.off_pinv64);
  a.pinv32 = complement_dims(P) > 0 ? reinterpret_cast<const float*>(base + L.off_pinv32) : nullptr;
  a.pi16 = reinterpret_cast<const half8*>(base + (complement_dims(P) > 0 ? L.off_nc16 : L.off_pi16));
  a.ntiles = L.ntiles;
  const double gamma = std::sqrt(double(P)) * 0x1p-10 * (1.0 + 0x1p-6) + 0x1p-14;
  a.one_minus_gamma = float(1.0 - gamma);
  a.seed_out = d_seed;
  a.exp_out = d_exp;
  a.q_out = d_q;
  a.err_out = d_err;
  // Sequential chunks of the seed tiles (SEEDQ_SEED_CHUNK_TILES overrides the
  // chunk length; 0 = one chunk; at least 8 tiles per chunk).
  const int64_t chunk_tiles = env_int("SEEDQ_SEED_CHUNK_TILES", kChunkTiles);
  const int64_t nseq =
      chunk_tiles > 0 ? std::max<int64_t>(1, std::min<int64_t>(L.ntiles / 8, L.ntiles / chunk_tiles)) : 1;
  unsigned long long* carry = reinterpret_cast<unsigned long long*>(d_q);
  const dim3 grid = dim3(unsigned(blocks), 1u, 1u);
  for (int64_t c = 0; c < nseq; ++c) {
    if constexpr (P == 4) {
      auto kern = search_mfma_remat_kernel<P, false>;
      if constexpr (P == kRecordP)
        if (K >= kRecordMinK) kern = search_mfma_remat_kernel<P, true>;
      hipLaunchKernelGGL(kern, grid, dim3(kWaves * 64), 0,
                         stream, a.W, a.nblocks, a.list, a.off, a.rung, a.K, a.mask, a.ub, a.pinv64,
                         a.pi16, a.ntiles, a.one_minus_gamma, a.seed_out, a.exp_out, a.q_out,
                         a.err_out, int(nseq), int(c), carry);
    } else {
      hipLaunchKernelGGL(search_mfma_kernel<P>, grid, dim3(kWaves * 64), 0, stream,
                         a.W, a.nblocks, a.list, a.off, a.rung, a.K, a.mask, a.ub, a.pinv32,
                         a.pinv64, a.pi16,
                         a.ntiles, a.one_minus_gamma, a.seed_out, a.exp_out, a.q_out, a.err_out,
                         int(nseq), int(c), carry);
    }
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_search(const float* d_W, int64_t nblocks, const int32_t* d_list,
                         const int32_t* d_off, int rung_index, int K, int P, const void* d_bases,
                         uint32_t* d_seed, uint8_t* d_exp, int8_t* d_q, float* d_err,
                         hipStream_t stream) {
  switch (P) {
#define SEEDQ_CASE(PP)                                                                    \
  case PP:                                                                                \
    return launch_mfma_p<PP>(d_W, nblocks, d_list, d_off, rung_index, K, d_bases, d_seed, \
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

}  // namespace seedq
