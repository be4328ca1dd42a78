// Internal declarations shared by the translation units of libseedq.so.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "seedq.h"

namespace seedq {

constexpr int kC = 8;            // weights per block (section 3.1, B = 8)
constexpr int kMaxP = SEEDQ_MAX_P;

// Feedback masks of maximal-length Galois LFSRs, K = 8 .. 24 (bit K-1 set).
// Right-shift Galois form: x <- (x >> 1) ^ (x odd ? mask : 0).
__host__ __device__ inline uint32_t lfsr_mask(int K) {
  switch (K) {
    case 8: return 0xB8u;
    case 9: return 0x110u;
    case 10: return 0x240u;
    case 11: return 0x500u;
    case 12: return 0x829u;
    case 13: return 0x100Du;
    case 14: return 0x2015u;
    case 15: return 0x6000u;
    case 16: return 0xD008u;
    case 17: return 0x12000u;
    case 18: return 0x20400u;
    case 19: return 0x40023u;
    case 20: return 0x90000u;
    case 21: return 0x140000u;
    case 22: return 0x300000u;
    case 23: return 0x420000u;
    case 24: return 0xE10000u;
    default: return 0u;
  }
}

__host__ __device__ __forceinline__ uint32_t lfsr_step(uint32_t x, uint32_t mask) {
  return (x >> 1) ^ ((0u - (x & 1u)) & mask);
}

// The least-squares residual bound of the search is a quadratic form in the
// block: ||Q_s^T w||^2 = w^T Pi_s w = sum over pairs i <= j of Pi_s[i][j] z_ij,
// z_ij = c_ij w_i w_j (c = 1 on the diagonal, 2 off it). The 36 pairs, padded
// to 48, form the reduction dimension of three 32x32x16 fp16 MFMAs.
constexpr int kPairs = 36;
constexpr int kPairsPadded = 48;
constexpr int kSeedTile = 32;                   // seeds per MFMA tile (rows)
constexpr float kOperandScale = 4096.0f;        // 2^12 on both fp16 operands
constexpr int kTileBytes = kPairsPadded * kSeedTile * 2;   // 3 KB per seed tile

// Pair index k of (i, j), i <= j, row-major over the upper triangle.
__host__ __device__ constexpr int pair_index(int i, int j) { return i * kC - i * (i - 1) / 2 + (j - i); }

// Rungs whose screen projects blocks onto an orthonormal basis of the
// complement of range(U(s)) (8 - P vectors per seed) instead of forming the
// quadratic form w^T Pi_s w: for large P that complement is small, and its
// projection gives the least-squares residual without cancellation.
constexpr int kComplementMinP = 5;
__host__ __device__ constexpr int complement_dims(int P) { return P >= kComplementMinP ? kC - P : 0; }
// 2^4 on the complement operand: the squared projections of a block scaled to
// max |w_i| in [1, 2) stay below 2^13, inside fp16's range (the P = 6 records)
constexpr float kComplementScale = 16.0f;

// Layout of the opaque per-rung basis stack (all sections 256-byte aligned):
//   pinv64: double [S][P][8]   pinv(U(s)), row-major per seed
//   ub:     uint32 [S][W] the integer basis u[j][i] = x_{8j+i} - 2^(K-1) of
//           every seed (x_0 = s) as pairs of int16, W = basis_words(K, P):
//           word j*8 + i = u[2j][i] | u[2j+1][i] << 16 (zero high half past P);
//           empty above kPackedMaxK. The P >= 5 exact evaluation reads it
//           instead of stepping the LFSR
//   pi16:   fp16 [ntiles][3][64][8] (empty from kComplementMinP on) 2^12 Pi_s[k]
//           as MFMA A-operand fragments:
//           tile T holds seeds 32T+1 .. 32T+32; fragment t, lane l, element e
//           is pair k = 16t + 8(l/32) + e of seed 32T + (l%32) + 1 (zero for
//           k >= 36 and for seeds beyond 2^K - 1)
//   nc16:   fp16 [ntiles][M][64][8], M = complement_dims(P) (empty below
//           kComplementMinP): MFMA A fragments of the complement basis n_c of
//           range(U(s)), c < M; fragment c of tile T, lane l, element e is
//           hi(2^4 n_c[e]) for l < 32 and lo(2^4 n_c[e]) = fp16(2^4 n_c[e] -
//           hi) for l >= 32, of seed 32T + (l % 32) + 1 (zero beyond 2^K - 1)
//   pinv32: float [S][P][8] (empty below kComplementMinP): pinv64 rounded to
//           fp32, from which the many evaluations of these rungs decide their
//           exponent and mantissas when the rounding provably cannot matter
// Widest LFSR whose centred states fit int16 (|x - 2^(K-1)| <= 2^(K-1)).
constexpr int kPackedMaxK = 16;
__host__ __device__ constexpr int basis_words(int K, int P) {
  return K <= kPackedMaxK ? kC * ((P + 1) / 2) : 0;
}

struct BasesLayout {
  int64_t nseeds, ntiles;
  size_t off_pinv64, off_ub, off_pi16, off_nc16, off_pinv32, total;
};

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

inline BasesLayout bases_layout(int K, int P) {
  BasesLayout L;
  L.nseeds = (int64_t(1) << K) - 1;
  L.ntiles = (L.nseeds + kSeedTile - 1) / kSeedTile;
  L.off_pinv64 = 0;
  L.off_ub = align256(L.off_pinv64 + size_t(L.nseeds) * P * kC * sizeof(double));
  L.off_pi16 = align256(L.off_ub + size_t(L.nseeds) * basis_words(K, P) * sizeof(uint32_t));
  L.off_nc16 = align256(L.off_pi16 + (complement_dims(P) > 0 ? 0 : size_t(L.ntiles) * kTileBytes));
  L.off_pinv32 = align256(L.off_nc16 + size_t(L.ntiles) * complement_dims(P) * 64 * kC * 2);
  L.total = align256(L.off_pinv32 +
                     (complement_dims(P) > 0 ? size_t(L.nseeds) * P * kC * sizeof(float) : 0));
  return L;
}

inline bool rung_supported(int K, int P) {
  return K >= SEEDQ_MIN_K && K <= SEEDQ_MAX_K && P >= 1 && P <= kMaxP;
}

// Rung table passed to kernels by value.
struct RungTable {
  int32_t n;
  int32_t K[SEEDQ_MAX_RUNGS];
  int32_t P[SEEDQ_MAX_RUNGS];
};

// Launchers (return hipSuccess or the launch error).
hipError_t launch_build_bases(int K, int P, void* d_bases, int32_t* d_U, float* d_pinv,
                              hipStream_t stream);

// Deterministic, order-preserving split of the blocks by rung:
// lists: int32 [nblocks] (the per-rung lists back to back), meta: see .hip.
size_t compaction_workspace_bytes(int64_t nblocks, int nrungs);
hipError_t launch_compaction(const uint8_t* d_rung, int64_t nblocks, int nrungs, void* d_ws,
                             uint32_t* d_seed_invalid, hipStream_t stream);
// Device pointers into the workspace after launch_compaction.
const int32_t* compaction_list(void* d_ws, int64_t nblocks, int nrungs);
const int32_t* compaction_offsets(void* d_ws, int64_t nblocks, int nrungs);

// Search over all seeds of rung (K, P) for the blocks listed at
// list[off[r] .. off[r+1]) (list == nullptr: all nblocks blocks in order), on
// the matrix cores (seedq_search_mfma.hip).
hipError_t launch_search(const float* d_W, int64_t nblocks, const int32_t* d_list,
                         const int32_t* d_off, int rung_index, int K, int P, const void* d_bases,
                         uint32_t* d_seed, uint8_t* d_exp, int8_t* d_q, float* d_err,
                         hipStream_t stream);

// seedq_compress without its workspace checks (seedq_api.cpp): argument checks
// shared by the compress entry points, then the compaction (nrungs > 1, in
// d_workspace, 256-byte aligned and at least compaction_workspace_bytes) and one
// search per rung. SEEDQ_OK or an error code.
int check_compress_args(const float* d_W, int64_t nrows, int64_t ncols, int32_t C,
                        const uint8_t* d_rung_of_block, int32_t nrungs, const seedq_bases* bases,
                        const uint32_t* d_seed, const uint8_t* d_exp, const int8_t* d_q);
int run_compress(const float* d_W, int64_t nrows, int64_t ncols, const uint8_t* d_rung_of_block,
                 int32_t nrungs, const seedq_bases* bases, uint32_t* d_seed, uint8_t* d_exp,
                 int8_t* d_q, float* d_err, void* d_workspace, hipStream_t stream);

hipError_t launch_decompress(const uint32_t* d_seed, const uint8_t* d_exp, const int8_t* d_q,
                             const uint8_t* d_rung, const RungTable& rt, int64_t nblocks,
                             float* d_W_hat, int32_t* d_acc, hipStream_t stream);

// Code stream (seedq_stream.hip). The workspace holds one int64 per chunk of
// 2048 blocks plus one.
int64_t stream_chunks(int64_t nblocks);
size_t stream_workspace_bytes(int64_t nblocks, int64_t nrows);
hipError_t launch_pack(const uint32_t* d_seed, const uint8_t* d_exp, const int8_t* d_q,
                       const uint8_t* d_rung, const RungTable& rt, int64_t nblocks,
                       uint32_t* d_stream, int64_t nwords, void* d_ws, hipStream_t stream);
// Codes out when d_W_hat is null, reconstructed weights out otherwise.
hipError_t launch_parse(const uint32_t* d_stream, int64_t nwords, const uint8_t* d_rung,
                        const RungTable& rt, int64_t nblocks, void* d_ws, uint32_t* d_seed,
                        uint8_t* d_exp, int8_t* d_q, float* d_W_hat, hipStream_t stream);

// y_v = W_hat x_v for nv in {1, 2, 4, 8} vectors (x_v = d_x + v * ldx).
hipError_t launch_gemv_stream(const uint32_t* d_stream, int64_t nwords, const uint8_t* d_rung,
                              const RungTable& rt, int64_t nrows, int64_t ncols, void* d_ws,
                              const float* d_x, int64_t ldx, float* d_y, int64_t ldy, int nv,
                              hipStream_t stream);

// Fault footprint (seedq_footprint.hip): *d_count = N_flip, d_sums = {sum of
// squared differences, sum of squared clean weights}.
size_t footprint_workspace_bytes();
hipError_t launch_footprint(const float* d_clean, const float* d_corrupt, int64_t n, void* d_ws,
                            long long* d_count, double* d_sums, hipStream_t stream);

// Importance front end (seedq_frontend.hip, seedq_frontend_host.cpp).
size_t sq_gemv_workspace_bytes(int64_t nrows, int64_t ncols, int transpose);
hipError_t launch_sq_gemv(const float* d_W, int64_t nrows, int64_t ncols, const float* d_v,
                          int transpose, double* d_out, void* d_ws, hipStream_t stream);
hipError_t launch_column_stats(const float* d_W, int64_t nrows, int64_t ncols, double* d_max,
                               double* d_median, hipStream_t stream);
hipError_t launch_expect_silu_sq(const double* d_var, int64_t n, int nodes, const double* x,
                                 const double* w, const double* d_scale, double* d_out,
                                 hipStream_t stream);
hipError_t launch_gamma_importance(const float* d_gamma, int64_t n, double* d_a,
                                   hipStream_t stream);
size_t propagate_workspace_bytes(int64_t nrows, int64_t ncols);
hipError_t launch_propagate_o(const float* d_Wv, int64_t nrows, int64_t ncols, int n_heads,
                              int n_kv_heads, const double* d_a_in, double* d_a_o, void* d_ws,
                              hipStream_t stream);
hipError_t launch_propagate_down(const float* d_Wgate, const float* d_Wup, int64_t nrows,
                                 int64_t ncols, const double* d_a_in, int nodes, const double* x,
                                 const double* w, double* d_a_down, void* d_ws,
                                 hipStream_t stream);
hipError_t launch_permute_columns(const float* d_in, int64_t nrows, int64_t ncols,
                                  const int32_t* d_perm, int inverse, float* d_out,
                                  hipStream_t stream);
hipError_t launch_columns_fp16(float* d_W, int64_t nrows, int64_t ncols, int32_t ncol,
                               const int32_t* d_cols, void* d_f16, int apply, hipStream_t stream);
int gauss_hermite(int n, double* x, double* w);
void channel_order(const float* a, int64_t n, int32_t* perm);
int select_outliers(int32_t ntensors, const int64_t* ncols, const double* const* maxabs,
                    const double* const* median, const double* const* a, int32_t keep,
                    int32_t* out_tensor, int32_t* out_col, int32_t* out_count);

// Host planner (seedq_schedule.cpp).
int derive_schedule(const seedq_schedule_desc* desc, double lambda, double floor_q,
                    int64_t tie_count, uint8_t* rung_of_block);
int plan_schedule(const seedq_schedule_desc* desc, uint8_t* rung_of_block,
                  seedq_schedule_report* report);

}  // namespace seedq
