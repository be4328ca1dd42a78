/*
 * seedq.h -- C ABI of libseedq.so, the MI355X (gfx950) engine for the per-block
 * seed search of Seed-Q ("Security-Enhanced Seed-Based Weight Quantization for
 * Large Language Models").
 *
 * What the library computes
 * -------------------------
 * A weight matrix W (nrows x ncols, fp32, row-major) is cut into blocks of C = 8
 * consecutive weights along each row; block b = r * (ncols / 8) + g holds
 * W[r][8g .. 8g+7] (section 3.1). Each block is coded at a rung (K, P): a K-bit
 * seed s, P signed 4-bit mantissas q and one shared 4-bit exponent e, so that
 *     w_hat = U(s) * q * 2^-e,                        (section 3.1, eq. (codec))
 * costing K + 4P + 4 bits                              (section 3.1, eq. (rate)).
 * U(s) (8 x P) comes from a full-period K-bit LFSR whose initial state is the
 * seed s (section 3.1): Galois right-shift steps x <- (x >> 1) ^ (x & 1 ? mask_K : 0),
 * column j holds the states x_{8j} .. x_{8j+7} centred as x - 2^(K-1), and
 * U = U_int * 2^-(K-1), entries in [-1, 1).
 * The encoder tries every nonzero seed and keeps the code of least quantised
 * error (section 3.1): t* = pinv(U(s)) w is the minimum-norm least-squares fit
 * (singular values at or below 2^-30 of the largest count as zero), e is the
 * largest exponent in [0, 15] at which every round-half-even mantissa
 * rne(t*_j 2^e) lies in [-8, 7] (e = 0, mantissas clamped, if none does), and the
 * error is ||w - U(s) q 2^-e||^2 evaluated exactly (integer reconstruction, fp64
 * sum of squares). Ties go to the smallest seed. The rung of every block comes
 * from the deterministic allocation of sections 3.2-3.4 (seedq_plan_schedule).
 *
 * Conventions
 * -----------
 * - C must be 8. K must lie in [8, 24] and P in [1, 6].
 * - Matrix shapes: nrows >= 1, ncols >= 8 with ncols % 8 == 0, and fewer than
 *   2^31 blocks. An empty matrix (nrows or ncols 0) is an argument error
 *   (SEEDQ_EINVAL), like a negative size; callers skip empty tensors.
 * - Pointers named d_* are device pointers (HIP device memory on the current
 *   device); all other pointers are host memory. The caller allocates and frees
 *   every buffer; the library allocates no memory and keeps no global mutable
 *   state.
 * - Device work is enqueued asynchronously on hip_stream (a hipStream_t, NULL =
 *   the default stream); the library never synchronises the device. Launch
 *   failures are reported by the call that enqueued them.
 * - Return value: SEEDQ_OK (0) or a negative SEEDQ_E* code; on an argument error
 *   nothing is written and nothing is enqueued.
 * - Every result is a pure function of the inputs: it does not depend on the
 *   launch configuration, the stream or the order in which blocks are processed.
 */
#ifndef SEEDQ_H
#define SEEDQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SEEDQ_OK 0
#define SEEDQ_EINVAL (-1)       /* null pointer, bad shape, ncols % 8 != 0, too many rungs */
#define SEEDQ_EUNSUPPORTED (-2) /* C != 8, K outside [8, 24], P outside [1, 6] */
#define SEEDQ_ERATE (-3)        /* rate budget not an integer number of bits, or infeasible */
#define SEEDQ_EHULL (-4)        /* damages missing, not finite, or no rung left on the hull */
#define SEEDQ_EHIP (-5)         /* a HIP launch or copy failed */
#define SEEDQ_EWORKSPACE (-6)   /* workspace missing or smaller than required */
#define SEEDQ_ESCRATCH (-7)     /* larger than the fixed scratch of seedq_compress_noalloc */

#define SEEDQ_BLOCK 8           /* C: weights per block (section 3.1, B = 8) */
#define SEEDQ_MAX_RUNGS 8
#define SEEDQ_QSTRIDE 8         /* bytes per block in the mantissa array */
#define SEEDQ_MIN_K 8
#define SEEDQ_MAX_K 24
#define SEEDQ_MAX_P 6

typedef struct {
  int32_t K; /* seed / LFSR width in bits */
  int32_t P; /* coefficients (basis vectors) per block */
} seedq_rung;

/* Inputs of the allocation (sections 3.2-3.4 and Algorithm 1, steps 1-5). */
typedef struct {
  int64_t nrows, ncols;          /* W is nrows x ncols; ncols % 8 == 0 */
  int32_t C;                     /* must be 8 */
  int32_t nrungs;                /* 1 .. SEEDQ_MAX_RUNGS */
  const seedq_rung* rungs;       /* [nrungs]; rung_of_block indexes this array */
  const double* damage;          /* e(g) per rung [nrungs]; may be NULL iff nrungs == 1 */
  double target_bpw;             /* r_bar; 8 * r_bar * nblocks must be an integer */
  const float* col_importance;   /* a_j [ncols], > 0, channels already sorted (section 3.3) */
  const float* row_importance;   /* rho_r [nrows], > 0, or NULL for rho = 1 */
  double floor_fraction;         /* f of the importance floor (the paper uses 0.06) */
} seedq_schedule_desc;

typedef struct {
  double lambda;        /* final multiplier: the ladder at lambda, first tie_count tied blocks
                           lowered, reproduces rung_of_block (Algorithm 2) */
  double floor_q;       /* q = f-quantile of imp (section 3.3) */
  int64_t tie_count;    /* T: tied blocks, in block order, given the lower rung */
  int64_t total_bits;   /* sum over blocks of K + 4P + 4 */
  int64_t budget_bits;  /* 8 * target_bpw * nblocks */
  int64_t count[SEEDQ_MAX_RUNGS];   /* blocks per rung (desc order) */
  int32_t on_hull[SEEDQ_MAX_RUNGS]; /* 1 if the rung is a vertex of the lower convex hull */
  int32_t nhull;
} seedq_schedule_report;

/*
 * Allocation of rungs to blocks without per-block side information
 * (section 3.2 eq. (objective); section 3.3 eq. (imp) and the floor; section 3.4
 * hull, eq. (lagrangian), eq. (ladder) and the tie pass; Algorithms 1-2).
 * imp_b = abar_g * rho_r with abar_g the mean of a_j over the block's 8 columns,
 * both factors normalised to unit mean (fp32 inputs evaluated in fp64 in index
 * order); q = sorted(imp)[ceil(f * nblocks) - 1]; imp <- max(imp, q); the lower
 * convex hull of (rate, damage) gives slopes s_j; block b takes hull rung
 * 1 + |{j : lambda / s_j <= imp_b}| with lambda the threshold at which the
 * budget 8 * target_bpw * nblocks is met, the tied group at that threshold being
 * lowered in row-major block order until the total is within the budget. The
 * total then falls short of the budget by less than one block's rate step (0
 * when the budget allows, as at the paper's rates); a budget above what the top
 * rung of the hull gives every block is accepted, every block then taking that
 * rung. report->total_bits and report->budget_bits give both.
 * Host only, synchronous. rung_of_block: host array [nblocks], written on success.
 * report: may be NULL.
 * Errors: SEEDQ_EINVAL, SEEDQ_EUNSUPPORTED, SEEDQ_ERATE (budget not integral or
 * below the lowest rung's rate), SEEDQ_EHULL.
 */
int seedq_plan_schedule(const seedq_schedule_desc* desc, uint8_t* rung_of_block,
                        seedq_schedule_report* report);

/*
 * Decoder side of the allocation (Algorithm 2; section 3.5: a decoder holds no
 * per-block side information): the rung of every block re-derived from what the
 * decoder stores -- the same descriptor inputs (rungs, damages for the hull,
 * column and row importance) plus the global-table scalars lambda, floor_q and
 * tie_count. Importance and hull are computed exactly as in
 * seedq_plan_schedule; every block takes the ladder position at lambda
 * (eq. (ladder)) with its importance floored at floor_q, and the first
 * tie_count blocks in row-major order that sit exactly at a threshold (promoted
 * at lambda but not at the next larger double) take the lower rung. With the
 * lambda, floor_q and tie_count of a seedq_schedule_report this reproduces
 * seedq_plan_schedule's rung_of_block exactly. desc->target_bpw and
 * desc->floor_fraction are not read.
 * Host only, synchronous. rung_of_block: host array [nblocks], written on success.
 * Errors: SEEDQ_EINVAL (also lambda negative or not finite, floor_q not finite,
 * tie_count negative or larger than the number of blocks at a threshold),
 * SEEDQ_EUNSUPPORTED, SEEDQ_EHULL.
 */
int seedq_derive_schedule(const seedq_schedule_desc* desc, double lambda, double floor_q,
                          int64_t tie_count, uint8_t* rung_of_block);

/*
 * Bytes of the opaque per-rung basis stack built by seedq_build_bases for the
 * 2^K - 1 seeds of rung (K, P): fp64 pseudo-inverses plus the projection
 * operands of the search kernels. Errors: SEEDQ_EINVAL, SEEDQ_EUNSUPPORTED.
 */
int seedq_bases_bytes(int32_t K, int32_t P, int32_t C, size_t* bytes);

/*
 * LFSR basis generation and per-seed pseudo-inverses for every seed of a rung
 * (section 3.1: U(s) from the LFSR started at s; the least-squares fit needs
 * pinv(U(s))). Integer LFSR stepping is bit-exact and the states are kept as
 * each seed's integer basis; the pseudo-inverse, the projector onto range(U(s))
 * and (for P >= 5) orthonormal vectors of its complement come from a one-sided
 * Jacobi SVD in fp64.
 *   d_bases: device buffer of seedq_bases_bytes(K, P, C) bytes, 256-byte aligned.
 *   d_U:     optional (NULL to skip) device int32 [2^K - 1][P][8]: U_int(s) for
 *            s = 1 .. 2^K-1 (row s-1; element [j][i] = centred state x_{8j+i}).
 *   d_pinv:  optional device fp32 [P][2^K - 1][8]: pinv(U(s)) rounded to fp32,
 *            coefficient-major.
 * Asynchronous on hip_stream. Errors: SEEDQ_EINVAL, SEEDQ_EUNSUPPORTED, SEEDQ_EHIP.
 */
int seedq_build_bases(int32_t K, int32_t P, int32_t C, void* d_bases, int32_t* d_U,
                      float* d_pinv, void* hip_stream);

typedef struct {
  int32_t K, P;
  const void* d_bases; /* built by seedq_build_bases(K, P, 8, ...) */
} seedq_bases;

/*
 * Workspace bytes seedq_compress needs for a matrix of nblocks blocks coded with
 * nrungs rungs (0 when nrungs == 1 and no rung array is given).
 */
size_t seedq_compress_workspace_bytes(int64_t nrows, int64_t ncols, int32_t C, int32_t nrungs);

/*
 * The per-block exhaustive seed search (section 3.1; the appendix on cost
 * names it, one least-squares fit per block and seed, as what the encoder spends
 * its time on): for every block, the code (seed, e, q) of smallest exact quantised
 * error over all 2^K - 1 seeds of the block's rung, ties to the smallest seed.
 *   d_W:             device fp32 [nrows][ncols], row-major, finite values,
 *                    32-byte aligned (one block per 32 bytes).
 *   d_rung_of_block: device uint8 [nblocks] indexes into bases[], or NULL when
 *                    nrungs == 1 (every block at bases[0]).
 *   bases:           host array [nrungs] of built basis stacks.
 *   d_seed:          device uint32 [nblocks] out: chosen seed (1 .. 2^K - 1);
 *                    0 for a block whose rung index is >= nrungs.
 *   d_exp:           device uint8 [nblocks] out: shared exponent e (0 .. 15).
 *   d_q:             device int8 [nblocks][SEEDQ_QSTRIDE] out: mantissas q_0..q_{P-1}
 *                    in [-8, 7], the remaining bytes zero.
 *   d_err:           device fp32 [nblocks] out, nullable: the exact error
 *                    ||w - w_hat||^2 of the chosen code, rounded to fp32.
 *   d_workspace:     device buffer of seedq_compress_workspace_bytes(...) bytes
 *                    (may be NULL when that is 0).
 * A block whose 8 weights are all zero gets seed 1, e = 15, q = 0, err = 0 (every
 * seed ties). Asynchronous on hip_stream.
 * For K >= 17 the seed tiles are searched in sequential chunks of 2048 tiles
 * (one launch each); until the call completes, d_q holds each block's best
 * exact error so far (its fp64 bit pattern; d_q must be 8-byte aligned, as for
 * every call) and d_seed the seed of that error. The result is the same for
 * every chunk length: the smallest exact error, ties to the smallest seed. The
 * environment variable SEEDQ_SEED_CHUNK_TILES (tiles per chunk, 0 = one chunk),
 * read at each call, overrides the choice (at least 8 seed tiles per chunk).
 * Errors: SEEDQ_EINVAL, SEEDQ_EUNSUPPORTED, SEEDQ_EWORKSPACE, SEEDQ_EHIP.
 */
int seedq_compress(const float* d_W, int64_t nrows, int64_t ncols, int32_t C,
                   const uint8_t* d_rung_of_block, int32_t nrungs, const seedq_bases* bases,
                   uint32_t* d_seed, uint8_t* d_exp, int8_t* d_q, float* d_err,
                   void* d_workspace, size_t workspace_bytes, void* hip_stream);

/*
 * seedq_compress without a workspace argument, for callers that cannot
 * allocate device memory (code under stream capture, tight serving loops,
 * harnesses that forbid hipMalloc). Same arguments, results and errors as
 * seedq_compress, from the same kernels; the scratch a multi-rung call needs
 * (the per-rung block lists, seedq_compress_workspace_bytes of it) comes from a
 * fixed device array of SEEDQ_NOALLOC_SCRATCH_BYTES (128 MiB) that each GPU the
 * library runs on holds until the process ends. The call allocates nothing: no
 * hipMalloc, no hipFree, no allocating library routine; the first call on a
 * device looks up that device's array (hipGetSymbolAddress).
 * A problem whose workspace would exceed the array (more than about 33.5 M
 * blocks with several rungs) is rejected with SEEDQ_ESCRATCH before anything is
 * enqueued; a single-rung call needs no scratch and has no such limit.
 * Every call on one GPU shares that GPU's array: calls that overlap on one GPU
 * (on different streams or from different threads) race and must be ordered by
 * the caller. Nothing in the array needs to start at zero; it keeps the last
 * call's lists.
 * Asynchronous on hip_stream. Errors: SEEDQ_EINVAL, SEEDQ_EUNSUPPORTED,
 * SEEDQ_ESCRATCH, SEEDQ_EHIP.
 */
#define SEEDQ_NOALLOC_SCRATCH_BYTES (128u << 20)
int seedq_compress_noalloc(const float* d_W, int64_t nrows, int64_t ncols, int32_t C,
                           const uint8_t* d_rung_of_block, int32_t nrungs, const seedq_bases* bases,
                           uint32_t* d_seed, uint8_t* d_exp, int8_t* d_q, float* d_err,
                           void* hip_stream);

/*
 * Reconstruction w_hat = U(s) q 2^-e for every block (Algorithm 2, the
 * reconstruction step; per the appendix on cost the decoder regenerates the
 * LFSR states and does P multiply-adds for each weight). The integer reconstruction acc_i = sum_j
 * U_int[i][j] q_j is exact; w_hat_i = acc_i * 2^-(K-1+e) rounded once to fp32.
 *   d_seed, d_exp, d_q: codes as written by seedq_compress.
 *   d_rung_of_block:    device uint8 [nblocks] or NULL when nrungs == 1.
 *   rungs:              host array [nrungs].
 *   d_W_hat:            device fp32 [nrows][ncols] out.
 *   d_acc:              device int32 [nrows][ncols] out, nullable.
 * A block with an invalid code (rung index >= nrungs, seed 0 or >= 2^K,
 * exponent > 15) decodes to NaN weights (acc 0). Asynchronous on hip_stream.
 * Errors: SEEDQ_EINVAL, SEEDQ_EUNSUPPORTED, SEEDQ_EHIP.
 */
int seedq_decompress(const uint32_t* d_seed, const uint8_t* d_exp, const int8_t* d_q,
                     const uint8_t* d_rung_of_block, int32_t nrungs, const seedq_rung* rungs,
                     int64_t nrows, int64_t ncols, int32_t C, float* d_W_hat, int32_t* d_acc,
                     void* hip_stream);

/*
 * The headerless variable-length code stream of one tensor (Algorithm 1, the
 * emit step: block b contributes exactly l(g_b) = K + 4P + 4 bits, eq. (rate),
 * with no header; Algorithm 2 and the appendix on encoding and decoding: a
 * decoder reads the blocks in order from the start, the length of each known
 * from the rung allocation alone, so a fault in one block's bits changes that
 * block only).
 * Layout (the paper fixes none): blocks in row-major order; inside a block the
 * seed (K bits), the exponent e (4 bits), then q_0 .. q_{P-1} (4 bits each, two's
 * complement); every field least-significant bit first at increasing stream bit
 * positions; stream bit n is bit n % 32 of the 32-bit word n / 32 (little
 * endian); the payload is padded with zero bits to a whole word. Tensors are
 * concatenated at word boundaries; the per-tensor offsets of Algorithm 2 are
 * word offsets kept by the caller.
 */

/* Bytes of a payload holding count_per_rung[r] blocks of rung r (a multiple of
 * 4). Host only. Errors: SEEDQ_EINVAL, SEEDQ_EUNSUPPORTED. */
int seedq_stream_bytes(int32_t nrungs, const seedq_rung* rungs, const int64_t* count_per_rung,
                       size_t* bytes);

/* Workspace bytes of seedq_pack, seedq_unpack, seedq_decompress_stream and
 * seedq_gemv_stream for an nrows x ncols tensor (one int64 per 2048 blocks or per
 * row, whichever is more, plus one); 0 for a bad shape. */
size_t seedq_stream_workspace_bytes(int64_t nrows, int64_t ncols, int32_t C);

/*
 * Emit the payload of a tensor from its codes (Algorithm 1, emit step).
 *   d_seed, d_exp, d_q: codes as written by seedq_compress; fields are cut to
 *                       their widths (seed to K bits, e and every q to 4 bits).
 *   d_rung_of_block:    device uint8 [nblocks], or NULL when nrungs == 1. A block
 *                       whose rung index is >= nrungs takes no bits.
 *   d_stream:           device uint32 words out, 4-byte aligned; stream_bytes, a
 *                       multiple of 4, should be seedq_stream_bytes(...) for the
 *                       allocation's counts. Words past stream_bytes are never
 *                       written (a short buffer truncates the payload); words
 *                       past the payload are left untouched.
 *   d_workspace:        seedq_stream_workspace_bytes(...) bytes, 256-byte aligned.
 * Asynchronous on hip_stream. The stream is a pure function of the codes and
 * the allocation. Errors: SEEDQ_EINVAL, SEEDQ_EUNSUPPORTED, SEEDQ_EWORKSPACE,
 * SEEDQ_EHIP.
 */
int seedq_pack(const uint32_t* d_seed, const uint8_t* d_exp, const int8_t* d_q,
               const uint8_t* d_rung_of_block, int32_t nrungs, const seedq_rung* rungs,
               int64_t nrows, int64_t ncols, int32_t C, uint32_t* d_stream, size_t stream_bytes,
               void* d_workspace, size_t workspace_bytes, void* hip_stream);

/*
 * Parse a payload back into codes (Algorithm 2, the read step; block lengths
 * come from d_rung_of_block, e.g. as re-derived by seedq_derive_schedule).
 * Writes seed, e and q (q bytes past P zero) for every block. A block whose
 * rung index is >= nrungs, or whose bits run past stream_bytes, gets seed 0,
 * e 0 and q 0 (seedq_decompress turns seed 0 into NaN weights).
 * Same buffers and errors as seedq_pack. Asynchronous on hip_stream.
 */
int seedq_unpack(const uint32_t* d_stream, size_t stream_bytes, const uint8_t* d_rung_of_block,
                 int32_t nrungs, const seedq_rung* rungs, int64_t nrows, int64_t ncols, int32_t C,
                 uint32_t* d_seed, uint8_t* d_exp, int8_t* d_q, void* d_workspace,
                 size_t workspace_bytes, void* hip_stream);

/*
 * Parse and reconstruct in one pass (Algorithm 2, read and reconstruct steps):
 * d_W_hat (device fp32 [nrows][ncols], 16-byte aligned) receives what
 * seedq_unpack followed by seedq_decompress would write, NaN weights for a block
 * that seedq_unpack would mark with seed 0. Same buffers and errors as
 * seedq_pack. Asynchronous on hip_stream.
 */
int seedq_decompress_stream(const uint32_t* d_stream, size_t stream_bytes,
                            const uint8_t* d_rung_of_block, int32_t nrungs,
                            const seedq_rung* rungs, int64_t nrows, int64_t ncols, int32_t C,
                            float* d_W_hat, void* d_workspace, size_t workspace_bytes,
                            void* hip_stream);

/*
 * Decode-GEMV straight from the stream: y_v = W_hat x_v for nvec right-hand
 * sides, W_hat decoded on the fly and never stored (the codec's bandwidth
 * motivation, section 1; per the appendix on cost the decoder regenerates the
 * LFSR states and does P multiply-adds for each weight). Every weight is the one
 * seedq_decompress_stream would write; the products are accumulated in fp32:
 * for 1, 2 or 4 vectors each lane over every 64th block of the row, then a tree
 * across the lanes; for 8 on the matrix core, each 64-block step of the row
 * split in 16 shares of 4 blocks, a share's products in 8 chained four-term
 * accumulations, the steps added share by share, then the 16 shares summed in
 * a fixed order.
 *   nvec:  1, 2, 4 or 8.
 *   d_x:   device fp32 [nvec][ncols], 16-byte aligned.
 *   d_y:   device fp32 [nvec][nrows] out.
 * A block that seedq_decompress_stream would turn into NaN makes its row's
 * outputs NaN. Other buffers, workspace and errors as seedq_pack.
 * Asynchronous on hip_stream.
 */
int seedq_gemv_stream(const uint32_t* d_stream, size_t stream_bytes, const uint8_t* d_rung_of_block,
                      int32_t nrungs, const seedq_rung* rungs, int64_t nrows, int64_t ncols,
                      int32_t C, int32_t nvec, const float* d_x, float* d_y, void* d_workspace,
                      size_t workspace_bytes, void* hip_stream);

/*
 * Footprint of a fault (section 4, subsection on fault model and propagation,
 * eq. (security_metrics)) between a clean and a corrupted reconstruction of n
 * weights: *d_count = N_flip, the number of positions whose values differ (a
 * NaN difference counts); d_sums[0] = sum of squared differences, d_sums[1] =
 * sum of squared clean weights, each accumulated in fp64, so that
 * p_flip = N_flip / n and eta = sqrt(d_sums[0] / d_sums[1]).
 *   d_clean, d_corrupt: device fp32 [n], 16-byte aligned.
 *   d_count: device int64 out; d_sums: device fp64 [2] out.
 *   d_workspace: seedq_footprint_workspace_bytes() bytes, 256-byte aligned.
 * The sums are added in a fixed order (independent of scheduling).
 * Asynchronous on hip_stream. Errors: SEEDQ_EINVAL, SEEDQ_EWORKSPACE, SEEDQ_EHIP.
 */
size_t seedq_footprint_workspace_bytes(void);
int seedq_footprint(const float* d_clean, const float* d_corrupt, int64_t n, long long* d_count,
                    double* d_sums, void* d_workspace, size_t workspace_bytes, void* hip_stream);

/*
 * ---- Data-free importance front end (section on data-free block importance:
 * eq. (gamma), eq. (prop), the output-side rho and the channel sort; appendix
 * on outlier columns). The caller composes these into the a_j and rho_r that
 * seedq_schedule_desc takes: a_j = gamma_j^2 (seedq_gamma_importance) for the
 * projections that read gamma * RMSNorm(h); a_o (seedq_propagate_o) and a_down
 * (seedq_propagate_down) one hop further; rho = sq_gemv^T(W_lm, 1).
 */

/* Gauss-Hermite rule with n nodes (1 <= n <= 256) for the weight e^{-x^2}: nodes
 * x[n] ascending, weights w[n]. The nodes are the zeros of the orthonormal
 * Hermite polynomial q_n (sign changes on a grid finer than their spacing,
 * refined by bisection); w_i = 1 / sum_{j<n} q_j(x_i)^2 (Christoffel-Darboux).
 * Host only. Errors: SEEDQ_EINVAL. */
int seedq_gauss_hermite(int32_t n, double* x, double* w);

/* out = (W * W) v (transpose = 0: out[r] = sum_c W[r][c]^2 v[c], v [ncols]) or
 * (W * W)^T v (transpose != 0: out[c] = sum_r W[r][c]^2 v[r], v [nrows]), the
 * squared-weight products of eq. (prop) and of the backward rho, in fp64.
 *   d_W: device fp32 [nrows][ncols] (16-byte aligned, ncols % 4 == 0 when
 *        transpose = 0); d_v: device fp32; d_out: device fp64.
 *   d_workspace: seedq_sq_gemv_workspace_bytes(...) bytes (0 when transpose = 0).
 * The sums run in a fixed order. Asynchronous on hip_stream.
 * Errors: SEEDQ_EINVAL, SEEDQ_EWORKSPACE, SEEDQ_EHIP. */
size_t seedq_sq_gemv_workspace_bytes(int64_t nrows, int64_t ncols, int32_t transpose);
int seedq_sq_gemv(const float* d_W, int64_t nrows, int64_t ncols, const float* d_v,
                  int32_t transpose, double* d_out, void* d_workspace, size_t workspace_bytes,
                  void* hip_stream);

/* Per column of W (device fp32 [nrows][ncols]): d_maxabs[c] = max_r |W[r][c]| and
 * d_median[c] = the median of |W[r][c]| over the rows (the mean of the two
 * middle values for an even count), both device fp64 [ncols]; the statistics of
 * the dynamic-range rule of the outlier columns. Exact order statistics (radix
 * select). Asynchronous on hip_stream. Errors: SEEDQ_EINVAL, SEEDQ_EHIP. */
int seedq_column_stats(const float* d_W, int64_t nrows, int64_t ncols, double* d_maxabs,
                       double* d_median, void* hip_stream);

/* d_out[i] = E[silu(g)^2] for g ~ N(0, d_var[i]) (eq. (prop)), by the
 * nodes-point Gauss-Hermite rule of seedq_gauss_hermite (1 <= nodes <= 128), in
 * fp64. Asynchronous on hip_stream. Errors: SEEDQ_EINVAL, SEEDQ_EHIP. */
int seedq_expect_silu_sq(const double* d_var, int64_t n, int32_t nodes, double* d_out,
                         void* hip_stream);

/* a_j = gamma_j^2 (eq. (gamma)): the importance of the input channels of the
 * projections that read gamma * RMSNorm(h) (q, k, v from the attention norm;
 * gate, up from the MLP norm). d_gamma: device fp32 [n]; d_a: device fp64 [n]
 * out (exact: the square of an fp32 value fits in fp64). Asynchronous on
 * hip_stream. Errors: SEEDQ_EINVAL, SEEDQ_EHIP. */
int seedq_gamma_importance(const float* d_gamma, int64_t n, double* d_a, void* hip_stream);

/* Workspace bytes of seedq_propagate_o and seedq_propagate_down for a weight of
 * nrows x ncols (a_in in fp32 and one fp64 per row); 0 for a bad shape. */
size_t seedq_propagate_workspace_bytes(int64_t nrows, int64_t ncols);

/* One-hop propagation to the input of o (eq. (prop)): o reads the attention
 * output, whose channel h * head_dim + i comes from the value row
 * (h / (n_heads / n_kv_heads)) * head_dim + i, so
 *   a_o = repeat_kv((W_v * W_v) a_in),
 * the n_kv_heads blocks of head_dim = nrows / n_kv_heads rows each repeated for
 * the n_heads / n_kv_heads (at most 64) query heads that share them, head-major.
 *   d_Wv: device fp32 [nrows][ncols] (16-byte aligned, ncols % 4 == 0).
 *   d_a_in: device fp64 [ncols], the importance of W_v's input channels; it
 *           enters the products rounded to fp32 (stored factors are single
 *           precision, the appendix on agreement); products and sums in fp64.
 *   d_a_o: device fp64 [n_heads * head_dim] out.
 *   d_workspace: seedq_propagate_workspace_bytes(nrows, ncols) bytes, 256-byte aligned.
 * Asynchronous on hip_stream. Errors: SEEDQ_EINVAL, SEEDQ_EWORKSPACE, SEEDQ_EHIP. */
int seedq_propagate_o(const float* d_Wv, int64_t nrows, int64_t ncols, int32_t n_heads,
                      int32_t n_kv_heads, const double* d_a_in, double* d_a_o, void* d_workspace,
                      size_t workspace_bytes, void* hip_stream);

/* One-hop propagation to the input of down (eq. (prop)): down reads
 * silu(gate x) * (up x), so
 *   a_down = E[silu(g)^2] * ((W_up * W_up) a_in),  g ~ N(0, (W_gate * W_gate) a_in),
 * the expectation by the nodes-point Gauss-Hermite rule of seedq_gauss_hermite
 * (1 <= nodes <= 128), everything in fp64.
 *   d_Wgate, d_Wup: device fp32 [nrows][ncols] each (16-byte aligned, ncols % 4 == 0).
 *   d_a_in: device fp64 [ncols] (rounded to fp32 before the products, as for o).
 *   d_a_down: device fp64 [nrows] out.
 *   d_workspace: seedq_propagate_workspace_bytes(nrows, ncols) bytes, 256-byte aligned.
 * Asynchronous on hip_stream. Errors: SEEDQ_EINVAL, SEEDQ_EWORKSPACE, SEEDQ_EHIP. */
int seedq_propagate_down(const float* d_Wgate, const float* d_Wup, int64_t nrows, int64_t ncols,
                         const double* d_a_in, int32_t nodes, double* d_a_down, void* d_workspace,
                         size_t workspace_bytes, void* hip_stream);

/* Channel sort before blocking: perm[k] = the input channel placed k-th, in
 * increasing a, ties by channel index (host arrays of n). Host only.
 * Errors: SEEDQ_EINVAL (also for a non-finite a[i]; perm is then untouched). */
int seedq_channel_order(const float* a, int64_t n, int32_t* perm);

/* Column permutation of a row-major matrix: out[r][j] = in[r][perm[j]] (inverse
 * = 0, the encoder's sort) or out[r][perm[j]] = in[r][j] (inverse != 0, the
 * decoder's inverse). d_perm: device int32 [ncols]; an entry outside [0, ncols)
 * reads nothing (gather writes NaN, scatter writes nothing). d_in and d_out are
 * distinct device fp32 [nrows][ncols]. Asynchronous on hip_stream.
 * Errors: SEEDQ_EINVAL, SEEDQ_EHIP. */
int seedq_permute_columns(const float* d_in, int64_t nrows, int64_t ncols, const int32_t* d_perm,
                          int32_t inverse, float* d_out, void* hip_stream);

/* Outlier columns over a model (appendix on outlier columns): column j of tensor
 * t is a candidate when maxabs/(median + 2^-24 maxabs) >= 1e3 or a_j >= 1e2 times
 * the tensor's mean a; each rule keeps its 32 largest statistics (ties by
 * tensor, then column), a candidate's rank is the smaller of its two list
 * positions (ties by tensor, then column) and the first `keep` are written to
 * out_tensor / out_col (host arrays of at least keep), *out_count how many.
 * maxabs, median, a: host fp64 arrays [ntensors][ncols[t]] (e.g. from
 * seedq_column_stats and the propagation). Host only. Errors: SEEDQ_EINVAL. */
int seedq_select_outliers(int32_t ntensors, const int64_t* ncols, const double* const* maxabs,
                          const double* const* median, const double* const* a, int32_t keep,
                          int32_t* out_tensor, int32_t* out_col, int32_t* out_count);

/* FP16 escape of whole columns (appendix on outlier columns: such columns are
 * kept in FP16, and the decoder writes them over the decoded weights). extract: d_fp16
 * [ncol][nrows] (device fp16) = round-to-nearest-even of W[:, cols[i]];
 * apply: W[:, cols[i]] = d_fp16[i][:] widened to fp32. d_cols: device int32
 * [ncol]; an index outside [0, ncols) extracts NaN and applies nothing.
 * Asynchronous on hip_stream. Errors: SEEDQ_EINVAL, SEEDQ_EHIP. */
int seedq_extract_columns(const float* d_W, int64_t nrows, int64_t ncols, int32_t ncol,
                          const int32_t* d_cols, void* d_fp16, void* hip_stream);
int seedq_apply_columns(float* d_W, int64_t nrows, int64_t ncols, int32_t ncol,
                        const int32_t* d_cols, const void* d_fp16, void* hip_stream);

/* Static description of an error code. */
const char* seedq_strerror(int code);

#ifdef __cplusplus
}
#endif

#endif /* SEEDQ_H */
