// C ABI entry points of libseedq.so: argument checks and launches.
#include <cmath>
#include <cstring>

#include "seedq_internal.h"

using namespace seedq;

namespace {

bool shape_ok(int64_t nrows, int64_t ncols) {
  if (nrows <= 0 || ncols <= 0 || ncols % kC != 0) return false;
  const int64_t G = ncols / kC;
  return nrows <= (int64_t(1) << 31) / G && nrows * G < (int64_t(1) << 31);
}

}  // namespace

namespace seedq {

int check_compress_args(const float* d_W, int64_t nrows, int64_t ncols, int32_t C,
                        const uint8_t* d_rung_of_block, int32_t nrungs, const seedq_bases* bases,
                        const uint32_t* d_seed, const uint8_t* d_exp, const int8_t* d_q) {
  if (C != kC) return SEEDQ_EUNSUPPORTED;
  if (!d_W || !bases || !d_seed || !d_exp || !d_q) return SEEDQ_EINVAL;
  if (!shape_ok(nrows, ncols) || nrungs < 1 || nrungs > SEEDQ_MAX_RUNGS) return SEEDQ_EINVAL;
  if (reinterpret_cast<uintptr_t>(d_W) & 31u || reinterpret_cast<uintptr_t>(d_q) & 7u)
    return SEEDQ_EINVAL;
  for (int r = 0; r < nrungs; ++r) {
    if (!rung_supported(bases[r].K, bases[r].P)) return SEEDQ_EUNSUPPORTED;
    if (!bases[r].d_bases) return SEEDQ_EINVAL;
  }
  if (nrungs > 1 && !d_rung_of_block) return SEEDQ_EINVAL;
  return SEEDQ_OK;
}

int run_compress(const float* d_W, int64_t nrows, int64_t ncols, const uint8_t* d_rung_of_block,
                 int32_t nrungs, const seedq_bases* bases, uint32_t* d_seed, uint8_t* d_exp,
                 int8_t* d_q, float* d_err, void* d_workspace, hipStream_t stream) {
  const int64_t nb = nrows * (ncols / kC);
  if (nrungs == 1) {
    const hipError_t e = launch_search(d_W, nb, nullptr, nullptr, 0, bases[0].K, bases[0].P,
                                       bases[0].d_bases, d_seed, d_exp, d_q, d_err, stream);
    return e == hipSuccess ? SEEDQ_OK : SEEDQ_EHIP;
  }
  hipError_t e = launch_compaction(d_rung_of_block, nb, nrungs, d_workspace, d_seed, stream);
  if (e != hipSuccess) return SEEDQ_EHIP;
  const int32_t* list = compaction_list(d_workspace, nb, nrungs);
  const int32_t* off = compaction_offsets(d_workspace, nb, nrungs);
  for (int r = 0; r < nrungs; ++r) {
    e = launch_search(d_W, nb, list, off, r, bases[r].K, bases[r].P, bases[r].d_bases, d_seed,
                      d_exp, d_q, d_err, stream);
    if (e != hipSuccess) return SEEDQ_EHIP;
  }
  return SEEDQ_OK;
}

}  // namespace seedq

extern "C" {

const char* seedq_strerror(int code) {
  switch (code) {
    case SEEDQ_OK: return "success";
    case SEEDQ_EINVAL: return "invalid argument (null pointer, shape, or rung count)";
    case SEEDQ_EUNSUPPORTED: return "unsupported parameter (C must be 8, K in [8,24], P in [1,6])";
    case SEEDQ_ERATE: return "rate budget not integral or infeasible";
    case SEEDQ_EHULL: return "damages missing or no usable rung on the lower convex hull";
    case SEEDQ_EHIP: return "HIP launch failed";
    case SEEDQ_EWORKSPACE: return "workspace missing or too small";
    case SEEDQ_ESCRATCH:
      return "problem larger than the fixed scratch of the allocation-free compress call";
    default: return "unknown error";
  }
}

int seedq_plan_schedule(const seedq_schedule_desc* desc, uint8_t* rung_of_block,
                        seedq_schedule_report* report) {
  return plan_schedule(desc, rung_of_block, report);
}

int seedq_derive_schedule(const seedq_schedule_desc* desc, double lambda, double floor_q,
                          int64_t tie_count, uint8_t* rung_of_block) {
  return derive_schedule(desc, lambda, floor_q, tie_count, rung_of_block);
}

int seedq_bases_bytes(int32_t K, int32_t P, int32_t C, size_t* bytes) {
  if (!bytes) return SEEDQ_EINVAL;
  if (C != kC || !rung_supported(K, P)) return SEEDQ_EUNSUPPORTED;
  *bytes = bases_layout(K, P).total;
  return SEEDQ_OK;
}

int seedq_build_bases(int32_t K, int32_t P, int32_t C, void* d_bases, int32_t* d_U,
                      float* d_pinv, void* hip_stream) {
  if (C != kC || !rung_supported(K, P)) return SEEDQ_EUNSUPPORTED;
  if (!d_bases || (reinterpret_cast<uintptr_t>(d_bases) & 255u)) return SEEDQ_EINVAL;
  const hipError_t err =
      launch_build_bases(K, P, d_bases, d_U, d_pinv, static_cast<hipStream_t>(hip_stream));
  return err == hipSuccess ? SEEDQ_OK : SEEDQ_EHIP;
}

size_t seedq_compress_workspace_bytes(int64_t nrows, int64_t ncols, int32_t C, int32_t nrungs) {
  if (C != kC || !shape_ok(nrows, ncols) || nrungs <= 1 || nrungs > SEEDQ_MAX_RUNGS) return 0;
  return compaction_workspace_bytes(nrows * (ncols / kC), nrungs);
}

int seedq_compress(const float* d_W, int64_t nrows, int64_t ncols, int32_t C,
                   const uint8_t* d_rung_of_block, int32_t nrungs, const seedq_bases* bases,
                   uint32_t* d_seed, uint8_t* d_exp, int8_t* d_q, float* d_err,
                   void* d_workspace, size_t workspace_bytes, void* hip_stream) {
  const int rc = check_compress_args(d_W, nrows, ncols, C, d_rung_of_block, nrungs, bases, d_seed,
                                     d_exp, d_q);
  if (rc != SEEDQ_OK) return rc;
  if (nrungs > 1) {
    const size_t need = compaction_workspace_bytes(nrows * (ncols / kC), nrungs);
    if (!d_workspace || workspace_bytes < need ||
        (reinterpret_cast<uintptr_t>(d_workspace) & 255u))
      return SEEDQ_EWORKSPACE;
  }
  return run_compress(d_W, nrows, ncols, d_rung_of_block, nrungs, bases, d_seed, d_exp, d_q, d_err,
                      d_workspace, static_cast<hipStream_t>(hip_stream));
}

int seedq_decompress(const uint32_t* d_seed, const uint8_t* d_exp, const int8_t* d_q,
                     const uint8_t* d_rung_of_block, int32_t nrungs, const seedq_rung* rungs,
                     int64_t nrows, int64_t ncols, int32_t C, float* d_W_hat, int32_t* d_acc,
                     void* hip_stream) {
  if (C != kC) return SEEDQ_EUNSUPPORTED;
  if (!d_seed || !d_exp || !d_q || !rungs || !d_W_hat) return SEEDQ_EINVAL;
  if (!shape_ok(nrows, ncols) || nrungs < 1 || nrungs > SEEDQ_MAX_RUNGS) return SEEDQ_EINVAL;
  if (nrungs > 1 && !d_rung_of_block) return SEEDQ_EINVAL;
  if (reinterpret_cast<uintptr_t>(d_q) & 7u || reinterpret_cast<uintptr_t>(d_W_hat) & 15u ||
      reinterpret_cast<uintptr_t>(d_acc) & 15u)
    return SEEDQ_EINVAL;
  RungTable rt;
  std::memset(&rt, 0, sizeof(rt));
  rt.n = nrungs;
  for (int r = 0; r < nrungs; ++r) {
    if (!rung_supported(rungs[r].K, rungs[r].P)) return SEEDQ_EUNSUPPORTED;
    rt.K[r] = rungs[r].K;
    rt.P[r] = rungs[r].P;
  }
  const hipError_t e = launch_decompress(d_seed, d_exp, d_q, nrungs > 1 ? d_rung_of_block : nullptr,
                                         rt, nrows * (ncols / kC), d_W_hat, d_acc,
                                         static_cast<hipStream_t>(hip_stream));
  return e == hipSuccess ? SEEDQ_OK : SEEDQ_EHIP;
}

}  // extern "C"

namespace {

// Rung table of a decoder call; SEEDQ_OK or the error code.
int rung_table(int32_t nrungs, const seedq_rung* rungs, RungTable& rt) {
  if (!rungs || nrungs < 1 || nrungs > SEEDQ_MAX_RUNGS) return SEEDQ_EINVAL;
  std::memset(&rt, 0, sizeof(rt));
  rt.n = nrungs;
  for (int r = 0; r < nrungs; ++r) {
    if (!rung_supported(rungs[r].K, rungs[r].P)) return SEEDQ_EUNSUPPORTED;
    rt.K[r] = rungs[r].K;
    rt.P[r] = rungs[r].P;
  }
  return SEEDQ_OK;
}

// Common checks of the stream calls.
int stream_args(int64_t nrows, int64_t ncols, int32_t C, const void* d_stream, size_t stream_bytes,
                const uint8_t* d_rung, int32_t nrungs, const seedq_rung* rungs, void* d_ws,
                size_t ws_bytes, RungTable& rt) {
  if (C != kC) return SEEDQ_EUNSUPPORTED;
  if (!d_stream || !shape_ok(nrows, ncols)) return SEEDQ_EINVAL;
  if ((reinterpret_cast<uintptr_t>(d_stream) & 3u) || (stream_bytes & 3u)) return SEEDQ_EINVAL;
  const int rc = rung_table(nrungs, rungs, rt);
  if (rc != SEEDQ_OK) return rc;
  if (nrungs > 1 && !d_rung) return SEEDQ_EINVAL;
  if (!d_ws || ws_bytes < stream_workspace_bytes(nrows * (ncols / kC), nrows) ||
      (reinterpret_cast<uintptr_t>(d_ws) & 255u))
    return SEEDQ_EWORKSPACE;
  return SEEDQ_OK;
}

}  // namespace

extern "C" {

int seedq_stream_bytes(int32_t nrungs, const seedq_rung* rungs, const int64_t* count_per_rung,
                       size_t* bytes) {
  if (!count_per_rung || !bytes) return SEEDQ_EINVAL;
  RungTable rt;
  const int rc = rung_table(nrungs, rungs, rt);
  if (rc != SEEDQ_OK) return rc;
  uint64_t bits = 0;
  for (int r = 0; r < nrungs; ++r) {
    if (count_per_rung[r] < 0 || count_per_rung[r] > (int64_t(1) << 40)) return SEEDQ_EINVAL;
    bits += uint64_t(count_per_rung[r]) * uint64_t(rt.K[r] + 4 + 4 * rt.P[r]);
  }
  *bytes = size_t((bits + 31) / 32 * 4);
  return SEEDQ_OK;
}

size_t seedq_stream_workspace_bytes(int64_t nrows, int64_t ncols, int32_t C) {
  if (C != kC || !shape_ok(nrows, ncols)) return 0;
  return stream_workspace_bytes(nrows * (ncols / kC), nrows);
}

int seedq_pack(const uint32_t* d_seed, const uint8_t* d_exp, const int8_t* d_q,
               const uint8_t* d_rung_of_block, int32_t nrungs, const seedq_rung* rungs,
               int64_t nrows, int64_t ncols, int32_t C, uint32_t* d_stream, size_t stream_bytes,
               void* d_workspace, size_t workspace_bytes, void* hip_stream) {
  RungTable rt;
  const int rc = stream_args(nrows, ncols, C, d_stream, stream_bytes, d_rung_of_block, nrungs,
                             rungs, d_workspace, workspace_bytes, rt);
  if (rc != SEEDQ_OK) return rc;
  if (!d_seed || !d_exp || !d_q || (reinterpret_cast<uintptr_t>(d_q) & 7u)) return SEEDQ_EINVAL;
  const hipError_t e = launch_pack(d_seed, d_exp, d_q, nrungs > 1 ? d_rung_of_block : nullptr, rt,
                                   nrows * (ncols / kC), d_stream, int64_t(stream_bytes / 4),
                                   d_workspace, static_cast<hipStream_t>(hip_stream));
  return e == hipSuccess ? SEEDQ_OK : SEEDQ_EHIP;
}

int seedq_unpack(const uint32_t* d_stream, size_t stream_bytes, const uint8_t* d_rung_of_block,
                 int32_t nrungs, const seedq_rung* rungs, int64_t nrows, int64_t ncols, int32_t C,
                 uint32_t* d_seed, uint8_t* d_exp, int8_t* d_q, void* d_workspace,
                 size_t workspace_bytes, void* hip_stream) {
  RungTable rt;
  const int rc = stream_args(nrows, ncols, C, d_stream, stream_bytes, d_rung_of_block, nrungs,
                             rungs, d_workspace, workspace_bytes, rt);
  if (rc != SEEDQ_OK) return rc;
  if (!d_seed || !d_exp || !d_q || (reinterpret_cast<uintptr_t>(d_q) & 7u)) return SEEDQ_EINVAL;
  const hipError_t e = launch_parse(d_stream, int64_t(stream_bytes / 4),
                                    nrungs > 1 ? d_rung_of_block : nullptr, rt,
                                    nrows * (ncols / kC), d_workspace, d_seed, d_exp, d_q, nullptr,
                                    static_cast<hipStream_t>(hip_stream));
  return e == hipSuccess ? SEEDQ_OK : SEEDQ_EHIP;
}

int seedq_decompress_stream(const uint32_t* d_stream, size_t stream_bytes,
                            const uint8_t* d_rung_of_block, int32_t nrungs,
                            const seedq_rung* rungs, int64_t nrows, int64_t ncols, int32_t C,
                            float* d_W_hat, void* d_workspace, size_t workspace_bytes,
                            void* hip_stream) {
  RungTable rt;
  const int rc = stream_args(nrows, ncols, C, d_stream, stream_bytes, d_rung_of_block, nrungs,
                             rungs, d_workspace, workspace_bytes, rt);
  if (rc != SEEDQ_OK) return rc;
  if (!d_W_hat || (reinterpret_cast<uintptr_t>(d_W_hat) & 15u)) return SEEDQ_EINVAL;
  const hipError_t e = launch_parse(d_stream, int64_t(stream_bytes / 4),
                                    nrungs > 1 ? d_rung_of_block : nullptr, rt,
                                    nrows * (ncols / kC), d_workspace, nullptr, nullptr, nullptr,
                                    d_W_hat, static_cast<hipStream_t>(hip_stream));
  return e == hipSuccess ? SEEDQ_OK : SEEDQ_EHIP;
}

int seedq_gemv_stream(const uint32_t* d_stream, size_t stream_bytes, const uint8_t* d_rung_of_block,
                      int32_t nrungs, const seedq_rung* rungs, int64_t nrows, int64_t ncols,
                      int32_t C, int32_t nvec, const float* d_x, float* d_y, void* d_workspace,
                      size_t workspace_bytes, void* hip_stream) {
  RungTable rt;
  const int rc = stream_args(nrows, ncols, C, d_stream, stream_bytes, d_rung_of_block, nrungs,
                             rungs, d_workspace, workspace_bytes, rt);
  if (rc != SEEDQ_OK) return rc;
  if (!(nvec == 1 || nvec == 2 || nvec == 4 || nvec == 8)) return SEEDQ_EINVAL;
  if (!d_x || !d_y || (reinterpret_cast<uintptr_t>(d_x) & 15u) ||
      (reinterpret_cast<uintptr_t>(d_y) & 3u))
    return SEEDQ_EINVAL;
  const hipError_t e = launch_gemv_stream(d_stream, int64_t(stream_bytes / 4),
                                          nrungs > 1 ? d_rung_of_block : nullptr, rt, nrows, ncols,
                                          d_workspace, d_x, ncols, d_y, nrows, nvec,
                                          static_cast<hipStream_t>(hip_stream));
  return e == hipSuccess ? SEEDQ_OK : SEEDQ_EHIP;
}

size_t seedq_footprint_workspace_bytes(void) { return footprint_workspace_bytes(); }

int seedq_footprint(const float* d_clean, const float* d_corrupt, int64_t n, long long* d_count,
                    double* d_sums, void* d_workspace, size_t workspace_bytes, void* hip_stream) {
  if (!d_clean || !d_corrupt || !d_count || !d_sums || n < 0) return SEEDQ_EINVAL;
  if ((reinterpret_cast<uintptr_t>(d_clean) & 15u) || (reinterpret_cast<uintptr_t>(d_corrupt) & 15u) ||
      (reinterpret_cast<uintptr_t>(d_count) & 7u) || (reinterpret_cast<uintptr_t>(d_sums) & 7u))
    return SEEDQ_EINVAL;
  if (!d_workspace || workspace_bytes < footprint_workspace_bytes() ||
      (reinterpret_cast<uintptr_t>(d_workspace) & 255u))
    return SEEDQ_EWORKSPACE;
  const hipError_t e = launch_footprint(d_clean, d_corrupt, n, d_workspace, d_count, d_sums,
                                        static_cast<hipStream_t>(hip_stream));
  return e == hipSuccess ? SEEDQ_OK : SEEDQ_EHIP;
}

int seedq_gauss_hermite(int32_t n, double* x, double* w) { return gauss_hermite(n, x, w); }

size_t seedq_sq_gemv_workspace_bytes(int64_t nrows, int64_t ncols, int32_t transpose) {
  if (nrows <= 0 || ncols <= 0) return 0;
  return sq_gemv_workspace_bytes(nrows, ncols, transpose ? 1 : 0);
}

int seedq_sq_gemv(const float* d_W, int64_t nrows, int64_t ncols, const float* d_v,
                  int32_t transpose, double* d_out, void* d_workspace, size_t workspace_bytes,
                  void* hip_stream) {
  if (!d_W || !d_v || !d_out || nrows <= 0 || ncols <= 0) return SEEDQ_EINVAL;
  if (!transpose && ((ncols & 3) || (reinterpret_cast<uintptr_t>(d_W) & 15u) ||
                     (reinterpret_cast<uintptr_t>(d_v) & 15u)))
    return SEEDQ_EINVAL;
  const size_t need = sq_gemv_workspace_bytes(nrows, ncols, transpose ? 1 : 0);
  if (need && (!d_workspace || workspace_bytes < need ||
               (reinterpret_cast<uintptr_t>(d_workspace) & 255u)))
    return SEEDQ_EWORKSPACE;
  const hipError_t e = launch_sq_gemv(d_W, nrows, ncols, d_v, transpose ? 1 : 0, d_out, d_workspace,
                                      static_cast<hipStream_t>(hip_stream));
  return e == hipSuccess ? SEEDQ_OK : SEEDQ_EHIP;
}

int seedq_column_stats(const float* d_W, int64_t nrows, int64_t ncols, double* d_maxabs,
                       double* d_median, void* hip_stream) {
  if (!d_W || !d_maxabs || !d_median || nrows <= 0 || ncols <= 0) return SEEDQ_EINVAL;
  const hipError_t e = launch_column_stats(d_W, nrows, ncols, d_maxabs, d_median,
                                           static_cast<hipStream_t>(hip_stream));
  return e == hipSuccess ? SEEDQ_OK : SEEDQ_EHIP;
}

int seedq_expect_silu_sq(const double* d_var, int64_t n, int32_t nodes, double* d_out,
                         void* hip_stream) {
  if (!d_var || !d_out || n < 0 || nodes < 1 || nodes > 128) return SEEDQ_EINVAL;
  if (n == 0) return SEEDQ_OK;
  double x[128], w[128];
  const int rc = gauss_hermite(nodes, x, w);
  if (rc != SEEDQ_OK) return rc;
  const hipError_t e = launch_expect_silu_sq(d_var, n, nodes, x, w, nullptr, d_out,
                                             static_cast<hipStream_t>(hip_stream));
  return e == hipSuccess ? SEEDQ_OK : SEEDQ_EHIP;
}

int seedq_gamma_importance(const float* d_gamma, int64_t n, double* d_a, void* hip_stream) {
  if (!d_gamma || !d_a || n < 0) return SEEDQ_EINVAL;
  if (n == 0) return SEEDQ_OK;
  const hipError_t e = launch_gamma_importance(d_gamma, n, d_a, static_cast<hipStream_t>(hip_stream));
  return e == hipSuccess ? SEEDQ_OK : SEEDQ_EHIP;
}

size_t seedq_propagate_workspace_bytes(int64_t nrows, int64_t ncols) {
  if (nrows <= 0 || ncols <= 0) return 0;
  return propagate_workspace_bytes(nrows, ncols);
}

namespace {

int propagate_args(const float* d_W, int64_t nrows, int64_t ncols, const double* d_a_in,
                   const double* d_out, void* d_ws, size_t ws_bytes) {
  if (!d_W || !d_a_in || !d_out || nrows <= 0 || ncols <= 0 || (ncols & 3)) return SEEDQ_EINVAL;
  if (reinterpret_cast<uintptr_t>(d_W) & 15u) return SEEDQ_EINVAL;
  if (!d_ws || ws_bytes < propagate_workspace_bytes(nrows, ncols) ||
      (reinterpret_cast<uintptr_t>(d_ws) & 255u))
    return SEEDQ_EWORKSPACE;
  return SEEDQ_OK;
}

}  // namespace

int seedq_propagate_o(const float* d_Wv, int64_t nrows, int64_t ncols, int32_t n_heads,
                      int32_t n_kv_heads, const double* d_a_in, double* d_a_o, void* d_workspace,
                      size_t workspace_bytes, void* hip_stream) {
  if (n_kv_heads < 1 || n_heads < n_kv_heads || n_heads % n_kv_heads || nrows % n_kv_heads ||
      n_heads / n_kv_heads > 64)
    return SEEDQ_EINVAL;
  const int rc = propagate_args(d_Wv, nrows, ncols, d_a_in, d_a_o, d_workspace, workspace_bytes);
  if (rc != SEEDQ_OK) return rc;
  const hipError_t e = launch_propagate_o(d_Wv, nrows, ncols, n_heads, n_kv_heads, d_a_in, d_a_o,
                                          d_workspace, static_cast<hipStream_t>(hip_stream));
  return e == hipSuccess ? SEEDQ_OK : SEEDQ_EHIP;
}

int seedq_propagate_down(const float* d_Wgate, const float* d_Wup, int64_t nrows, int64_t ncols,
                         const double* d_a_in, int32_t nodes, double* d_a_down, void* d_workspace,
                         size_t workspace_bytes, void* hip_stream) {
  if (!d_Wup || (reinterpret_cast<uintptr_t>(d_Wup) & 15u) || nodes < 1 || nodes > 128)
    return SEEDQ_EINVAL;
  const int rc =
      propagate_args(d_Wgate, nrows, ncols, d_a_in, d_a_down, d_workspace, workspace_bytes);
  if (rc != SEEDQ_OK) return rc;
  double x[128], w[128];
  const int grc = gauss_hermite(nodes, x, w);
  if (grc != SEEDQ_OK) return grc;
  const hipError_t e =
      launch_propagate_down(d_Wgate, d_Wup, nrows, ncols, d_a_in, nodes, x, w, d_a_down,
                            d_workspace, static_cast<hipStream_t>(hip_stream));
  return e == hipSuccess ? SEEDQ_OK : SEEDQ_EHIP;
}

int seedq_channel_order(const float* a, int64_t n, int32_t* perm) {
  if (!a || !perm || n < 0 || n > (int64_t(1) << 31) - 1) return SEEDQ_EINVAL;
  for (int64_t i = 0; i < n; ++i)
    if (!std::isfinite(a[i])) return SEEDQ_EINVAL;   // the sort needs a total order
  channel_order(a, n, perm);
  return SEEDQ_OK;
}

int seedq_permute_columns(const float* d_in, int64_t nrows, int64_t ncols, const int32_t* d_perm,
                          int32_t inverse, float* d_out, void* hip_stream) {
  if (!d_in || !d_out || !d_perm || nrows <= 0 || ncols <= 0 || d_in == d_out) return SEEDQ_EINVAL;
  const hipError_t e = launch_permute_columns(d_in, nrows, ncols, d_perm, inverse ? 1 : 0, d_out,
                                              static_cast<hipStream_t>(hip_stream));
  return e == hipSuccess ? SEEDQ_OK : SEEDQ_EHIP;
}

int seedq_select_outliers(int32_t ntensors, const int64_t* ncols, const double* const* maxabs,
                          const double* const* median, const double* const* a, int32_t keep,
                          int32_t* out_tensor, int32_t* out_col, int32_t* out_count) {
  return select_outliers(ntensors, ncols, maxabs, median, a, keep, out_tensor, out_col, out_count);
}

int seedq_extract_columns(const float* d_W, int64_t nrows, int64_t ncols, int32_t ncol,
                          const int32_t* d_cols, void* d_fp16, void* hip_stream) {
  if (!d_W || nrows <= 0 || ncols <= 0 || ncol < 0 || ncol > 65535) return SEEDQ_EINVAL;
  if (ncol == 0) return SEEDQ_OK;
  if (!d_cols || !d_fp16) return SEEDQ_EINVAL;
  const hipError_t e = launch_columns_fp16(const_cast<float*>(d_W), nrows, ncols, ncol, d_cols,
                                           d_fp16, 0, static_cast<hipStream_t>(hip_stream));
  return e == hipSuccess ? SEEDQ_OK : SEEDQ_EHIP;
}

int seedq_apply_columns(float* d_W, int64_t nrows, int64_t ncols, int32_t ncol,
                        const int32_t* d_cols, const void* d_fp16, void* hip_stream) {
  if (!d_W || nrows <= 0 || ncols <= 0 || ncol < 0 || ncol > 65535) return SEEDQ_EINVAL;
  if (ncol == 0) return SEEDQ_OK;
  if (!d_cols || !d_fp16) return SEEDQ_EINVAL;
  const hipError_t e = launch_columns_fp16(d_W, nrows, ncols, ncol, d_cols,
                                           const_cast<void*>(d_fp16), 1,
                                           static_cast<hipStream_t>(hip_stream));
  return e == hipSuccess ? SEEDQ_OK : SEEDQ_EHIP;
}

}  // extern "C"
