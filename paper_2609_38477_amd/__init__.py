"""Seed-Q per-block LFSR seed search on MI355X (gfx950).

Thin Python binding of libseedq.so (C ABI in ``include/seedq.h``). Every
function of the C ABI has a wrapper of the same name that only marshals
arguments: device buffers are torch tensors on a ROCm device, streams are torch
streams. The compute runs in the library's HIP kernels; there is no fallback,
and every call raises ``SeedqError`` when the library is missing or returns an
error.

Convenience helpers (``build_bases``, ``compress``, ``decompress``,
``plan_schedule``) allocate the outputs and call the wrappers.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libseedq.so")

SEEDQ_OK = 0
SEEDQ_BLOCK = 8
SEEDQ_MAX_RUNGS = 8
SEEDQ_QSTRIDE = 8


class SeedqError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__(f"{where}: {seedq_strerror(code)} ({code})" if _lib is not None
                         else f"{where}: error {code}")


class Rung(ctypes.Structure):
    _fields_ = [("K", ctypes.c_int32), ("P", ctypes.c_int32)]


class ScheduleDesc(ctypes.Structure):
    _fields_ = [("nrows", ctypes.c_int64), ("ncols", ctypes.c_int64), ("C", ctypes.c_int32),
                ("nrungs", ctypes.c_int32), ("rungs", ctypes.POINTER(Rung)),
                ("damage", ctypes.POINTER(ctypes.c_double)), ("target_bpw", ctypes.c_double),
                ("col_importance", ctypes.POINTER(ctypes.c_float)),
                ("row_importance", ctypes.POINTER(ctypes.c_float)),
                ("floor_fraction", ctypes.c_double)]


class ScheduleReport(ctypes.Structure):
    _fields_ = [("lambda_", ctypes.c_double), ("floor_q", ctypes.c_double),
                ("tie_count", ctypes.c_int64), ("total_bits", ctypes.c_int64),
                ("budget_bits", ctypes.c_int64), ("count", ctypes.c_int64 * SEEDQ_MAX_RUNGS),
                ("on_hull", ctypes.c_int32 * SEEDQ_MAX_RUNGS), ("nhull", ctypes.c_int32)]


class BasesRef(ctypes.Structure):
    _fields_ = [("K", ctypes.c_int32), ("P", ctypes.c_int32), ("d_bases", ctypes.c_void_p)]


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded libseedq.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2609_38477_amd.build` (hipcc, gfx950)")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        L.seedq_strerror.restype = ctypes.c_char_p
        L.seedq_strerror.argtypes = [ctypes.c_int]
        L.seedq_plan_schedule.restype = ctypes.c_int
        L.seedq_plan_schedule.argtypes = [ctypes.POINTER(ScheduleDesc), vp,
                                          ctypes.POINTER(ScheduleReport)]
        L.seedq_derive_schedule.restype = ctypes.c_int
        L.seedq_derive_schedule.argtypes = [ctypes.POINTER(ScheduleDesc), ctypes.c_double,
                                            ctypes.c_double, i64, vp]
        L.seedq_bases_bytes.restype = ctypes.c_int
        L.seedq_bases_bytes.argtypes = [i32, i32, i32, ctypes.POINTER(sz)]
        L.seedq_build_bases.restype = ctypes.c_int
        L.seedq_build_bases.argtypes = [i32, i32, i32, vp, vp, vp, vp]
        L.seedq_compress_workspace_bytes.restype = sz
        L.seedq_compress_workspace_bytes.argtypes = [i64, i64, i32, i32]
        L.seedq_compress.restype = ctypes.c_int
        L.seedq_compress.argtypes = [vp, i64, i64, i32, vp, i32, ctypes.POINTER(BasesRef), vp, vp,
                                     vp, vp, vp, sz, vp]
        L.seedq_compress_noalloc.restype = ctypes.c_int
        L.seedq_compress_noalloc.argtypes = [vp, i64, i64, i32, vp, i32, ctypes.POINTER(BasesRef),
                                             vp, vp, vp, vp, vp]
        L.seedq_decompress.restype = ctypes.c_int
        L.seedq_decompress.argtypes = [vp, vp, vp, vp, i32, ctypes.POINTER(Rung), i64, i64, i32,
                                       vp, vp, vp]
        L.seedq_stream_bytes.restype = ctypes.c_int
        L.seedq_stream_bytes.argtypes = [i32, ctypes.POINTER(Rung), vp, ctypes.POINTER(sz)]
        L.seedq_stream_workspace_bytes.restype = sz
        L.seedq_stream_workspace_bytes.argtypes = [i64, i64, i32]
        L.seedq_pack.restype = ctypes.c_int
        L.seedq_pack.argtypes = [vp, vp, vp, vp, i32, ctypes.POINTER(Rung), i64, i64, i32, vp, sz,
                                 vp, sz, vp]
        L.seedq_unpack.restype = ctypes.c_int
        L.seedq_unpack.argtypes = [vp, sz, vp, i32, ctypes.POINTER(Rung), i64, i64, i32, vp, vp, vp,
                                   vp, sz, vp]
        L.seedq_decompress_stream.restype = ctypes.c_int
        L.seedq_decompress_stream.argtypes = [vp, sz, vp, i32, ctypes.POINTER(Rung), i64, i64, i32,
                                              vp, vp, sz, vp]
        L.seedq_gemv_stream.restype = ctypes.c_int
        L.seedq_gemv_stream.argtypes = [vp, sz, vp, i32, ctypes.POINTER(Rung), i64, i64, i32, i32,
                                        vp, vp, vp, sz, vp]
        L.seedq_footprint_workspace_bytes.restype = sz
        L.seedq_footprint_workspace_bytes.argtypes = []
        L.seedq_footprint.restype = ctypes.c_int
        L.seedq_footprint.argtypes = [vp, vp, i64, vp, vp, vp, sz, vp]
        dp = ctypes.POINTER(ctypes.c_double)
        L.seedq_gauss_hermite.restype = ctypes.c_int
        L.seedq_gauss_hermite.argtypes = [i32, vp, vp]
        L.seedq_sq_gemv_workspace_bytes.restype = sz
        L.seedq_sq_gemv_workspace_bytes.argtypes = [i64, i64, i32]
        L.seedq_sq_gemv.restype = ctypes.c_int
        L.seedq_sq_gemv.argtypes = [vp, i64, i64, vp, i32, vp, vp, sz, vp]
        L.seedq_column_stats.restype = ctypes.c_int
        L.seedq_column_stats.argtypes = [vp, i64, i64, vp, vp, vp]
        L.seedq_expect_silu_sq.restype = ctypes.c_int
        L.seedq_expect_silu_sq.argtypes = [vp, i64, i32, vp, vp]
        L.seedq_gamma_importance.restype = ctypes.c_int
        L.seedq_gamma_importance.argtypes = [vp, i64, vp, vp]
        L.seedq_propagate_workspace_bytes.restype = sz
        L.seedq_propagate_workspace_bytes.argtypes = [i64, i64]
        L.seedq_propagate_o.restype = ctypes.c_int
        L.seedq_propagate_o.argtypes = [vp, i64, i64, i32, i32, vp, vp, vp, sz, vp]
        L.seedq_propagate_down.restype = ctypes.c_int
        L.seedq_propagate_down.argtypes = [vp, vp, i64, i64, vp, i32, vp, vp, sz, vp]
        L.seedq_channel_order.restype = ctypes.c_int
        L.seedq_channel_order.argtypes = [vp, i64, vp]
        L.seedq_permute_columns.restype = ctypes.c_int
        L.seedq_permute_columns.argtypes = [vp, i64, i64, vp, i32, vp, vp]
        L.seedq_select_outliers.restype = ctypes.c_int
        L.seedq_select_outliers.argtypes = [i32, vp, ctypes.POINTER(dp), ctypes.POINTER(dp),
                                            ctypes.POINTER(dp), i32, vp, vp,
                                            ctypes.POINTER(ctypes.c_int32)]
        L.seedq_extract_columns.restype = ctypes.c_int
        L.seedq_extract_columns.argtypes = [vp, i64, i64, i32, vp, vp, vp]
        L.seedq_apply_columns.restype = ctypes.c_int
        L.seedq_apply_columns.argtypes = [vp, i64, i64, i32, vp, vp, vp]
        _lib = L
    return _lib


def _ptr(t) -> int | None:
    """Device (or host numpy) pointer of a buffer, None for None."""
    if t is None:
        return None
    if isinstance(t, np.ndarray):
        return t.ctypes.data
    return t.data_ptr()


def _stream(stream) -> int | None:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


def _check(rc: int, where: str) -> None:
    if rc != SEEDQ_OK:
        raise SeedqError(rc, where)


# ---------------------------------------------------------------- C ABI wrappers

def seedq_strerror(code: int) -> str:
    return lib().seedq_strerror(code).decode()


def seedq_plan_schedule(desc: ScheduleDesc, rung_of_block: np.ndarray,
                        report: ScheduleReport | None = None) -> None:
    assert rung_of_block.dtype == np.uint8 and rung_of_block.flags.c_contiguous
    rc = lib().seedq_plan_schedule(ctypes.byref(desc), rung_of_block.ctypes.data,
                                   ctypes.byref(report) if report is not None else None)
    _check(rc, "seedq_plan_schedule")


def seedq_derive_schedule(desc: ScheduleDesc, lam: float, floor_q: float, tie_count: int,
                          rung_of_block: np.ndarray) -> None:
    assert rung_of_block.dtype == np.uint8 and rung_of_block.flags.c_contiguous
    rc = lib().seedq_derive_schedule(ctypes.byref(desc), float(lam), float(floor_q),
                                     int(tie_count), rung_of_block.ctypes.data)
    _check(rc, "seedq_derive_schedule")


def seedq_bases_bytes(K: int, P: int, C: int = SEEDQ_BLOCK) -> int:
    out = ctypes.c_size_t(0)
    _check(lib().seedq_bases_bytes(K, P, C, ctypes.byref(out)), "seedq_bases_bytes")
    return int(out.value)


def seedq_build_bases(K: int, P: int, C: int, d_bases, d_U=None, d_pinv=None, stream=None) -> None:
    rc = lib().seedq_build_bases(K, P, C, _ptr(d_bases), _ptr(d_U), _ptr(d_pinv), _stream(stream))
    _check(rc, "seedq_build_bases")


def seedq_compress_workspace_bytes(nrows: int, ncols: int, C: int, nrungs: int) -> int:
    return int(lib().seedq_compress_workspace_bytes(nrows, ncols, C, nrungs))


def seedq_compress(d_W, nrows: int, ncols: int, C: int, d_rung_of_block, bases: list,
                   d_seed, d_exp, d_q, d_err, d_workspace, workspace_bytes: int,
                   stream=None) -> None:
    arr = (BasesRef * len(bases))(*[BasesRef(b.K, b.P, _ptr(b.buffer)) for b in bases])
    rc = lib().seedq_compress(_ptr(d_W), nrows, ncols, C, _ptr(d_rung_of_block), len(bases), arr,
                              _ptr(d_seed), _ptr(d_exp), _ptr(d_q), _ptr(d_err),
                              _ptr(d_workspace), workspace_bytes, _stream(stream))
    _check(rc, "seedq_compress")


def seedq_compress_noalloc(d_W, nrows: int, ncols: int, C: int, d_rung_of_block, bases: list,
                           d_seed, d_exp, d_q, d_err, stream=None) -> None:
    arr = (BasesRef * len(bases))(*[BasesRef(b.K, b.P, _ptr(b.buffer)) for b in bases])
    rc = lib().seedq_compress_noalloc(_ptr(d_W), nrows, ncols, C, _ptr(d_rung_of_block), len(bases),
                                      arr, _ptr(d_seed), _ptr(d_exp), _ptr(d_q), _ptr(d_err),
                                      _stream(stream))
    _check(rc, "seedq_compress_noalloc")


def seedq_decompress(d_seed, d_exp, d_q, d_rung_of_block, rungs, nrows: int, ncols: int, C: int,
                     d_W_hat, d_acc=None, stream=None) -> None:
    arr = (Rung * len(rungs))(*[Rung(int(K), int(P)) for K, P in rungs])
    rc = lib().seedq_decompress(_ptr(d_seed), _ptr(d_exp), _ptr(d_q), _ptr(d_rung_of_block),
                                len(rungs), arr, nrows, ncols, C, _ptr(d_W_hat), _ptr(d_acc),
                                _stream(stream))
    _check(rc, "seedq_decompress")


def _rungs(rungs):
    return (Rung * len(rungs))(*[Rung(int(K), int(P)) for K, P in rungs])


def seedq_stream_bytes(rungs, count_per_rung) -> int:
    cnt = np.ascontiguousarray(count_per_rung, dtype=np.int64)
    out = ctypes.c_size_t(0)
    _check(lib().seedq_stream_bytes(len(rungs), _rungs(rungs), cnt.ctypes.data, ctypes.byref(out)),
           "seedq_stream_bytes")
    return int(out.value)


def seedq_stream_workspace_bytes(nrows: int, ncols: int, C: int = SEEDQ_BLOCK) -> int:
    return int(lib().seedq_stream_workspace_bytes(nrows, ncols, C))


def seedq_pack(d_seed, d_exp, d_q, d_rung_of_block, rungs, nrows: int, ncols: int, C: int,
               d_stream, stream_bytes: int, d_workspace, workspace_bytes: int, stream=None) -> None:
    rc = lib().seedq_pack(_ptr(d_seed), _ptr(d_exp), _ptr(d_q), _ptr(d_rung_of_block), len(rungs),
                          _rungs(rungs), nrows, ncols, C, _ptr(d_stream), stream_bytes,
                          _ptr(d_workspace), workspace_bytes, _stream(stream))
    _check(rc, "seedq_pack")


def seedq_unpack(d_stream, stream_bytes: int, d_rung_of_block, rungs, nrows: int, ncols: int,
                 C: int, d_seed, d_exp, d_q, d_workspace, workspace_bytes: int, stream=None) -> None:
    rc = lib().seedq_unpack(_ptr(d_stream), stream_bytes, _ptr(d_rung_of_block), len(rungs),
                            _rungs(rungs), nrows, ncols, C, _ptr(d_seed), _ptr(d_exp), _ptr(d_q),
                            _ptr(d_workspace), workspace_bytes, _stream(stream))
    _check(rc, "seedq_unpack")


def seedq_decompress_stream(d_stream, stream_bytes: int, d_rung_of_block, rungs, nrows: int,
                            ncols: int, C: int, d_W_hat, d_workspace, workspace_bytes: int,
                            stream=None) -> None:
    rc = lib().seedq_decompress_stream(_ptr(d_stream), stream_bytes, _ptr(d_rung_of_block),
                                       len(rungs), _rungs(rungs), nrows, ncols, C, _ptr(d_W_hat),
                                       _ptr(d_workspace), workspace_bytes, _stream(stream))
    _check(rc, "seedq_decompress_stream")


def seedq_gemv_stream(d_stream, stream_bytes: int, d_rung_of_block, rungs, nrows: int, ncols: int,
                      C: int, nvec: int, d_x, d_y, d_workspace, workspace_bytes: int,
                      stream=None) -> None:
    rc = lib().seedq_gemv_stream(_ptr(d_stream), stream_bytes, _ptr(d_rung_of_block), len(rungs),
                                 _rungs(rungs), nrows, ncols, C, nvec, _ptr(d_x), _ptr(d_y),
                                 _ptr(d_workspace), workspace_bytes, _stream(stream))
    _check(rc, "seedq_gemv_stream")


def seedq_footprint_workspace_bytes() -> int:
    return int(lib().seedq_footprint_workspace_bytes())


def seedq_footprint(d_clean, d_corrupt, n: int, d_count, d_sums, d_workspace, workspace_bytes: int,
                    stream=None) -> None:
    rc = lib().seedq_footprint(_ptr(d_clean), _ptr(d_corrupt), n, _ptr(d_count), _ptr(d_sums),
                               _ptr(d_workspace), workspace_bytes, _stream(stream))
    _check(rc, "seedq_footprint")


def seedq_gauss_hermite(n: int):
    x = np.empty(n, dtype=np.float64)
    w = np.empty(n, dtype=np.float64)
    _check(lib().seedq_gauss_hermite(n, x.ctypes.data, w.ctypes.data), "seedq_gauss_hermite")
    return x, w


def seedq_sq_gemv_workspace_bytes(nrows: int, ncols: int, transpose: int) -> int:
    return int(lib().seedq_sq_gemv_workspace_bytes(nrows, ncols, int(transpose)))


def seedq_sq_gemv(d_W, nrows: int, ncols: int, d_v, transpose: int, d_out, d_workspace=None,
                  workspace_bytes: int = 0, stream=None) -> None:
    rc = lib().seedq_sq_gemv(_ptr(d_W), nrows, ncols, _ptr(d_v), int(transpose), _ptr(d_out),
                             _ptr(d_workspace), workspace_bytes, _stream(stream))
    _check(rc, "seedq_sq_gemv")


def seedq_column_stats(d_W, nrows: int, ncols: int, d_maxabs, d_median, stream=None) -> None:
    _check(lib().seedq_column_stats(_ptr(d_W), nrows, ncols, _ptr(d_maxabs), _ptr(d_median),
                                    _stream(stream)), "seedq_column_stats")


def seedq_expect_silu_sq(d_var, n: int, nodes: int, d_out, stream=None) -> None:
    _check(lib().seedq_expect_silu_sq(_ptr(d_var), n, nodes, _ptr(d_out), _stream(stream)),
           "seedq_expect_silu_sq")


def seedq_gamma_importance(d_gamma, n: int, d_a, stream=None) -> None:
    _check(lib().seedq_gamma_importance(_ptr(d_gamma), n, _ptr(d_a), _stream(stream)),
           "seedq_gamma_importance")


def seedq_propagate_workspace_bytes(nrows: int, ncols: int) -> int:
    return int(lib().seedq_propagate_workspace_bytes(nrows, ncols))


def seedq_propagate_o(d_Wv, nrows: int, ncols: int, n_heads: int, n_kv_heads: int, d_a_in, d_a_o,
                      d_workspace, workspace_bytes: int, stream=None) -> None:
    _check(lib().seedq_propagate_o(_ptr(d_Wv), nrows, ncols, n_heads, n_kv_heads, _ptr(d_a_in),
                                   _ptr(d_a_o), _ptr(d_workspace), workspace_bytes,
                                   _stream(stream)), "seedq_propagate_o")


def seedq_propagate_down(d_Wgate, d_Wup, nrows: int, ncols: int, d_a_in, nodes: int, d_a_down,
                         d_workspace, workspace_bytes: int, stream=None) -> None:
    _check(lib().seedq_propagate_down(_ptr(d_Wgate), _ptr(d_Wup), nrows, ncols, _ptr(d_a_in), nodes,
                                      _ptr(d_a_down), _ptr(d_workspace), workspace_bytes,
                                      _stream(stream)), "seedq_propagate_down")


def seedq_channel_order(a) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.float32)
    perm = np.empty(a.size, dtype=np.int32)
    _check(lib().seedq_channel_order(a.ctypes.data, a.size, perm.ctypes.data), "seedq_channel_order")
    return perm


def seedq_permute_columns(d_in, nrows: int, ncols: int, d_perm, inverse: int, d_out,
                          stream=None) -> None:
    _check(lib().seedq_permute_columns(_ptr(d_in), nrows, ncols, _ptr(d_perm), int(inverse),
                                       _ptr(d_out), _stream(stream)), "seedq_permute_columns")


def seedq_select_outliers(maxabs_list, median_list, a_list, keep: int = 4):
    """[(tensor, column)] of the kept outlier columns (host numpy fp64 inputs)."""
    T = len(maxabs_list)
    mx = [np.ascontiguousarray(m, dtype=np.float64) for m in maxabs_list]
    md = [np.ascontiguousarray(m, dtype=np.float64) for m in median_list]
    aa = [np.ascontiguousarray(m, dtype=np.float64) for m in a_list]
    ncols = np.array([m.size for m in mx], dtype=np.int64)
    dp = ctypes.POINTER(ctypes.c_double)
    arr = lambda lst: (dp * max(T, 1))(*[m.ctypes.data_as(dp) for m in lst])
    ot = np.empty(max(keep, 1), dtype=np.int32)
    oc = np.empty(max(keep, 1), dtype=np.int32)
    cnt = ctypes.c_int32(0)
    rc = lib().seedq_select_outliers(T, ncols.ctypes.data, arr(mx), arr(md), arr(aa), keep,
                                     ot.ctypes.data, oc.ctypes.data, ctypes.byref(cnt))
    _check(rc, "seedq_select_outliers")
    return [(int(ot[i]), int(oc[i])) for i in range(cnt.value)]


def seedq_extract_columns(d_W, nrows: int, ncols: int, ncol: int, d_cols, d_fp16,
                          stream=None) -> None:
    _check(lib().seedq_extract_columns(_ptr(d_W), nrows, ncols, ncol, _ptr(d_cols), _ptr(d_fp16),
                                       _stream(stream)), "seedq_extract_columns")


def seedq_apply_columns(d_W, nrows: int, ncols: int, ncol: int, d_cols, d_fp16,
                        stream=None) -> None:
    _check(lib().seedq_apply_columns(_ptr(d_W), nrows, ncols, ncol, _ptr(d_cols), _ptr(d_fp16),
                                     _stream(stream)), "seedq_apply_columns")


# ---------------------------------------------------------------- helpers

@dataclass
class Bases:
    """A built basis stack for rung (K, P) and its optional verification outputs."""
    K: int
    P: int
    buffer: object            # torch uint8 device tensor (opaque)
    U: object = None          # int32 [2^K-1, P, 8] or None
    pinv: object = None       # fp32 [P, 2^K-1, 8] or None


def _schedule_desc(nrows, ncols, rungs, damage, target_bpw, col_importance, row_importance,
                   floor_fraction):
    """A ScheduleDesc and the arrays it points into (keep them alive while it is used)."""
    rungs = [tuple(int(v) for v in r) for r in rungs]
    R = len(rungs)
    rung_arr = (Rung * R)(*[Rung(K, P) for K, P in rungs])
    dmg_np = None if damage is None else np.ascontiguousarray(damage, dtype=np.float64)
    a = np.ascontiguousarray(col_importance, dtype=np.float32)
    rho = None if row_importance is None else np.ascontiguousarray(row_importance, dtype=np.float32)
    desc = ScheduleDesc(nrows, ncols, SEEDQ_BLOCK, R, rung_arr,
                        None if dmg_np is None else dmg_np.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                        float(target_bpw), a.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
                        None if rho is None else rho.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
                        float(floor_fraction))
    return desc, (rung_arr, dmg_np, a, rho)


def derive_schedule(nrows: int, ncols: int, rungs, damage, col_importance, lam: float,
                    floor_q: float, tie_count: int, row_importance=None,
                    out: np.ndarray | None = None) -> np.ndarray:
    """Decoder-side rung index per block from the stored lambda, floor value and
    tie count (numpy uint8 [nblocks])."""
    desc, keep = _schedule_desc(nrows, ncols, rungs, damage, 0.0, col_importance, row_importance,
                                0.0)
    if out is None:
        out = np.empty(nrows * (ncols // SEEDQ_BLOCK), dtype=np.uint8)
    seedq_derive_schedule(desc, lam, floor_q, tie_count, out)
    del keep
    return out


def plan_schedule(nrows: int, ncols: int, rungs, damage, target_bpw: float, col_importance,
                  row_importance=None, floor_fraction: float = 0.06, out: np.ndarray | None = None):
    """Rung index per block (numpy uint8 [nblocks], written into ``out`` when
    given) and the report as a dict."""
    R = len(rungs)
    desc, keep = _schedule_desc(nrows, ncols, rungs, damage, target_bpw, col_importance,
                                row_importance, floor_fraction)
    if out is None:
        out = np.empty(nrows * (ncols // SEEDQ_BLOCK), dtype=np.uint8)
    rep = ScheduleReport()
    seedq_plan_schedule(desc, out, rep)
    report = dict(lam=rep.lambda_, floor_q=rep.floor_q, tie_count=rep.tie_count,
                  total_bits=rep.total_bits, budget_bits=rep.budget_bits,
                  count=list(rep.count)[:R], on_hull=list(rep.on_hull)[:R], nhull=rep.nhull)
    return out, report


def build_bases(K: int, P: int, with_U: bool = False, with_pinv: bool = False, device="cuda",
                stream=None) -> Bases:
    import torch
    nbytes = seedq_bases_bytes(K, P)
    buf = torch.empty(nbytes, dtype=torch.uint8, device=device)
    S = (1 << K) - 1
    U = torch.empty((S, P, SEEDQ_BLOCK), dtype=torch.int32, device=device) if with_U else None
    pinv = torch.empty((P, S, SEEDQ_BLOCK), dtype=torch.float32, device=device) if with_pinv else None
    seedq_build_bases(K, P, SEEDQ_BLOCK, buf, U, pinv, stream)
    return Bases(K, P, buf, U, pinv)


def compress(W, bases: list, rung_of_block=None, with_err: bool = True, stream=None):
    """Seed search for every block of W (torch fp32 [nrows, ncols] on the GPU).
    Returns (seed uint32->int64 view as torch.int32, exp uint8, q int8 [nb, 8], err fp32)."""
    import torch
    nrows, ncols = W.shape
    nb = nrows * ncols // SEEDQ_BLOCK
    dev = W.device
    seed = torch.empty(nb, dtype=torch.int32, device=dev)
    exp = torch.empty(nb, dtype=torch.uint8, device=dev)
    q = torch.empty((nb, SEEDQ_QSTRIDE), dtype=torch.int8, device=dev)
    err = torch.empty(nb, dtype=torch.float32, device=dev) if with_err else None
    nws = seedq_compress_workspace_bytes(nrows, ncols, SEEDQ_BLOCK, len(bases))
    ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=dev) if nws else None
    seedq_compress(W, nrows, ncols, SEEDQ_BLOCK, rung_of_block, bases, seed, exp, q, err, ws, nws,
                   stream)
    return seed, exp, q, err


def compress_row_tiles(W_host, bases: list, rung_of_block=None, row_tiles: int = 8,
                       with_err: bool = True):
    """Seed search of a matrix that stays in host memory, streamed through the
    GPU in ``row_tiles`` contiguous row ranges (blocks are independent once the
    rungs are planned, so every tile is one seedq_compress call on its rows and
    their slice of the rung array). W_host: torch fp32 [nrows, ncols] on the
    host, pinned for asynchronous copies. Two tile buffers alternate, each with
    its own compute stream (the current one and a second) and workspace: the
    copy of the next tile (on a copy stream) overlaps the search of this one,
    and consecutive searches overlap each other's tails. Outputs as
    ``compress`` (device tensors), complete on the current stream; only two
    tiles of W are ever resident in device memory."""
    import torch
    nrows, ncols = W_host.shape
    G = ncols // SEEDQ_BLOCK
    nb = nrows * G
    dev = torch.device("cuda", torch.cuda.current_device())
    seed = torch.empty(nb, dtype=torch.int32, device=dev)
    exp = torch.empty(nb, dtype=torch.uint8, device=dev)
    q = torch.empty((nb, SEEDQ_QSTRIDE), dtype=torch.int8, device=dev)
    err = torch.empty(nb, dtype=torch.float32, device=dev) if with_err else None
    bounds = [nrows * t // row_tiles for t in range(row_tiles + 1)]
    rows_max = max(bounds[t + 1] - bounds[t] for t in range(row_tiles))
    bufs = [torch.empty((rows_max, ncols), dtype=torch.float32, device=dev) for _ in range(2)]
    nws = seedq_compress_workspace_bytes(rows_max, ncols, SEEDQ_BLOCK, len(bases))
    wss = [torch.empty(max(nws, 256), dtype=torch.uint8, device=dev) if nws else None
           for _ in range(2)]
    current = torch.cuda.current_stream()
    computes = [current, torch.cuda.Stream(device=dev)]
    copy = torch.cuda.Stream(device=dev)
    copied = [torch.cuda.Event() for _ in range(2)]
    searched = [torch.cuda.Event() for _ in range(2)]
    # the buffers come from the current stream's pool, whose pending work may
    # still read the memory they reuse, and the rung array may still be being
    # written there: the other streams start after that work
    copy.wait_stream(current)
    computes[1].wait_stream(current)

    def upload(t):
        r0, r1 = bounds[t], bounds[t + 1]
        k = t % 2
        if t >= 2:
            copy.wait_event(searched[k])     # the buffer's previous tile is done
        with torch.cuda.stream(copy):
            bufs[k][: r1 - r0].copy_(W_host[r0:r1], non_blocking=True)
            copied[k].record(copy)

    upload(0)
    for t in range(row_tiles):
        r0, r1 = bounds[t], bounds[t + 1]
        if t + 1 < row_tiles:
            upload(t + 1)
        k = t % 2
        cs = computes[k]   # buffer k, workspace k and stream k go together
        cs.wait_event(copied[k])
        if r1 > r0:
            b0, b1 = r0 * G, r1 * G
            seedq_compress(bufs[k][: r1 - r0], r1 - r0, ncols, SEEDQ_BLOCK,
                           None if rung_of_block is None else rung_of_block[b0:b1], bases,
                           seed[b0:b1], exp[b0:b1], q[b0:b1], None if err is None else err[b0:b1],
                           wss[k], nws, cs)
        searched[k].record(cs)
    # everything after this call on the current stream (and the allocator's
    # reuse of the buffers) comes after the second stream's searches
    current.wait_stream(computes[1])
    return seed, exp, q, err


def decompress(seed, exp, q, rungs, nrows: int, ncols: int, rung_of_block=None,
               with_acc: bool = False, stream=None):
    import torch
    dev = seed.device
    W_hat = torch.empty((nrows, ncols), dtype=torch.float32, device=dev)
    acc = torch.empty((nrows, ncols), dtype=torch.int32, device=dev) if with_acc else None
    seedq_decompress(seed, exp, q, rung_of_block, rungs, nrows, ncols, SEEDQ_BLOCK, W_hat, acc,
                     stream)
    return W_hat, acc


def _stream_ws(nrows, ncols, dev):
    import torch
    n = seedq_stream_workspace_bytes(nrows, ncols)
    return torch.empty(max(n, 256), dtype=torch.uint8, device=dev), n


def pack(seed, exp, q, rungs, nrows: int, ncols: int, rung_of_block=None, count_per_rung=None,
         stream=None):
    """Payload words (torch uint32-as-int32 tensor) of the codes. The length comes
    from count_per_rung (blocks per rung), by default every block at rungs[0]."""
    import torch
    nb = nrows * ncols // SEEDQ_BLOCK
    if count_per_rung is None:
        assert len(rungs) == 1
        count_per_rung = [nb]
    nbytes = seedq_stream_bytes(rungs, count_per_rung)
    dev = seed.device
    words = torch.empty(max(nbytes // 4, 1), dtype=torch.int32, device=dev)
    ws, nws = _stream_ws(nrows, ncols, dev)
    seedq_pack(seed, exp, q, rung_of_block, rungs, nrows, ncols, SEEDQ_BLOCK, words, nbytes, ws, nws,
               stream)
    return words[: nbytes // 4]


def unpack(words, rungs, nrows: int, ncols: int, rung_of_block=None, stream=None):
    import torch
    nb = nrows * ncols // SEEDQ_BLOCK
    dev = words.device
    seed = torch.empty(nb, dtype=torch.int32, device=dev)
    exp = torch.empty(nb, dtype=torch.uint8, device=dev)
    q = torch.empty((nb, SEEDQ_QSTRIDE), dtype=torch.int8, device=dev)
    ws, nws = _stream_ws(nrows, ncols, dev)
    seedq_unpack(words, words.numel() * 4, rung_of_block, rungs, nrows, ncols, SEEDQ_BLOCK, seed,
                 exp, q, ws, nws, stream)
    return seed, exp, q


def decompress_stream(words, rungs, nrows: int, ncols: int, rung_of_block=None, stream=None):
    import torch
    dev = words.device
    W_hat = torch.empty((nrows, ncols), dtype=torch.float32, device=dev)
    ws, nws = _stream_ws(nrows, ncols, dev)
    seedq_decompress_stream(words, words.numel() * 4, rung_of_block, rungs, nrows, ncols,
                            SEEDQ_BLOCK, W_hat, ws, nws, stream)
    return W_hat


def gemv_stream(words, rungs, nrows: int, ncols: int, x, rung_of_block=None, stream=None):
    """y = W_hat x with W_hat decoded from the stream; x is fp32 [nvec, ncols]
    (or [ncols]) on the GPU, nvec in {1, 2, 4, 8}; returns y [nvec, nrows] (or [nrows])."""
    import torch
    squeeze = x.dim() == 1
    xx = x.reshape(-1, ncols).contiguous()
    y = torch.empty((xx.shape[0], nrows), dtype=torch.float32, device=x.device)
    ws, nws = _stream_ws(nrows, ncols, x.device)
    seedq_gemv_stream(words, words.numel() * 4, rung_of_block, rungs, nrows, ncols, SEEDQ_BLOCK,
                      xx.shape[0], xx, y, ws, nws, stream)
    return y[0] if squeeze else y


def footprint(clean, corrupt, stream=None):
    """(N_flip, p_flip, eta) of eq. (security_metrics) for two fp32 GPU tensors."""
    import torch
    n = clean.numel()
    cnt = torch.zeros(1, dtype=torch.int64, device=clean.device)
    sums = torch.zeros(2, dtype=torch.float64, device=clean.device)
    nws = seedq_footprint_workspace_bytes()
    ws = torch.empty(nws, dtype=torch.uint8, device=clean.device)
    seedq_footprint(clean.contiguous(), corrupt.contiguous(), n, cnt, sums, ws, nws, stream)
    c = int(cnt.item())
    s = sums.cpu().numpy()
    return c, c / n, float(np.sqrt(s[0] / s[1])) if s[1] > 0 else float("nan")
