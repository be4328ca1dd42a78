"""Seed-Q CPU oracle: test infrastructure only.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package. The product (``paper_2609_38477_amd``)
never imports it and shares no code with it.

Everything here is the plain, slow definition of what the Seed-Q encoder
computes for one weight matrix, in fp64:

* ``states`` / ``basis_int``: the LFSR basis U(s) of section 3.1, eq. (codec)
  (a full-period S-bit LFSR whose initial state is the seed s; per the hardware
  appendix its states are centred and its taps depend on the width). Reading: Galois
  right-shift LFSR with the mask table in ``seedq_oracle.c``, column j of U holds
  the centred states x_{8j}..x_{8j+7}, U = U_int * 2^-(K-1).
* ``pinv_stack``: per-seed Moore-Penrose pseudo-inverse of U(s) (LAPACK SVD via
  numpy, singular values at or below 2^-30 of the largest count as zero), so
  ``pinv @ w`` is the minimum-norm least-squares coefficient vector t* of
  section 3.1.
* ``quantize``: P signed 4-bit mantissas under one shared 4-bit exponent
  (section 3.1, m = e = 4), by its definition (loop over the exponent).
* ``code_error``: ||w - U(s) q 2^-e||^2 with exact integer reconstruction.
* ``search`` (C, OpenMP) and ``search_numpy`` (vectorised numpy): the
  exhaustive search of section 3.1 over all 2^K - 1 seeds, ties to the smallest
  seed. Per the appendix on cost (section A.8) the encoder's time goes into
  this search, one least-squares fit for every seed of every block.
* ``decompress``: w_hat = U(s) t_hat (Algorithm 2), exact.
* ``schedule``: the allocation of sections 3.2-3.4 (eq. (objective), (imp),
  the floor, eq. (ladder), Everett bisection and the tie pass of Algorithm 1).

* ``stream`` (submodule): the headerless variable-length code stream of
  Algorithm 1's emit step, bit by bit, and the fault footprint metrics of
  eq. (security_metrics).

* ``importance`` (submodule): the data-free importance front end (eq. (gamma),
  eq. (prop), the backward rho, the channel sort and the outlier-column rule).

Parity pins for each function live in ``tests/test_oracle_*.py``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

C = 8
HERE = os.path.dirname(os.path.abspath(__file__))
# SEEDQ_ORACLE_LIB points the loader at another build of the C half (the
# mutation tests use it to run the pins against copies with planted mistakes).
LIB_PATH = os.environ.get("SEEDQ_ORACLE_LIB") or os.path.join(HERE, "liboq.so")
SRC_PATH = os.path.join(HERE, "seedq_oracle.c")

# Numerical rank rule for the pseudo-inverse: singular values at or below
# RANK_RTOL times the largest are treated as zero.
RANK_RTOL = 2.0 ** -30


def build(force: bool = True) -> str:
    """Compile the C half of the oracle into oracle/liboq.so."""
    if not force and os.path.exists(LIB_PATH) and \
            os.path.getmtime(LIB_PATH) >= os.path.getmtime(SRC_PATH):
        return LIB_PATH
    tmp = LIB_PATH + ".tmp"
    cmd = ["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math", "-shared", "-fPIC",
           SRC_PATH, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build()
        L = ctypes.CDLL(LIB_PATH)
        L.oq_lfsr_mask.restype = ctypes.c_uint32
        L.oq_lfsr_mask.argtypes = [ctypes.c_int]
        L.oq_period.restype = ctypes.c_uint64
        L.oq_period.argtypes = [ctypes.c_int]
        L.oq_states.restype = ctypes.c_int
        L.oq_states.argtypes = [ctypes.c_int, ctypes.c_uint32, ctypes.c_int, ctypes.c_void_p]
        L.oq_quantize.restype = None
        L.oq_quantize.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
        L.oq_code_error.restype = ctypes.c_int
        L.oq_code_error.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_uint32,
                                    ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
        L.oq_search.restype = ctypes.c_int
        L.oq_search.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_int,
                                ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p,
                                ctypes.c_void_p, ctypes.c_void_p]
        L.oq_decompress.restype = ctypes.c_int
        L.oq_decompress.argtypes = [ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                    ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p,
                                    ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        _lib = L
    return _lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


# ---------------------------------------------------------------- LFSR basis

def lfsr_mask(K: int) -> int:
    return int(lib().oq_lfsr_mask(K))


def period(K: int) -> int:
    """Steps for the state started at 1 to return to 1."""
    return int(lib().oq_period(K))


def states(K: int, seed: int, n: int) -> np.ndarray:
    """Centred LFSR states u_0..u_{n-1} (int64), x_0 = seed."""
    out = np.empty(n, dtype=np.int32)
    if lib().oq_states(K, seed, n, _p(out)) != 0:
        raise ValueError(f"bad LFSR width {K} or seed {seed}")
    return out.astype(np.int64)


def states_all(K: int, n: int) -> np.ndarray:
    """(2^K - 1) x n centred states for every seed 1..2^K-1 (row s-1)."""
    S = (1 << K) - 1
    mask = lfsr_mask(K)
    x = np.arange(1, S + 1, dtype=np.int64)
    out = np.empty((S, n), dtype=np.int64)
    for i in range(n):
        out[:, i] = x
        x = (x >> 1) ^ np.where(x & 1, mask, 0)
    return out - (1 << (K - 1))


def basis_int(K: int, P: int, seed: int) -> np.ndarray:
    """U_int(s) as an 8 x P int64 matrix (column j = states 8j..8j+7)."""
    return states(K, seed, C * P).reshape(P, C).T.copy()


def basis_int_all(K: int, P: int) -> np.ndarray:
    """(2^K - 1) x 8 x P int64 stack of U_int(s)."""
    st = states_all(K, C * P)
    return st.reshape(-1, P, C).transpose(0, 2, 1).copy()


def basis(K: int, P: int, seed: int) -> np.ndarray:
    """U(s) = U_int(s) * 2^-(K-1), entries in [-1, 1)."""
    return basis_int(K, P, seed).astype(np.float64) * 2.0 ** -(K - 1)


# ---------------------------------------------------------------- least squares

def pinv_of(U: np.ndarray) -> np.ndarray:
    """Moore-Penrose pseudo-inverse (LAPACK SVD) with the rank rule above.
    Accepts one matrix or a stack."""
    return np.linalg.pinv(U, rcond=RANK_RTOL)


def pinv_stack(K: int, P: int, chunk: int = 1 << 16) -> np.ndarray:
    """(2^K - 1) x P x 8 fp64 stack: pinv(U(s)) for s = 1..2^K-1."""
    Ui = basis_int_all(K, P)
    out = np.empty((Ui.shape[0], P, C), dtype=np.float64)
    for s in range(0, Ui.shape[0], chunk):
        U = Ui[s:s + chunk].astype(np.float64) * 2.0 ** -(K - 1)
        out[s:s + chunk] = pinv_of(U)
    return out


def ls_solve(U: np.ndarray, w: np.ndarray) -> np.ndarray:
    """Minimum-norm least-squares coefficients t* = argmin ||w - U t||."""
    return pinv_of(U) @ np.asarray(w, dtype=np.float64)


def rank_of(U: np.ndarray) -> int:
    s = np.linalg.svd(U, compute_uv=False)
    return int((s > RANK_RTOL * s[0]).sum()) if s[0] > 0 else 0


# ---------------------------------------------------------------- quantiser

def quantize(t) -> tuple[int, np.ndarray]:
    """(e, q) for coefficients t, via the C definition."""
    t = np.ascontiguousarray(t, dtype=np.float64)
    q = np.empty(t.shape[0], dtype=np.int32)
    e = np.zeros(1, dtype=np.int32)
    lib().oq_quantize(_p(t), t.shape[0], _p(e), _p(q))
    return int(e[0]), q.astype(np.int64)


def quantize_numpy(t: np.ndarray) -> tuple[np.ndarray, np.ndarray]:
    """Vectorised quantiser over the last axis (same definition)."""
    t = np.asarray(t, dtype=np.float64)
    e = np.zeros(t.shape[:-1], dtype=np.int64)
    found = np.zeros(t.shape[:-1], dtype=bool)
    for ee in range(15, -1, -1):
        r = np.rint(np.ldexp(t, ee))
        fits = ((r <= 7) & (r >= -8)).all(axis=-1) & ~found
        e = np.where(fits, ee, e)
        found |= fits
    q = np.clip(np.rint(np.ldexp(t, e[..., None])), -8, 7).astype(np.int64)
    return e, q


# ---------------------------------------------------------------- error / search

def code_error(w, K: int, P: int, seed: int, e: int, q) -> float:
    """Exact ||w - U(s) q 2^-e||^2 (fp64, index order, no fused multiply-add)."""
    w = np.ascontiguousarray(w, dtype=np.float32)
    q = np.ascontiguousarray(np.asarray(q)[:P], dtype=np.int32)
    out = np.zeros(1, dtype=np.float64)
    if lib().oq_code_error(_p(w), K, P, int(seed), int(e), _p(q), _p(out)) != 0:
        raise ValueError("bad code")
    return float(out[0])


def codes_error(blocks: np.ndarray, K: int, P: int, seeds, es, qs) -> np.ndarray:
    """Exact error of many codes (one per block)."""
    blocks = np.ascontiguousarray(blocks, dtype=np.float32).reshape(-1, C)
    return np.array([code_error(blocks[i], K, P, int(seeds[i]), int(es[i]), qs[i])
                     for i in range(blocks.shape[0])])


@dataclass
class SearchResult:
    seed: np.ndarray   # uint32 [nb]
    e: np.ndarray      # int32 [nb]
    q: np.ndarray      # int32 [nb, P]
    err: np.ndarray    # float64 [nb]


_PINV_CACHE: dict = {}


def clear_pinv_cache() -> None:
    """Drop the cached pseudo-inverse stacks (memory only; no arithmetic)."""
    _PINV_CACHE.clear()


def cached_pinv_stack(K: int, P: int) -> np.ndarray:
    key = (K, P)
    if key not in _PINV_CACHE:
        _PINV_CACHE[key] = np.ascontiguousarray(pinv_stack(K, P))
    return _PINV_CACHE[key]


def search(blocks: np.ndarray, K: int, P: int, threads: int = 0,
           pinv: np.ndarray | None = None) -> SearchResult:
    """Exhaustive seed search (C, OpenMP) for nb blocks of 8 fp32 weights."""
    blocks = np.ascontiguousarray(blocks, dtype=np.float32).reshape(-1, C)
    nb = blocks.shape[0]
    if pinv is None:
        pinv = cached_pinv_stack(K, P)
    pinv = np.ascontiguousarray(pinv, dtype=np.float64)
    seed = np.zeros(nb, dtype=np.uint32)
    e = np.zeros(nb, dtype=np.int32)
    q = np.zeros((nb, P), dtype=np.int32)
    err = np.zeros(nb, dtype=np.float64)
    rc = lib().oq_search(_p(blocks), nb, K, P, _p(pinv), int(threads), _p(seed), _p(e), _p(q),
                         _p(err))
    if rc != 0:
        raise RuntimeError(f"oq_search failed ({rc})")
    return SearchResult(seed, e, q, err)


def search_numpy(blocks: np.ndarray, K: int, P: int) -> SearchResult:
    """Independent vectorised version of the same search (small K only)."""
    blocks = np.asarray(blocks, dtype=np.float32).reshape(-1, C)
    Ui = basis_int_all(K, P)                                   # S x 8 x P
    A = pinv_of(Ui.astype(np.float64) * 2.0 ** -(K - 1))       # S x P x 8
    res = SearchResult(np.zeros(len(blocks), np.uint32), np.zeros(len(blocks), np.int32),
                       np.zeros((len(blocks), P), np.int32), np.zeros(len(blocks)))
    for b, w in enumerate(blocks):
        wd = w.astype(np.float64)
        t = A @ wd                                            # S x P
        e, q = quantize_numpy(t)
        acc = np.einsum("sij,sj->si", Ui, q)                  # exact integers
        what = np.ldexp(acc.astype(np.float64), -(K - 1 + e)[:, None])
        d = wd[None, :] - what
        err = np.zeros(len(t))
        for i in range(C):
            err = err + d[:, i] * d[:, i]
        s = int(np.argmin(err))                               # first minimum
        res.seed[b], res.e[b], res.q[b], res.err[b] = s + 1, e[s], q[s], err[s]
    return res


def decompress(seed, e, q, K_of_block, P_of_block) -> tuple[np.ndarray, np.ndarray]:
    """w_hat (fp32, nb x 8) and the exact integer reconstruction acc (nb x 8)."""
    seed = np.ascontiguousarray(seed, dtype=np.uint32)
    nb = seed.shape[0]
    e = np.ascontiguousarray(e, dtype=np.uint8)
    q = np.ascontiguousarray(q, dtype=np.int8).reshape(nb, -1)
    Ks = np.ascontiguousarray(np.broadcast_to(K_of_block, (nb,)), dtype=np.int32)
    Ps = np.ascontiguousarray(np.broadcast_to(P_of_block, (nb,)), dtype=np.int32)
    w_hat = np.zeros((nb, C), dtype=np.float32)
    acc = np.zeros((nb, C), dtype=np.int32)
    rc = lib().oq_decompress(nb, _p(seed), _p(e), _p(q), q.shape[1], _p(Ks), _p(Ps), _p(w_hat),
                             _p(acc))
    if rc != 0:
        raise ValueError("bad code in decompress")
    return w_hat, acc


def rate_bits(K: int, P: int, m: int = 4, e: int = 4) -> int:
    """Bits per block, eq. (rate): l(S, k) = S + m k + e."""
    return K + m * P + e


from .allocation import schedule, ScheduleResult, hull, hull_slopes, decode_rungs, block_importance, ladder  # noqa: E402,F401
