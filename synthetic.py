"""Seeded synthetic inputs for the Seed-Q block seed search.

This module only draws random numbers and shapes them into the workloads the
parity tests and the benchmark use. It holds none of the codec's arithmetic
(no LFSR, no least squares, no quantiser, no allocation): both the HIP path and
the CPU oracle receive what it returns as plain arrays.

Random numbers come from one counter-based generator, SplitMix64 (Steele, Lea
and Flood, "Fast splittable pseudorandom number generators", OOPSLA 2014):
output n of stream k under key s is the SplitMix64 finaliser applied to
``base(s, k) + (n + 1) * 0x9E3779B97F4A7C15``. Uniforms take the top 53 bits,
normals use the Box-Muller transform, Student-t(3) variates are
``Z0 / sqrt((Z1^2 + Z2^2 + Z3^2) / 3)``.

The weight distributions follow the shapes of LLM projection matrices the paper
compresses (the paper's checkpoints are not available): i.i.d. N(0, sigma^2)
entries, a fraction of which (0.1 %) is replaced by heavy-tailed
0.1 * Student-t(3) outliers. The column-importance profile is a stand-in for the
RMSNorm-gain importance a_j ~ gamma_j^2 of the paper's eq. (gamma): log-normal
quantiles exp(Phi^-1((j + 1/2) / N)), ascending, so the paper's sort of input
channels by importance before blocking is the identity permutation.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

_GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)

# Stream identifiers: every independent draw of a workload uses its own stream.
STREAM_GAUSS = 1
STREAM_OUTLIER_POS = 2
STREAM_OUTLIER_VAL = 3
STREAM_PLANT = 4
STREAM_CODES = 5
STREAM_MISC = 6


def _finalize(z: np.ndarray) -> np.ndarray:
    z = (z ^ (z >> np.uint64(30))) * _M1
    z = (z ^ (z >> np.uint64(27))) * _M2
    return z ^ (z >> np.uint64(31))


def _base(key: int, stream: int) -> np.uint64:
    k = np.array([(int(key) & 0xFFFFFFFF) << 20 ^ (int(stream) & 0xFFFFF)], dtype=np.uint64)
    with np.errstate(over="ignore"):
        return _finalize(k * _GAMMA + _GAMMA)[0]


def splitmix64(key: int, stream: int, n: int, start: int = 0) -> np.ndarray:
    """``n`` consecutive 64-bit outputs of stream ``stream`` under ``key``."""
    ctr = np.arange(start, start + n, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = _base(key, stream) + (ctr + np.uint64(1)) * _GAMMA
        return _finalize(z)


def uniform(key: int, stream: int, n: int, start: int = 0) -> np.ndarray:
    """Uniform doubles in the open interval (0, 1)."""
    z = splitmix64(key, stream, n, start)
    return ((z >> np.uint64(11)).astype(np.float64) + 0.5) * (2.0 ** -53)


def normal(key: int, stream: int, n: int, start: int = 0) -> np.ndarray:
    """Standard normal doubles by Box-Muller over pairs of uniforms."""
    m = (n + 1) // 2
    u = uniform(key, stream, 2 * m, 2 * start)
    r = np.sqrt(-2.0 * np.log(u[0::2]))
    th = 2.0 * np.pi * u[1::2]
    out = np.empty(2 * m, dtype=np.float64)
    out[0::2] = r * np.cos(th)
    out[1::2] = r * np.sin(th)
    return out[:n]


def student_t3(key: int, stream: int, n: int) -> np.ndarray:
    z = normal(key, stream, 4 * n).reshape(n, 4)
    return z[:, 0] / np.sqrt((z[:, 1] ** 2 + z[:, 2] ** 2 + z[:, 3] ** 2) / 3.0)


def weights(nrows: int, ncols: int, sigma: float, key: int,
            outlier_frac: float = 0.0, outlier_scale: float = 0.1,
            chunk: int = 1 << 24) -> np.ndarray:
    """Row-major fp32 ``nrows x ncols`` matrix: N(0, sigma^2) entries drawn in
    fp64, with exactly ``round(outlier_frac * nrows * ncols)`` distinct
    positions replaced by ``outlier_scale * t3``. Generated in chunks so that
    the 235M-entry layer fits comfortably in host memory."""
    n = int(nrows) * int(ncols)
    w = np.empty(n, dtype=np.float32)
    for s in range(0, n, chunk):
        m = min(chunk, n - s)
        w[s:s + m] = (normal(key, STREAM_GAUSS, m, s) * sigma).astype(np.float32)
    m = int(round(outlier_frac * n))
    if m > 0:
        # The m positions with the smallest 64-bit hash: a seeded sample
        # without replacement that does not depend on numpy's RNG.
        best_keys = np.empty(0, dtype=np.uint64)
        best_idx = np.empty(0, dtype=np.int64)
        for s in range(0, n, chunk):
            c = min(chunk, n - s)
            h = splitmix64(key, STREAM_OUTLIER_POS, c, s)
            k = min(m, c)
            part = np.argpartition(h, k - 1)[:k]
            best_keys = np.concatenate([best_keys, h[part]])
            best_idx = np.concatenate([best_idx, part.astype(np.int64) + s])
            if best_keys.size > m:
                keep = np.argpartition(best_keys, m - 1)[:m]
                best_keys, best_idx = best_keys[keep], best_idx[keep]
        order = np.argsort(best_keys, kind="stable")
        pos = best_idx[order]
        w[pos] = (outlier_scale * student_t3(key, STREAM_OUTLIER_VAL, m)).astype(np.float32)
    return w.reshape(nrows, ncols)


def importance_profile(ncols: int) -> np.ndarray:
    """fp32 a_j = exp(Phi^-1((j + 1/2) / ncols)), ascending."""
    from scipy.special import ndtri
    j = np.arange(ncols, dtype=np.float64)
    return np.exp(ndtri((j + 0.5) / ncols)).astype(np.float32)


def random_codes(n: int, K: int, P: int, key: int, exps=(7, 8, 9),
                 canonical: bool = True) -> tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Random block codes (seed in [1, 2^K - 1], exponent from ``exps``,
    P signed 4-bit mantissas in [-8, 7]). With ``canonical`` the mantissas are
    nonzero and at least one lies outside [-4, 3] (or the exponent is 15), so
    that no finer exponent represents the same coefficients."""
    u = splitmix64(key, STREAM_CODES, n * (2 + 4 * P))
    seeds = (u[0:n] % np.uint64((1 << K) - 1)).astype(np.int64) + 1
    e = np.asarray(exps, dtype=np.int64)[(u[n:2 * n] % np.uint64(len(exps))).astype(np.int64)]
    if canonical:
        # nonzero mantissas: a zero first (last) mantissa would make the code
        # reproducible by the seed 8 LFSR steps later (earlier) as well
        qs = ((u[2 * n:].reshape(n, 4, P) >> np.uint64(7)) % np.uint64(15)).astype(np.int64) - 8
        qs = np.where(qs >= 0, qs + 1, qs)
    else:
        qs = ((u[2 * n:].reshape(n, 4, P) >> np.uint64(7)) % np.uint64(16)).astype(np.int64) - 8
    q = qs[:, 0, :].copy()
    if canonical:
        for tries in range(1, 4):
            bad = ~(((q < -4) | (q > 3)).any(axis=1) | (e == 15))
            if not bad.any():
                break
            q[bad] = qs[bad, tries, :]
        bad = ~(((q < -4) | (q > 3)).any(axis=1) | (e == 15))
        q[bad, 0] = 7
    return seeds.astype(np.uint32), e.astype(np.uint8), q.astype(np.int8)


@dataclass(frozen=True)
class Workload:
    name: str
    nrows: int
    ncols: int
    sigma: float
    key: int
    outlier_frac: float
    rungs: tuple          # ((K, P), ...) ascending rate
    damage: tuple | None  # e(g) per rung, None for a single rung
    target_bpw: float
    planted: int = 0      # planted blocks appended as extra rows
    note: str = ""

    @property
    def nblocks(self) -> int:
        return self.nrows * self.ncols // 8


# The five workloads. Rung damages (4, 1, 0.25) stand in for the measured
# excess losses e(g) of the paper's damage curve: convex, every added
# coefficient cuts the damage by a large factor.
_THREE = ((12, 2), (16, 3), (20, 4))
_DAMAGE = (4.0, 1.0, 0.25)
WORKLOADS = {
    "tiny": Workload("tiny", 256, 256, 0.02, 0, 0.0, ((12, 3),), None, 3.5, planted=64,
                     note="256x256 N(0,0.02^2), uniform (12,3), +64 planted blocks"),
    "attn4096": Workload("attn4096", 4096, 4096, 0.02, 1, 0.001, ((16, 3),), None, 4.0,
                         note="4096x4096 attention projection, uniform (16,3), 4.0 bpw"),
    "mlp_up": Workload("mlp_up", 4096, 14336, 0.02, 2, 0.001, _THREE, _DAMAGE, 4.0,
                       note="4096x14336 MLP up-projection, three rungs at 4.0 bpw"),
    "reduced": Workload("reduced", 4096, 11008, 0.02, 3, 0.001, _THREE, _DAMAGE, 3.5,
                        note="4096x11008, three rungs at 3.5 bpw"),
    "l70b": Workload("l70b", 8192, 28672, 0.015, 4, 0.001, _THREE, _DAMAGE, 4.0,
                     note="8192x28672 70B-shaped layer, three rungs at 4.0 bpw"),
}


def workload_weights(wl: Workload) -> np.ndarray:
    return weights(wl.nrows, wl.ncols, wl.sigma, wl.key, wl.outlier_frac)


@dataclass
class SyntheticLayer:
    """One pre-norm transformer layer plus a language-model head, random weights
    (no checkpoint is read): RMSNorm gains around 1 with one massive-activation
    channel, projection weights N(0, sigma^2) with the workloads' outliers, and
    one planted super weight in W_down."""
    d: int
    f: int
    n_heads: int
    n_kv_heads: int
    vocab: int
    tensors: dict = field(default_factory=dict)   # name -> fp32 [out, in]
    gains: dict = field(default_factory=dict)     # "attn", "mlp" -> fp32 [d]
    super_weight: tuple = (0, 0)                  # (row, column) in W_down
    massive_channel: int = 0                      # channel of gains["mlp"]


def synthetic_layer(d: int = 512, f: int = 1536, n_heads: int = 8, n_kv_heads: int = 2,
                    vocab: int = 2048, key: int = 9, sigma: float = 0.02) -> SyntheticLayer:
    hd = d // n_heads
    L = SyntheticLayer(d, f, n_heads, n_kv_heads, vocab)
    shapes = {"q": (d, d), "k": (n_kv_heads * hd, d), "v": (n_kv_heads * hd, d), "o": (d, d),
              "gate": (f, d), "up": (f, d), "down": (d, f), "lm_head": (vocab, d)}
    for i, (name, (r, c)) in enumerate(shapes.items()):
        L.tensors[name] = weights(r, c, sigma, key * 16 + i, 0.001)
    for i, name in enumerate(("attn", "mlp")):
        z = normal(key * 16 + 10 + i, STREAM_MISC, d)
        L.gains[name] = np.exp(0.3 * z).astype(np.float32)
    u = splitmix64(key, STREAM_MISC, 3, start=1 << 20)
    L.massive_channel = int(u[0] % np.uint64(d))
    L.gains["mlp"][L.massive_channel] = 30.0
    L.super_weight = (int(u[1] % np.uint64(d)), int(u[2] % np.uint64(f)))
    L.tensors["down"][L.super_weight] = 20.0
    return L
