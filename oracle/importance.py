"""Oracle for the data-free importance front end (test infrastructure only).

Plain fp64 numpy, in the paper's order:

* input side (section on data-free block importance, eq. (gamma)): the five
  projections that read gamma * RMSNorm(h) get a_j = gamma_j^2;
* one-hop propagation (eq. (prop)): a_o = repeat_kv((W_v * W_v) a_in) for the
  output projection, and a_down_c = E[silu(g_c)^2] ((W_up * W_up) a_in)_c with
  g_c ~ N(0, ((W_gate * W_gate) a_in)_c) for the down projection, the
  expectation by Gauss-Hermite quadrature;
* output side: an isotropic unit gradient at the logits, one hop back through
  the language-model head, rho_c = sum_r W_lm[r, c]^2; it applies to the rows
  of W_o and W_down (the appendix on the approximations);
* channel sort: input channels in increasing a, ties by channel index, before
  blocking (paragraph on block importance);
* outlier columns (appendix on outlier columns): a column is a candidate when
  max_i |W_ij| / (median_i |W_ij| + eps) >= 1e3 or a_j >= 1e2 times the
  tensor mean of a; a rule's list holds up to 32 candidates, those with the
  largest statistic (ties by tensor, then column index), in decreasing order
  of it; a candidate's rank is the smaller of its two list positions (ties by
  tensor, then column) and the four best ranked are kept.

Readings where the paper is silent: the quadrature uses 128 Gauss-Hermite
nodes (relative error below 1e-12 for variances up to 4, 2.4e-6 at 25);
eps = 2^-24 times the column's largest
|W| (so an all-zero column has ratio 0 and a column that is zero except one
weight has ratio 2^24); the median is numpy's (the mean of the two middle
values for an even count); repeat_kv repeats each key-value head's channels
for the n_heads / n_kv_heads query heads that share it, head-major.
"""
from __future__ import annotations

import numpy as np

DR_THRESHOLD = 1.0e3       # dynamic-range rule
ACT_THRESHOLD = 1.0e2      # activation-scale rule, times the tensor mean
KEEP_PER_RULE = 32
KEEP = 4
EPS_REL = 2.0 ** -24


def gamma_importance(gain) -> np.ndarray:
    """eq. (gamma): a_j = gamma_j^2."""
    g = np.asarray(gain, dtype=np.float64)
    return g * g


def sq_matvec(W, v) -> np.ndarray:
    """(W * W) v in fp64."""
    W = np.asarray(W, dtype=np.float64)
    return (W * W) @ np.asarray(v, dtype=np.float64)


def sq_matvec_t(W, v) -> np.ndarray:
    """(W * W)^T v in fp64."""
    W = np.asarray(W, dtype=np.float64)
    return (W * W).T @ np.asarray(v, dtype=np.float64)


def silu(x):
    return x / (1.0 + np.exp(-x))


def e_silu_sq(var, nodes: int = 128) -> np.ndarray:
    """E[silu(g)^2] for g ~ N(0, var), Gauss-Hermite with ``nodes`` points:
    E[f(g)] = pi^-1/2 sum_i w_i f(sqrt(2 var) x_i)."""
    x, w = np.polynomial.hermite.hermgauss(nodes)
    var = np.asarray(var, dtype=np.float64)
    g = np.sqrt(2.0 * var)[..., None] * x
    return (w * silu(g) ** 2).sum(axis=-1) / np.sqrt(np.pi)


def propagate_o(W_v, a_in, n_heads: int, n_kv_heads: int) -> np.ndarray:
    """a_o of eq. (prop): the value channels' second moments, repeated for the
    query heads sharing each key-value head."""
    v = sq_matvec(W_v, a_in)                      # [n_kv_heads * head_dim]
    hd = v.size // n_kv_heads
    return np.repeat(v.reshape(n_kv_heads, hd), n_heads // n_kv_heads, axis=0).reshape(-1)


def propagate_down(W_gate, W_up, a_in, nodes: int = 128) -> np.ndarray:
    """a_down of eq. (prop)."""
    return e_silu_sq(sq_matvec(W_gate, a_in), nodes) * sq_matvec(W_up, a_in)


def rho_from_head(W_lm) -> np.ndarray:
    """Row scale of the residual stream: a unit gradient at every logit carried
    back through the output head."""
    return sq_matvec_t(W_lm, np.ones(np.asarray(W_lm).shape[0]))


def channel_order(a) -> np.ndarray:
    """Permutation sorting input channels by increasing a, ties by index."""
    return np.argsort(np.asarray(a, dtype=np.float64), kind="stable")


def column_stats(W):
    """(max_i |W_ij|, median_i |W_ij|) per column, fp64."""
    A = np.abs(np.asarray(W, dtype=np.float64))
    return A.max(axis=0), np.median(A, axis=0)


def dynamic_range(W) -> np.ndarray:
    mx, med = column_stats(W)
    out = np.zeros_like(mx)
    np.divide(mx, med + EPS_REL * mx, out=out, where=mx > 0)
    return out


def outlier_columns(tensors, a_list, keep: int = KEEP):
    """[(tensor index, column)] of the stored outlier columns over a list of
    weight matrices (columns = input channels) and their a vectors."""
    dr_c, act_c = [], []
    for t, (W, a) in enumerate(zip(tensors, a_list)):
        dr = dynamic_range(W)
        a = np.asarray(a, dtype=np.float64)
        for j in np.nonzero(dr >= DR_THRESHOLD)[0]:
            dr_c.append((-dr[j], t, int(j)))
        for j in np.nonzero(a >= ACT_THRESHOLD * a.mean())[0]:
            act_c.append((-a[j], t, int(j)))
    dr_c = sorted(dr_c)[:KEEP_PER_RULE]
    act_c = sorted(act_c)[:KEEP_PER_RULE]
    pos = {}
    for lst in (dr_c, act_c):
        for i, (_, t, j) in enumerate(lst):
            pos[(t, j)] = min(pos.get((t, j), i), i)
    ranked = sorted(pos, key=lambda tj: (pos[tj], tj[0], tj[1]))
    return ranked[:keep]
