"""Data-free importance front end for one transformer layer, and the layer's
encode / decode round trip through the library.

Importance (section on data-free block importance):
* q, k, v read gamma_attn * RMSNorm(h), gate and up read gamma_mlp *
  RMSNorm(h): a_j = gamma_j^2 (eq. (gamma));
* o reads the attention output: a_o = repeat_kv((W_v * W_v) a_attn);
  down reads silu(gate) * up: a_down = E[silu(g)^2] ((W_up * W_up) a_mlp) with
  var(g) = (W_gate * W_gate) a_mlp (eq. (prop));
* the outputs of o and down feed the residual stream, so their rows are scaled
  by the data-free gradient size rho = (W_lm * W_lm)^T 1 (a unit gradient at
  every logit, carried back through one layer; output side); the other rows
  get rho = 1;
* before blocking, every tensor's input channels are put in increasing order
  of a; the outlier
  columns (appendix on outlier columns) are kept in FP16 and overwrite the
  codec's reconstruction.
Every step of the importance runs in the library (seedq_gamma_importance,
seedq_propagate_o, seedq_propagate_down, seedq_sq_gemv, seedq_column_stats on
the GPU; the ranking and sorting in its host functions); this module only moves
arrays between them.

    python -m paper_2609_38477_amd.frontend [--d 4096 --f 14336 ...]

prints one JSON line: the importance spread, the outlier columns found, and per
tensor the encode / decode timings and errors.
"""
from __future__ import annotations

import argparse
import json
import sys
import time
from dataclasses import dataclass, field

import numpy as np

from . import (SEEDQ_BLOCK, build_bases, compress, decompress_stream, derive_schedule, pack,
               plan_schedule, seedq_apply_columns, seedq_channel_order, seedq_column_stats,
               seedq_extract_columns, seedq_gamma_importance, seedq_permute_columns,
               seedq_propagate_down, seedq_propagate_o, seedq_propagate_workspace_bytes,
               seedq_select_outliers, seedq_sq_gemv, seedq_sq_gemv_workspace_bytes)

PROJECTIONS = ("q", "k", "v", "o", "gate", "up", "down")
READS_ATTN_NORM = ("q", "k", "v")
READS_MLP_NORM = ("gate", "up")
WRITES_RESIDUAL = ("o", "down")
GH_NODES = 128
OUTLIER_COLUMNS = 4


def _dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def sq_gemv(W, v, transpose: bool = False) -> np.ndarray:
    """(W * W) v or (W * W)^T v on the GPU (fp64 result, host numpy)."""
    import torch
    nrows, ncols = W.shape
    out = torch.empty(ncols if transpose else nrows, dtype=torch.float64, device=W.device)
    nws = seedq_sq_gemv_workspace_bytes(nrows, ncols, int(transpose))
    ws = torch.empty(max(nws, 256), dtype=torch.uint8, device=W.device) if nws else None
    seedq_sq_gemv(W, nrows, ncols, v.float().contiguous(), int(transpose), out, ws, nws)
    return out.cpu().numpy()


@dataclass
class LayerImportance:
    a: dict = field(default_factory=dict)        # name -> fp64 [in channels]
    rho: dict = field(default_factory=dict)      # name -> fp64 [out channels] (o, down)
    perm: dict = field(default_factory=dict)     # name -> int32 channel order
    outliers: list = field(default_factory=list)  # [(name, column)]
    stats: dict = field(default_factory=dict)     # name -> (maxabs, median)


def layer_importance(layer, dW=None) -> LayerImportance:
    """a, rho, channel orders and outlier columns of a SyntheticLayer-like
    object (tensors: name -> [out, in] fp32, gains: attn / mlp)."""
    import torch
    dW = dW or {n: _dev(layer.tensors[n]) for n in (*PROJECTIONS, "lm_head")}
    imp = LayerImportance()
    d_a = {}
    for norm in ("attn", "mlp"):
        g = _dev(np.asarray(layer.gains[norm], dtype=np.float32))
        d_a[norm] = torch.empty(g.numel(), dtype=torch.float64, device="cuda")
        seedq_gamma_importance(g, g.numel(), d_a[norm])
    a_attn, a_mlp = d_a["attn"].cpu().numpy(), d_a["mlp"].cpu().numpy()
    for n in READS_ATTN_NORM:
        imp.a[n] = a_attn
    for n in READS_MLP_NORM:
        imp.a[n] = a_mlp
    Rv, Cv = layer.tensors["v"].shape
    a_o = torch.empty(layer.n_heads * (Rv // layer.n_kv_heads), dtype=torch.float64, device="cuda")
    nws = seedq_propagate_workspace_bytes(Rv, Cv)
    ws = torch.empty(nws, dtype=torch.uint8, device="cuda")
    seedq_propagate_o(dW["v"], Rv, Cv, layer.n_heads, layer.n_kv_heads, d_a["attn"], a_o, ws, nws)
    imp.a["o"] = a_o.cpu().numpy()
    Rg, Cg = layer.tensors["gate"].shape
    a_down = torch.empty(Rg, dtype=torch.float64, device="cuda")
    nws = seedq_propagate_workspace_bytes(Rg, Cg)
    ws = torch.empty(nws, dtype=torch.uint8, device="cuda")
    seedq_propagate_down(dW["gate"], dW["up"], Rg, Cg, d_a["mlp"], GH_NODES, a_down, ws, nws)
    imp.a["down"] = a_down.cpu().numpy()
    rho = sq_gemv(dW["lm_head"], torch.ones(layer.vocab, device="cuda"), transpose=True)
    for n in WRITES_RESIDUAL:
        imp.rho[n] = rho
    for n in PROJECTIONS:
        R, C = layer.tensors[n].shape
        mx = torch.empty(C, dtype=torch.float64, device="cuda")
        md = torch.empty_like(mx)
        seedq_column_stats(dW[n], R, C, mx, md)
        imp.stats[n] = (mx.cpu().numpy(), md.cpu().numpy())
        imp.perm[n] = seedq_channel_order(imp.a[n].astype(np.float32))
    names = list(PROJECTIONS)
    sel = seedq_select_outliers([imp.stats[n][0] for n in names], [imp.stats[n][1] for n in names],
                                [imp.a[n] for n in names], OUTLIER_COLUMNS)
    imp.outliers = [(names[t], c) for t, c in sel]
    return imp


@dataclass
class EncodedTensor:
    name: str
    shape: tuple
    rob: np.ndarray
    report: dict
    words: object
    perm: object          # device int32
    escape_cols: object   # device int32 (original column indices) or None
    escape_fp16: object   # device fp16 [ncol][rows] or None
    a_sorted: np.ndarray
    rho: np.ndarray | None
    seconds: dict = field(default_factory=dict)


def encode_tensor(name, W, a, rho, escape, rungs, damage, target_bpw) -> EncodedTensor:
    """Sort the input channels by a, plan the rungs, search every block and emit
    the stream; extract the escape columns (original indices) in FP16."""
    import torch
    R, C = W.shape
    sec = {}
    perm = seedq_channel_order(np.asarray(a, dtype=np.float32))
    d_perm = _dev(perm)
    Wp = torch.empty_like(W)
    seedq_permute_columns(W, R, C, d_perm, 0, Wp)
    a_sorted = np.asarray(a, dtype=np.float64)[perm].astype(np.float32)
    t = time.perf_counter()
    rob, rep = plan_schedule(R, C, rungs, damage, target_bpw, a_sorted,
                             None if rho is None else np.asarray(rho, np.float32), 0.06)
    sec["plan"] = time.perf_counter() - t
    d_rob = _dev(rob)
    bases = [build_bases(K, P) for K, P in rungs]
    torch.cuda.synchronize()
    t = time.perf_counter()
    seed, exp, q, _ = compress(Wp, bases, d_rob)
    torch.cuda.synchronize()
    sec["search"] = time.perf_counter() - t
    words = pack(seed, exp, q, list(rungs), R, C, d_rob, rep["count"])
    cols, f16 = None, None
    if escape:
        cols = _dev(np.asarray(escape, dtype=np.int32))
        f16 = torch.empty((len(escape), R), dtype=torch.float16, device="cuda")
        seedq_extract_columns(W, R, C, len(escape), cols, f16)
    return EncodedTensor(name, (R, C), rob, rep, words, d_perm, cols, f16, a_sorted,
                         None if rho is None else np.asarray(rho, np.float32), sec)


def decode_tensor(enc: EncodedTensor, rungs, damage):
    """Algorithm 2 for one tensor: rungs from the stored table, one-pass decode,
    inverse channel permutation, FP16 columns written over the reconstruction."""
    import torch
    R, C = enc.shape
    rob = derive_schedule(R, C, rungs, damage, enc.a_sorted, enc.report["lam"],
                          enc.report["floor_q"], enc.report["tie_count"], enc.rho)
    Wp = decompress_stream(enc.words, list(rungs), R, C, _dev(rob))
    W = torch.empty_like(Wp)
    seedq_permute_columns(Wp, R, C, enc.perm, 1, W)
    if enc.escape_cols is not None:
        seedq_apply_columns(W, R, C, enc.escape_cols.numel(), enc.escape_cols, enc.escape_fp16)
    return W


def main(argv=None) -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--d", type=int, default=1024)
    ap.add_argument("--f", type=int, default=2816)
    ap.add_argument("--heads", type=int, default=16)
    ap.add_argument("--kv-heads", type=int, default=4)
    ap.add_argument("--vocab", type=int, default=8192)
    ap.add_argument("--target-bpw", type=float, default=4.0)
    args = ap.parse_args(argv)
    import os
    import torch
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    if root not in sys.path:
        sys.path.insert(0, root)
    import synthetic
    layer = synthetic.synthetic_layer(args.d, args.f, args.heads, args.kv_heads, args.vocab)
    dW = {n: _dev(layer.tensors[n]) for n in (*PROJECTIONS, "lm_head")}
    torch.cuda.synchronize()
    t = time.perf_counter()
    imp = layer_importance(layer, dW)
    torch.cuda.synchronize()
    t_imp = time.perf_counter() - t
    rungs, damage = ((12, 2), (16, 3), (20, 4)), (4.0, 1.0, 0.25)
    rows = []
    for n in PROJECTIONS:
        esc = [c for (tn, c) in imp.outliers if tn == n]
        enc = encode_tensor(n, dW[n], imp.a[n], imp.rho.get(n), esc, rungs, damage, args.target_bpw)
        Wd = decode_tensor(enc, rungs, damage)
        W = dW[n].double()
        err = ((Wd.double() - W) ** 2).sum().item() / (W ** 2).sum().item()
        rows.append({"tensor": n, "shape": list(enc.shape), "escaped_columns": esc,
                     "rung_counts": enc.report["count"], "tie_count": enc.report["tie_count"],
                     "relative_sq_error": err, "search_s": enc.seconds["search"],
                     "plan_s": enc.seconds["plan"]})
    spread = {n: float(np.quantile(imp.a[n], 0.95) / np.quantile(imp.a[n], 0.05)) for n in PROJECTIONS}
    print(json.dumps({"layer": {"d": args.d, "f": args.f, "heads": args.heads,
                                "kv_heads": args.kv_heads, "vocab": args.vocab},
                      "importance_seconds": t_imp, "a_p95_over_p5": spread,
                      "outliers": imp.outliers, "planted_super_weight": list(layer.super_weight),
                      "massive_channel": layer.massive_channel, "tensors": rows}), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
