"""The importance front end of one 7B-shaped synthetic layer (d 4096, f 11008,
32 heads, 8 KV heads, vocabulary 32000) against the oracle (a one-off check at
full size; the suite runs the same comparison on a smaller layer): the column
importances of all seven projections (1e-12 relative), the channel orders, the
output-side row factors and the outlier columns.

    python3 tests/frontend_oracle_check.py

Prints one JSON line; exits non-zero if a check fails."""
import json
import os
import sys

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import synthetic  # noqa: E402
from oracle import importance as oimp  # noqa: E402


def main() -> int:
    from paper_2609_38477_amd import frontend
    L = synthetic.synthetic_layer(4096, 11008, 32, 8, 32000)
    imp = frontend.layer_importance(L)
    T = L.tensors
    a_attn = oimp.gamma_importance(L.gains["attn"])
    a_mlp = oimp.gamma_importance(L.gains["mlp"])
    ref = {"q": a_attn, "k": a_attn, "v": a_attn, "gate": a_mlp, "up": a_mlp,
           "o": oimp.propagate_o(T["v"], a_attn.astype(np.float32), L.n_heads, L.n_kv_heads),
           "down": oimp.propagate_down(T["gate"], T["up"], a_mlp.astype(np.float32))}
    out = {"layer": {"d": 4096, "f": 11008, "heads": 32, "kv_heads": 8, "vocab": 32000}}
    ok = True
    for n, a in ref.items():
        rel = float(np.max(np.abs(imp.a[n] - a) / np.abs(a)))
        same_order = bool(np.array_equal(imp.perm[n], oimp.channel_order(imp.a[n].astype(np.float32))))
        out[n] = {"columns": int(len(a)), "max_rel_err": rel, "order_same": same_order}
        ok = ok and rel <= 1e-12 and same_order
    rho = oimp.rho_from_head(T["lm_head"])
    rho_rel = float(np.max(np.abs(imp.rho["o"] - rho) / np.abs(rho)))
    names = list(frontend.PROJECTIONS)
    want = [(names[t], c) for t, c in oimp.outlier_columns([T[n] for n in names],
                                                           [ref[n] for n in names])]
    out["rho_max_rel_err"] = rho_rel
    out["outliers"] = len(want)
    out["outliers_same"] = imp.outliers == want
    out["planted_found"] = ("down", L.super_weight[1]) in imp.outliers and \
                           ("gate", L.massive_channel) in imp.outliers
    ok = ok and rho_rel <= 1e-12 and out["outliers_same"] and out["planted_found"]
    out["ok"] = bool(ok)
    print(json.dumps(out), flush=True)
    return 0 if ok else 1


if __name__ == "__main__":
    sys.exit(main())
