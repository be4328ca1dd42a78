"""The whole decoder path of a searched multi-rung layer against the oracle
(a one-off check, too long for the test suite): the codes of every block are
packed into the headerless stream, the rungs are re-derived on the host from
the stored lambda / floor / tie count, and then

  - the one-pass decode of the stream equals the oracle's exact reconstruction
    of every code, bit for bit (all weights of the layer);
  - unpacking the stream returns every code;
  - the decode-GEMV of one vector is within the fp32 accumulation bound of the
    fp64 product of the oracle's weights with that vector, on every row.

    python3 tests/decode_oracle_check.py [--workload l70b]

Prints one JSON line; exits non-zero if a check fails."""
import argparse
import json
import os
import sys

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import oracle  # noqa: E402
import synthetic  # noqa: E402


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="l70b")
    args = ap.parse_args()
    import torch
    import paper_2609_38477_amd as sq
    wl = synthetic.WORKLOADS[args.workload]
    W = synthetic.workload_weights(wl)
    a = synthetic.importance_profile(wl.ncols)
    rob, rep = sq.plan_schedule(wl.nrows, wl.ncols, wl.rungs, wl.damage, wl.target_bpw, a)
    d_rob = torch.from_numpy(rob).cuda()
    bases = [sq.build_bases(K, P) for K, P in wl.rungs]
    seed, e, q, _ = sq.compress(torch.from_numpy(W).cuda(), bases, rung_of_block=d_rob)
    del bases
    words = sq.pack(seed, e, q, wl.rungs, wl.nrows, wl.ncols, d_rob, rep["count"])
    dec = sq.derive_schedule(wl.nrows, wl.ncols, wl.rungs, wl.damage, a, rep["lam"],
                             rep["floor_q"], rep["tie_count"])
    rungs_same = bool(np.array_equal(dec, rob))
    d_dec = torch.from_numpy(dec).cuda()
    W_hat = sq.decompress_stream(words, wl.rungs, wl.nrows, wl.ncols, d_dec).cpu().numpy()
    s2, e2, q2 = sq.unpack(words, wl.rungs, wl.nrows, wl.ncols, d_dec)
    codes_same = bool(torch.equal(s2, seed) and torch.equal(e2, e) and torch.equal(q2, q))
    g = np.random.default_rng(5)
    x = g.standard_normal(wl.ncols).astype(np.float32)
    y = sq.gemv_stream(words, wl.rungs, wl.nrows, wl.ncols, torch.from_numpy(x).cuda(),
                       d_dec).cpu().numpy()
    seed_h = seed.cpu().numpy().view(np.uint32)
    K_of = np.array([k for k, _ in wl.rungs], dtype=np.int64)[rob]
    P_of = np.array([p for _, p in wl.rungs], dtype=np.int64)[rob]
    Wr, _ = oracle.decompress(seed_h, e.cpu().numpy(), q.cpu().numpy(), K_of, P_of)
    Wr = np.asarray(Wr, dtype=np.float32).reshape(wl.nrows, wl.ncols)
    weights_same = bool(np.array_equal(W_hat.view(np.uint32), Wr.view(np.uint32)))
    ref = Wr.astype(np.float64) @ x.astype(np.float64)
    n = (wl.ncols // 8 + 63) // 64 * 8 + 8
    bound = n * 2.0 ** -24 * (np.abs(Wr.astype(np.float64)) @ np.abs(x.astype(np.float64)))
    gemv_ok = bool(np.all(np.abs(y - ref) <= bound))
    out = {"workload": wl.name, "blocks": int(len(rob)), "weights": int(Wr.size),
           "stream_bytes": int(words.numel() * 4), "rungs_rederived_same": rungs_same,
           "unpacked_codes_same": codes_same, "decoded_weights_bit_exact": weights_same,
           "gemv_rows_within_bound": int(np.count_nonzero(np.abs(y - ref) <= bound)),
           "rows": int(wl.nrows),
           "gemv_max_err_over_bound": float(np.max(np.abs(y - ref) / np.maximum(bound, 1e-300)))}
    ok = rungs_same and codes_same and weights_same and gemv_ok
    out["ok"] = ok
    print(json.dumps(out), flush=True)
    return 0 if ok else 1


if __name__ == "__main__":
    sys.exit(main())
