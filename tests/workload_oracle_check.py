"""A multi-rung workload searched on the GPU exactly as the benchmark runs it
(schedule, bases, one compress call over every block), then checked against the
oracle's exhaustive search on an evenly spaced sample of the blocks of every
rung (a one-off check, too long for the test suite).

Per sampled block: the exact error of the GPU's code (re-scored by the oracle)
is within 1e-5 relative (plus 1e-7 ||w||^2) of the oracle's best error, the
reported error is that exact error rounded to fp32, and seed agreement is
counted (a difference is allowed only at a near-tie).

    python3 tests/workload_oracle_check.py --workload l70b [--sample 4096] [--threads 16]

Prints one JSON line per rung and a summary line; exits non-zero if a bar fails."""
import argparse
import json
import os
import sys

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import oracle  # noqa: E402
import synthetic  # noqa: E402

REL, TAU = 1e-5, 1e-7


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="l70b")
    ap.add_argument("--sample", type=int, default=4096)
    ap.add_argument("--threads", type=int, default=16)
    args = ap.parse_args()
    import torch
    import paper_2609_38477_amd as sq
    wl = synthetic.WORKLOADS[args.workload]
    W = synthetic.workload_weights(wl)
    a = synthetic.importance_profile(wl.ncols)
    rob, rep = sq.plan_schedule(wl.nrows, wl.ncols, wl.rungs, wl.damage, wl.target_bpw, a)
    bases = [sq.build_bases(K, P) for K, P in wl.rungs]
    seed, e, q, err = sq.compress(torch.from_numpy(W).cuda(), bases,
                                  rung_of_block=torch.from_numpy(rob).cuda())
    seed = seed.cpu().numpy().view(np.uint32).astype(np.int64)
    e, q, err = e.cpu().numpy().astype(np.int64), q.cpu().numpy().astype(np.int64), err.cpu().numpy()
    del bases
    blocks = W.reshape(-1, 8)
    bad = 0
    for r, (K, P) in enumerate(wl.rungs):
        sel = np.nonzero(rob == r)[0]
        idx = sel[np.linspace(0, len(sel) - 1, min(args.sample, len(sel))).round().astype(np.int64)]
        sub = np.ascontiguousarray(blocks[idx])
        ww = (sub.astype(np.float64) ** 2).sum(axis=1)
        ref = oracle.search(sub, K, P, threads=args.threads)
        oracle.clear_pinv_cache()
        mine = np.array([oracle.code_error(sub[i], K, P, int(seed[j]), int(e[j]), q[j, :P])
                         for i, j in enumerate(idx)])
        within = mine <= ref.err * (1 + REL) + TAU * ww
        reported = np.abs(err[idx].astype(np.float64) - mine) <= 1e-6 * mine + 1e-30
        same = seed[idx] == ref.seed
        ok = bool(within.all() and reported.all())
        bad += not ok
        print(json.dumps({"workload": wl.name, "rung": [K, P], "rung_blocks": int(len(sel)),
                          "checked": int(len(idx)), "within_bar": int(within.sum()),
                          "reported_exact": int(reported.sum()), "same_seed": int(same.sum()),
                          "ok": ok}), flush=True)
    print(json.dumps({"workload": wl.name, "rungs": len(wl.rungs), "failed": bad}), flush=True)
    return 1 if bad else 0


if __name__ == "__main__":
    sys.exit(main())
