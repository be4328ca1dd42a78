"""Every rung of the paper's grid (S in 8..16, k in 2..6) searched on the GPU
over all 2 097 152 blocks of the 4096x4096 attention workload, checked against
the oracle's exhaustive search on an evenly spaced sample of blocks (a one-off
check, too long for the test suite: minutes of host time).

Per rung and sampled block: the exact error of the GPU's code (re-scored by the
oracle) is within 1e-5 relative (plus 1e-7 ||w||^2) of the oracle's best error,
the GPU's reported error is that exact error rounded to fp32, and the seeds are
reported as agreeing or not (they may differ only at near-ties).

    python3 tests/grid_oracle_check.py [--sample 256] [--threads 16]

Prints one JSON line per rung and a summary line; exits non-zero if any bar fails."""
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
    ap.add_argument("--sample", type=int, default=256)
    ap.add_argument("--threads", type=int, default=16)
    args = ap.parse_args()
    import torch
    import paper_2609_38477_amd as sq
    from paper_2609_38477_amd import grid
    wl = synthetic.WORKLOADS["attn4096"]
    W = synthetic.workload_weights(wl)
    blocks = W.reshape(-1, 8)
    nb = len(blocks)
    idx = np.linspace(0, nb - 1, args.sample).round().astype(np.int64)
    sub = np.ascontiguousarray(blocks[idx])
    ww = (sub.astype(np.float64) ** 2).sum(axis=1)
    d = torch.from_numpy(W).cuda()
    bad = 0
    for K, P in grid.PAPER_GRID:
        b = sq.build_bases(K, P)
        seed, e, q, err = sq.compress(d, [b])
        seed = seed.cpu().numpy().view(np.uint32)[idx].astype(np.int64)
        e = e.cpu().numpy()[idx].astype(np.int64)
        q = q.cpu().numpy()[idx, :P].astype(np.int64)
        err = err.cpu().numpy()[idx].astype(np.float64)
        del b
        ref = oracle.search(sub, K, P, threads=args.threads)
        oracle.clear_pinv_cache()
        mine = np.array([oracle.code_error(sub[i], K, P, int(seed[i]), int(e[i]), q[i])
                         for i in range(len(sub))])
        within = mine <= ref.err * (1 + REL) + TAU * ww
        reported = np.abs(err - mine) <= 1e-6 * mine + 1e-30
        same = seed == ref.seed
        ok = bool(within.all() and reported.all())
        bad += not ok
        print(json.dumps({"rung": [K, P], "blocks": len(sub), "within_bar": int(within.sum()),
                          "reported_exact": int(reported.sum()), "same_seed": int(same.sum()),
                          "ok": ok}), flush=True)
    print(json.dumps({"rungs": len(grid.PAPER_GRID), "failed": bad}), flush=True)
    return 1 if bad else 0


if __name__ == "__main__":
    sys.exit(main())
