"""The search of a whole multi-rung layer is a pure function of its inputs (a
one-off check at full size; the suite checks the same on smaller cases): the
codes and errors of one compress call over every block are bit-identical to
those of a second call, of calls with other seed-chunk lengths (one walk, and
chunks of 512 seed tiles), of the allocation-free entry point, and of the layer
streamed from host memory in 7 uneven row tiles.

    python3 tests/invariance_check.py [--workload l70b]

Prints one JSON line; exits non-zero if any run differs."""
import argparse
import json
import os
import sys

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

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
    d_rob = torch.from_numpy(rob).cuda() if len(wl.rungs) > 1 else None
    bases = [sq.build_bases(K, P) for K, P in wl.rungs]
    dW = torch.from_numpy(W).cuda()

    def host(out):
        torch.cuda.synchronize()
        return [t.cpu() for t in out]

    def with_chunks(v):
        old = os.environ.get("SEEDQ_SEED_CHUNK_TILES")
        os.environ["SEEDQ_SEED_CHUNK_TILES"] = v
        try:
            return host(sq.compress(dW, bases, rung_of_block=d_rob))
        finally:
            if old is None:
                os.environ.pop("SEEDQ_SEED_CHUNK_TILES")
            else:
                os.environ["SEEDQ_SEED_CHUNK_TILES"] = old

    ref = host(sq.compress(dW, bases, rung_of_block=d_rob))
    runs = {"second call": host(sq.compress(dW, bases, rung_of_block=d_rob)),
            "one walk": with_chunks("0"),
            "chunks of 512 tiles": with_chunks("512")}
    nb = len(rob)
    seed = torch.empty(nb, dtype=torch.int32, device="cuda")
    exp = torch.empty(nb, dtype=torch.uint8, device="cuda")
    q = torch.empty((nb, 8), dtype=torch.int8, device="cuda")
    err = torch.empty(nb, dtype=torch.float32, device="cuda")
    sq.seedq_compress_noalloc(dW, wl.nrows, wl.ncols, 8, d_rob, bases, seed, exp, q, err)
    runs["allocation-free call"] = host((seed, exp, q, err))
    del dW
    runs["7 row tiles from host memory"] = host(
        sq.compress_row_tiles(torch.from_numpy(W).pin_memory(), bases, rung_of_block=d_rob,
                              row_tiles=7))
    same = {k: all(torch.equal(x, y) for x, y in zip(ref, v)) for k, v in runs.items()}
    out = {"workload": wl.name, "blocks": int(nb), "rungs": [list(r) for r in wl.rungs],
           "identical": same, "ok": all(same.values())}
    print(json.dumps(out), flush=True)
    return 0 if out["ok"] else 1


if __name__ == "__main__":
    sys.exit(main())
