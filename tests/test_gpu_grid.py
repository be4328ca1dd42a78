"""GPU rung-grid build (one uniform search per rung through the C ABI) against
the CPU oracle's exhaustive search at every rung.

Bar: for every block and rung the GPU's reported error is within 1e-5 relative
(plus 1e-7 ||w||^2) of the oracle's best error, which makes the ratio summary
of Table rungshape agree to the same relative precision."""
import numpy as np
import pytest

import synthetic

pytestmark = pytest.mark.gpu

RUNGS = ((8, 2), (9, 3), (10, 4), (11, 5), (12, 6), (12, 3), (10, 3))


def test_grid_errors_match_oracle(oq):
    import torch
    from paper_2609_38477_amd import grid
    W = synthetic.weights(24, 64, 0.02, 11, 0.01)       # 192 blocks incl. outliers
    W[3, 8:16] = 0.0                                     # one all-zero block
    res = grid.build_grid(torch.from_numpy(W).cuda(), rungs=RUNGS)
    blocks = W.reshape(-1, 8)
    ww = (blocks.astype(np.float64) ** 2).sum(axis=1)
    ref_err = {}
    for K, P in RUNGS:
        ref = oq.search(blocks, K, P)
        got = res.err[(K, P)].cpu().numpy().astype(np.float64)
        assert np.all(np.abs(got - ref.err) <= 1e-5 * ref.err + 1e-7 * ww), (K, P)
        assert got[3 * 8 + 1] == 0.0
        ref_err[(K, P)] = ref.err
        assert res.search_ms[(K, P)] > 0 and res.bases_ms[(K, P)] > 0
    rows = [((10, 3),), ((12, 6),), ((8, 2),)]
    for rr in rows:
        a = grid.rungshape(res.err, rungs=rr, ref=(12, 3))[0]
        b = grid.rungshape(ref_err, rungs=rr, ref=(12, 3))[0]
        assert a["blocks"] == b["blocks"] == len(blocks) - 1
        for k in ("median", "q10", "q90"):
            assert abs(a[k] - b[k]) <= 1e-4 * b[k], (rr, k)
        assert abs(a["sd_log"] - b["sd_log"]) <= 1e-4
