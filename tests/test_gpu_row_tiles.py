"""Row tiles (a layer streamed through the GPU in contiguous row ranges from
pinned host memory, two tiles resident at a time) give the codes of one call on
the whole resident matrix, bit for bit: blocks are independent once the rungs
are planned for the whole layer (section 3.4), so each tile is one
seedq_compress call on its rows and its slice of the rung array."""
import numpy as np
import pytest

import synthetic

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sq():
    import paper_2609_38477_amd as sq
    sq.lib()
    return sq


@pytest.mark.parametrize("tiles", [1, 3, 7, 60])
def test_row_tiles_equal_one_call(sq, tiles):
    import torch
    rungs = ((10, 2), (12, 3), (17, 4))
    damage = (4.0, 1.0, 0.25)
    nrows, ncols = 60, 8 * 300
    print(f"row tiles: {tiles} over {nrows}x{ncols}, rungs {rungs}", flush=True)
    a = synthetic.importance_profile(ncols)
    # 3.5 bits per weight: 4050 / 11250 / 2700 blocks and a tie split of 30 blocks
    rob, rep = sq.plan_schedule(nrows, ncols, rungs, damage, 3.5, a)
    assert all(c > 0 for c in rep["count"]) and rep["tie_count"] > 0
    W = synthetic.weights(nrows, ncols, 0.02, key=600 + tiles, outlier_frac=0.01)
    W[7, 16:24] = 0.0
    bases = [sq.build_bases(K, P) for K, P in rungs]
    d_rob = torch.from_numpy(rob).cuda()
    ref = sq.compress(torch.from_numpy(W).cuda(), bases, rung_of_block=d_rob)
    W_host = torch.from_numpy(W).pin_memory()
    got = sq.compress_row_tiles(W_host, bases, rung_of_block=d_rob, row_tiles=tiles)
    torch.cuda.synchronize()
    for x, y, name in zip(got, ref, ("seed", "exp", "q", "err")):
        assert torch.equal(x, y), (tiles, name)
