"""The allocation-free compress call against seedq_compress, through the C ABI.

seedq_compress_noalloc keeps the block lists of a multi-rung call in a fixed
device array instead of a caller workspace and runs the same kernels, so its
codes and errors must equal seedq_compress's bit for bit. Two multi-rung calls
in a row, the second smaller than the first (the array still holds the first
call's lists), then a single-rung call; the second multi-rung call is also
checked against the oracle's exhaustive search.
"""
import numpy as np
import pytest

import synthetic

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sq():
    import paper_2609_38477_amd as sq
    sq.lib()
    return sq


@pytest.fixture(scope="module")
def torch():
    import torch
    assert torch.cuda.is_available()
    return torch


def _dev(torch, a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _noalloc(sq, torch, dW, bases, rob):
    nrows, ncols = dW.shape
    nb = nrows * ncols // 8
    seed = torch.empty(nb, dtype=torch.int32, device="cuda")
    exp = torch.empty(nb, dtype=torch.uint8, device="cuda")
    q = torch.empty((nb, 8), dtype=torch.int8, device="cuda")
    err = torch.empty(nb, dtype=torch.float32, device="cuda")
    sq.seedq_compress_noalloc(dW, nrows, ncols, 8, rob, bases, seed, exp, q, err)
    return seed, exp, q, err


def _case(key, nrows, ngroups, nrungs):
    W = synthetic.weights(nrows, 8 * ngroups, 0.02, key=key, outlier_frac=0.02)
    W[nrows // 2, 16:24] = 0.0   # an all-zero block
    nb = nrows * ngroups
    rob = (synthetic.splitmix64(key, synthetic.STREAM_MISC, nb) % np.uint64(nrungs)).astype(np.uint8)
    return W, rob


def test_noalloc_equals_compress_on_two_calls_in_a_row(sq, oq, torch):
    from test_gpu_parity import check_search
    # first call: 12 rows x 1024 groups = 12288 blocks (six compaction chunks),
    # three rungs, the K = 17 one walked in sequential seed chunks
    rungs1 = ((10, 2), (12, 3), (17, 3))
    W1, rob1 = _case(701, 12, 1024, len(rungs1))
    # second call: 485 blocks (a ragged tail), other rungs and another split
    rungs2 = ((8, 2), (11, 4), (9, 5))
    W2, rob2 = _case(702, 5, 97, len(rungs2))
    for W, rob, rungs, label in ((W1, rob1, rungs1, "first"), (W2, rob2, rungs2, "second")):
        print(f"noalloc {label} call: {W.shape}, rungs {rungs}", flush=True)
        bases = [sq.build_bases(K, P) for K, P in rungs]
        dW, drob = _dev(torch, W), _dev(torch, rob)
        got = _noalloc(sq, torch, dW, bases, drob)
        ref = sq.compress(dW, bases, rung_of_block=drob)
        torch.cuda.synchronize()
        for a, b, name in zip(got, ref, ("seed", "exp", "q", "err")):
            assert torch.equal(a, b), (label, name)
    # the second call's codes meet the oracle bar rung by rung
    seed, e, q, err = (t.cpu().numpy() for t in got)
    blocks = W2.reshape(-1, 8)
    for r, (K, P) in enumerate(rungs2):
        sel = np.nonzero(rob2 == r)[0]
        check_search(oq, blocks[sel], K, P, seed[sel].view(np.uint32), e[sel], q[sel], err[sel],
                     f"noalloc rung{r}")


def test_noalloc_single_rung_needs_no_scratch(sq, torch):
    K, P = 12, 3
    W = synthetic.weights(4, 8 * 200, 0.02, key=703, outlier_frac=0.02)
    b = [sq.build_bases(K, P)]
    dW = _dev(torch, W)
    got = _noalloc(sq, torch, dW, b, None)
    ref = sq.compress(dW, b)
    torch.cuda.synchronize()
    for a, c in zip(got, ref):
        assert torch.equal(a, c)
