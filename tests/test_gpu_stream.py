"""GPU code stream through the C ABI against the stream oracle.

Bars: packed words, parsed codes and reconstructed weights are bit-exact
(integer and byte work); NaN marks exactly the blocks the contract names."""
import os

import numpy as np
import pytest

import synthetic
from oracle import stream as ostream

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "stream_three_blocks.txt")
MIXED = [(8, 1), (12, 2), (16, 3), (20, 4), (24, 6)]


@pytest.fixture(scope="module")
def sq():
    import paper_2609_38477_amd as sq
    sq.lib()
    return sq


def _t(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _codes(rng, rob, rungs):
    nb = len(rob)
    seed = np.array([int(rng.integers(1, 1 << rungs[r][0])) if r < len(rungs) else 0 for r in rob],
                    dtype=np.uint32)
    exp = rng.integers(0, 16, nb).astype(np.uint8)
    q = np.zeros((nb, 8), dtype=np.int8)
    for b in range(nb):
        if rob[b] < len(rungs):
            q[b, :rungs[rob[b]][1]] = rng.integers(-8, 8, rungs[rob[b]][1])
    return seed, exp, q


def _words(t):
    return t.cpu().numpy().view(np.uint32)


def test_pack_and_unpack_hand_derived_payload(sq):
    rob = np.array([0, 1, 0], dtype=np.uint8)
    rungs = [(8, 2), (9, 3)]
    seed = np.array([0xA5, 0x1C3, 0x01], dtype=np.uint32)
    exp = np.array([3, 9, 15], dtype=np.uint8)
    q = np.zeros((3, 8), dtype=np.int8)
    q[0, :2], q[1, :3], q[2, :2] = (-1, 5), (7, -8, 0), (2, -3)
    gold = np.array([0x3C35F3A5, 0xA5E0210F, 0x00000001], dtype=np.uint32)
    w = sq.pack(_t(seed.view(np.int32)), _t(exp), _t(q), rungs, 1, 24, _t(rob), [2, 1])
    assert np.array_equal(_words(w), gold)
    s, e, qq = sq.unpack(_t(gold.view(np.int32)), rungs, 1, 24, _t(rob))
    assert np.array_equal(s.cpu().numpy().view(np.uint32), seed)
    assert np.array_equal(e.cpu().numpy(), exp) and np.array_equal(qq.cpu().numpy(), q)


@pytest.mark.parametrize("shape", [(5, 8000), (1, 8), (3, 16392), (2, 32768)])
def test_pack_matches_oracle_mixed_rungs(sq, oq, shape):
    # several chunks of 2048 blocks with a ragged tail, every rung width, and
    # blocks with an out-of-range rung index (no bits, seed 0 / NaN on decode)
    nrows, ncols = shape
    nb = nrows * ncols // 8
    rng = np.random.default_rng(nb)
    rob = rng.integers(0, len(MIXED), nb).astype(np.uint8)
    rob[rng.random(nb) < 0.02] = 7
    seed, exp, q = _codes(rng, rob, MIXED)
    valid = rob < len(MIXED)
    ref = ostream.pack(seed[valid], exp[valid], q[valid], rob[valid], MIXED)
    cnt = np.bincount(rob[valid], minlength=len(MIXED))
    w = sq.pack(_t(seed.view(np.int32)), _t(exp), _t(q), MIXED, nrows, ncols, _t(rob), cnt)
    assert np.array_equal(_words(w), ref)
    s, e, qq = sq.unpack(w, MIXED, nrows, ncols, _t(rob))
    s, e, qq = s.cpu().numpy().view(np.uint32), e.cpu().numpy(), qq.cpu().numpy()
    assert np.array_equal(s[valid], seed[valid]) and np.array_equal(e[valid], exp[valid])
    assert np.array_equal(qq[valid], q[valid])
    assert np.all(s[~valid] == 0) and np.all(e[~valid] == 0) and np.all(qq[~valid] == 0)
    # one-pass decode equals parse + reconstruct, and the oracle's reconstruction
    Wh = sq.decompress_stream(w, MIXED, nrows, ncols, _t(rob)).cpu().numpy().reshape(-1, 8)
    K_of = np.array([MIXED[r][0] if r < len(MIXED) else 8 for r in rob])
    P_of = np.array([MIXED[r][1] if r < len(MIXED) else 1 for r in rob])
    idx = np.nonzero(valid)[0][:: max(1, nb // 3000)]
    ref_w, _ = oq.decompress(seed[idx], exp[idx], q[idx], K_of[idx], P_of[idx])
    assert np.array_equal(Wh[idx], np.asarray(ref_w, dtype=np.float32).reshape(-1, 8))
    assert np.all(np.isnan(Wh[~valid]))


def test_short_stream_marks_only_the_blocks_past_its_end(sq):
    nrows, ncols = 2, 8 * 3000
    nb = nrows * ncols // 8
    rng = np.random.default_rng(9)
    rob = rng.integers(0, len(MIXED), nb).astype(np.uint8)
    seed, exp, q = _codes(rng, rob, MIXED)
    cnt = np.bincount(rob, minlength=len(MIXED))
    w = sq.pack(_t(seed.view(np.int32)), _t(exp), _t(q), MIXED, nrows, ncols, _t(rob), cnt)
    cut = w[: w.numel() // 2]
    s, e, qq = sq.unpack(cut, MIXED, nrows, ncols, _t(rob))
    s = s.cpu().numpy().view(np.uint32)
    ends = np.cumsum([MIXED[r][0] + 4 + 4 * MIXED[r][1] for r in rob])
    inside = ends <= 32 * cut.numel()
    assert inside.any() and (~inside).any()
    assert np.array_equal(s[inside], seed[inside]) and np.all(s[~inside] == 0)
    Wh = sq.decompress_stream(cut, MIXED, nrows, ncols, _t(rob)).cpu().numpy().reshape(-1, 8)
    assert not np.isnan(Wh[inside]).any() and np.isnan(Wh[~inside]).all()


def test_full_size_round_trip_from_the_search(sq):
    # attn4096: real codes from the search, payload of exactly 32 bits per block
    import torch
    wl = synthetic.WORKLOADS["attn4096"]
    W = torch.from_numpy(synthetic.workload_weights(wl)).cuda()
    b = sq.build_bases(16, 3)
    seed, exp, q, _ = sq.compress(W, [b])
    w = sq.pack(seed, exp, q, [(16, 3)], wl.nrows, wl.ncols)
    assert w.numel() == wl.nblocks
    s, e, qq = sq.unpack(w, [(16, 3)], wl.nrows, wl.ncols)
    assert torch.equal(s, seed) and torch.equal(e, exp) and torch.equal(qq, q)
    W1, _ = sq.decompress(seed, exp, q, [(16, 3)], wl.nrows, wl.ncols)
    W2 = sq.decompress_stream(w, [(16, 3)], wl.nrows, wl.ncols)
    assert torch.equal(W1, W2)


def test_decoder_path_with_rederived_rungs(sq):
    # encoder: plan, search, pack; decoder: re-derive the rungs from the stored
    # lambda / floor / tie count, then parse and reconstruct in one pass
    import torch
    wl = synthetic.WORKLOADS["reduced"]
    nrows = 64
    a = synthetic.importance_profile(wl.ncols)
    W = synthetic.weights(nrows, wl.ncols, wl.sigma, 21, wl.outlier_frac)
    rob, rep = sq.plan_schedule(nrows, wl.ncols, wl.rungs, wl.damage, 3.296875, a, None, 0.06)
    assert rep["tie_count"] > 0
    bases = [sq.build_bases(K, P) for K, P in wl.rungs]
    seed, exp, q, _ = sq.compress(_t(W), bases, _t(rob))
    words = sq.pack(seed, exp, q, list(wl.rungs), nrows, wl.ncols, _t(rob), rep["count"])
    dec_rob = sq.derive_schedule(nrows, wl.ncols, wl.rungs, wl.damage, a, rep["lam"], rep["floor_q"],
                                 rep["tie_count"])
    assert np.array_equal(dec_rob, rob)
    Wd = sq.decompress_stream(words, list(wl.rungs), nrows, wl.ncols, _t(dec_rob))
    Wr, _ = sq.decompress(seed, exp, q, list(wl.rungs), nrows, wl.ncols, _t(rob))
    assert torch.equal(Wd, Wr)


def _gemv_bound(W, x):
    # fp32 accumulation, by the kernel that runs for x's number of vectors
    # (G = ncols / 8). Up to four: a lane adds at most ceil(G / 64) block
    # partials, each a chain of 8 fused products, then a 6-level tree: bound
    # (8 ceil(G / 64) + 8) u sum |w||x|. Eight (matrix core): a product passes
    # through at most 8 accumulations of 4 products in its 64-block step
    # (1 + 4 + 7 x 4 roundings), one addition per step and a sum of 16:
    # (50 + ceil(G / 64)) u sum |w||x|
    ncols = W.shape[1]
    G = ncols // 8
    n = 50 + (G + 63) // 64 if x.shape[0] >= 8 else (G + 63) // 64 * 8 + 8
    return n * 2.0 ** -24 * (np.abs(W.astype(np.float64)) @ np.abs(x.astype(np.float64)).T)


@pytest.mark.parametrize("nvec", [1, 2, 4, 8])
def test_gemv_stream_matches_oracle(sq, oq, nvec):
    import torch
    nrows, ncols = 37, 8 * 301                 # rows of 301 blocks: 4 lane rounds + a tail
    nb = nrows * ncols // 8
    rng = np.random.default_rng(40 + nvec)
    rob = rng.integers(0, len(MIXED), nb).astype(np.uint8)
    seed, exp, q = _codes(rng, rob, MIXED)
    cnt = np.bincount(rob, minlength=len(MIXED))
    w = sq.pack(_t(seed.view(np.int32)), _t(exp), _t(q), MIXED, nrows, ncols, _t(rob), cnt)
    x = rng.normal(0, 1, (nvec, ncols)).astype(np.float32)
    y = sq.gemv_stream(w, MIXED, nrows, ncols, _t(x), _t(rob)).cpu().numpy()
    K_of = np.array([MIXED[r][0] for r in rob])
    P_of = np.array([MIXED[r][1] for r in rob])
    Wr, _ = oq.decompress(seed, exp, q, K_of, P_of)
    Wr = np.asarray(Wr, dtype=np.float32).reshape(nrows, ncols)
    ref = (Wr.astype(np.float64) @ x.astype(np.float64).T).T
    assert np.all(np.abs(y - ref) <= _gemv_bound(Wr, x).T + 1e-30)


def _blocky_rungs(rng, nrows, G, R):
    # per row, each 64-block wave step is one rung (7 in 10) or mixed; the
    # decode-GEMV takes its one-rung path for the former
    rob = np.empty((nrows, G), dtype=np.uint8)
    for r in range(nrows):
        for g0 in range(0, G, 64):
            n = min(64, G - g0)
            if rng.random() < 0.7:
                rob[r, g0:g0 + n] = rng.integers(0, R)
            else:
                rob[r, g0:g0 + n] = rng.integers(0, R, n)
    return rob.reshape(-1)


@pytest.mark.parametrize("rungs", [
    [(12, 2), (16, 3), (20, 4)],                  # leap tables at K = 12 and 16, LFSR at 20
    [(8, 1), (13, 3), (16, 6), (23, 5), (24, 6)],  # (16, 6) past the LDS budget, K = 24
    [(16, 6)],                                     # leap tables, P = 6
    [(10, 5), (15, 1)],                            # leap tables, odd P
])
@pytest.mark.parametrize("nvec", [1, 4, 8])
def test_gemv_stream_one_rung_steps(sq, oq, rungs, nvec):
    nrows, ncols = 23, 8 * 301                 # 4 full wave steps + a 45-block tail
    nb = nrows * ncols // 8
    rng = np.random.default_rng(len(rungs) * 10 + nvec)
    rob = _blocky_rungs(rng, nrows, ncols // 8, len(rungs))
    seed, exp, q = _codes(rng, rob, rungs)
    G = ncols // 8
    seed[2 * G + 5] = seed[11 * G + 290] = 0     # invalid seeds poison their rows
    cnt = np.bincount(rob, minlength=len(rungs))
    w = sq.pack(_t(seed.view(np.int32)), _t(exp), _t(q), rungs, nrows, ncols, _t(rob), cnt)
    x = rng.normal(0, 1, (nvec, ncols)).astype(np.float32)
    y = sq.gemv_stream(w, rungs, nrows, ncols, _t(x), _t(rob)).cpu().numpy()
    K_of = np.array([rungs[r][0] for r in rob])
    P_of = np.array([rungs[r][1] for r in rob])
    Wr, _ = oq.decompress(np.where(seed == 0, 1, seed), exp, q, K_of, P_of)
    Wr = np.asarray(Wr, dtype=np.float32).reshape(nrows, ncols)
    bad = (seed == 0).reshape(nrows, -1).any(axis=1)
    assert bad.any() and not bad.all()
    assert np.isnan(y[:, bad]).all() and not np.isnan(y[:, ~bad]).any()
    Wg = Wr[~bad]
    ref = (Wg.astype(np.float64) @ x.astype(np.float64).T).T
    assert np.all(np.abs(y[:, ~bad] - ref) <= _gemv_bound(Wg, x).T + 1e-30)


@pytest.mark.parametrize("nrows,G", [(1, 1), (3, 1), (1, 65), (2, 64), (5, 257)])
@pytest.mark.parametrize("nvec", [1, 8])
def test_gemv_stream_edge_shapes(sq, oq, nrows, G, nvec):
    # one block per row, one lane of a wave step, exactly one or one past a
    # whole step, and a step of four sub-steps plus one block
    ncols = 8 * G
    nb = nrows * G
    rng = np.random.default_rng(1000 * nrows + G + nvec)
    rob = rng.integers(0, len(MIXED), nb).astype(np.uint8)
    seed, exp, q = _codes(rng, rob, MIXED)
    cnt = np.bincount(rob, minlength=len(MIXED))
    w = sq.pack(_t(seed.view(np.int32)), _t(exp), _t(q), MIXED, nrows, ncols, _t(rob), cnt)
    x = rng.normal(0, 1, (nvec, ncols)).astype(np.float32)
    y = sq.gemv_stream(w, MIXED, nrows, ncols, _t(x), _t(rob)).cpu().numpy()
    K_of = np.array([MIXED[r][0] for r in rob])
    P_of = np.array([MIXED[r][1] for r in rob])
    Wr, _ = oq.decompress(seed, exp, q, K_of, P_of)
    Wr = np.asarray(Wr, dtype=np.float32).reshape(nrows, ncols)
    ref = (Wr.astype(np.float64) @ x.astype(np.float64).T).T
    assert y.shape == (nvec, nrows)
    assert np.all(np.abs(y - ref) <= _gemv_bound(Wr, x).T + 1e-30)


@pytest.mark.parametrize("nvec", [1, 8])
def test_gemv_stream_invalid_block_poisons_its_row(sq, nvec):
    nrows, ncols = 6, 8 * 70
    nb = nrows * ncols // 8
    rng = np.random.default_rng(77)
    rob = rng.integers(0, len(MIXED), nb).astype(np.uint8)
    rob[3 * 70 + 5] = 7                          # out-of-range rung in row 3
    seed, exp, q = _codes(rng, rob, MIXED)
    valid = rob < len(MIXED)
    cnt = np.bincount(rob[valid], minlength=len(MIXED))
    w = sq.pack(_t(seed.view(np.int32)), _t(exp), _t(q), MIXED, nrows, ncols, _t(rob), cnt)
    x = rng.normal(0, 1, (nvec, ncols)).astype(np.float32)
    y = sq.gemv_stream(w, MIXED, nrows, ncols, _t(x), _t(rob)).cpu().numpy().reshape(nvec, nrows)
    assert np.isnan(y[:, 3]).all() and not np.isnan(np.delete(y, 3, axis=1)).any()


def test_gemv_stream_full_size(sq):
    import torch
    wl = synthetic.WORKLOADS["attn4096"]
    W = torch.from_numpy(synthetic.workload_weights(wl)).cuda()
    b = sq.build_bases(16, 3)
    seed, exp, q, _ = sq.compress(W, [b])
    w = sq.pack(seed, exp, q, [(16, 3)], wl.nrows, wl.ncols)
    Wh, _ = sq.decompress(seed, exp, q, [(16, 3)], wl.nrows, wl.ncols)
    g = torch.Generator(device="cuda").manual_seed(3)
    x = torch.randn(4, wl.ncols, device="cuda", generator=g)
    y = sq.gemv_stream(w, [(16, 3)], wl.nrows, wl.ncols, x).cpu().numpy()
    Wn, xn = Wh.cpu().numpy(), x.cpu().numpy()
    ref = (Wn.astype(np.float64) @ xn.astype(np.float64).T).T
    assert np.all(np.abs(y - ref) <= _gemv_bound(Wn, xn).T)


def test_stream_largest_block_count(sq, oq):
    # 32768 x 524280 = 2^31 - 32768 blocks at two rungs (16 and 24 bits each, so
    # about 4.3e10 stream bits, far past 2^32): random codes drawn on the GPU;
    # pack then unpack returns every code, the one-pass decode equals the decode
    # from code arrays bit for bit, a window of stream bits near the end equals
    # the oracle packer's bits for the same blocks, and sampled rows of the
    # decode-GEMV match the oracle's reconstruction times x in fp64
    import torch
    nrows, ncols = 32768, 524280
    nb = nrows * (ncols // 8)
    rungs = [(8, 1), (12, 2)]
    g = torch.Generator(device="cuda").manual_seed(32)
    rob = torch.randint(0, 2, (nb,), dtype=torch.uint8, device="cuda", generator=g)
    seed = torch.randint(1, 1 << 8, (nb,), dtype=torch.int32, device="cuda", generator=g)
    hi = torch.randint(1, 1 << 12, (nb,), dtype=torch.int32, device="cuda", generator=g)
    sel = rob.bool()
    seed = torch.where(sel, hi, seed)
    del hi
    exp = torch.randint(0, 16, (nb,), dtype=torch.uint8, device="cuda", generator=g)
    q = torch.zeros((nb, 8), dtype=torch.int8, device="cuda")
    q[:, 0] = torch.randint(-8, 8, (nb,), dtype=torch.int8, device="cuda", generator=g)
    q[:, 1] = torch.randint(-8, 8, (nb,), dtype=torch.int8, device="cuda", generator=g) * sel
    del sel
    n1 = int(rob.sum(dtype=torch.int64))
    cnt = [nb - n1, n1]
    w = sq.pack(seed, exp, q, rungs, nrows, ncols, rob, cnt)
    assert w.numel() * 32 >= 16 * (nb - n1) + 24 * n1 > (1 << 32)
    s2, e2, q2 = sq.unpack(w, rungs, nrows, ncols, rob)
    assert torch.equal(s2, seed) and torch.equal(e2, exp) and torch.equal(q2, q)
    del s2, e2, q2
    W1 = sq.decompress_stream(w, rungs, nrows, ncols, rob)
    W2, _ = sq.decompress(seed, exp, q, rungs, nrows, ncols, rung_of_block=rob)
    assert torch.equal(W1.view(torch.int32), W2.view(torch.int32))
    del W2
    # a window of 1000 blocks near the end against the oracle's packer
    b0, b1 = nb - 1100, nb - 100
    pre1 = int(rob[:b0].sum(dtype=torch.int64))
    off = 16 * (b0 - pre1) + 24 * pre1
    rw = rob[b0:b1].cpu().numpy()
    ref = ostream.pack(seed[b0:b1].cpu().numpy().view(np.uint32), exp[b0:b1].cpu().numpy(),
                       q[b0:b1].cpu().numpy(), rw, rungs)
    L = int(16 * np.count_nonzero(rw == 0) + 24 * np.count_nonzero(rw == 1))
    words = _words(w[off // 32: (off + L) // 32 + 1])
    bits = np.unpackbits(words.view(np.uint8), bitorder="little")[off % 32: off % 32 + L]
    ref_bits = np.unpackbits(ref.view(np.uint8), bitorder="little")[:L]
    assert np.array_equal(bits, ref_bits)
    # sampled blocks of the decode against the oracle's reconstruction
    idx = torch.from_numpy(np.concatenate([np.linspace(0, nb - 1, 512).astype(np.int64),
                                           np.arange(nb - 64, nb)])).cuda()
    r_of = rob[idx].cpu().numpy()
    Ks = np.array([rungs[r][0] for r in r_of])
    Ps = np.array([rungs[r][1] for r in r_of])
    ref_w, _ = oq.decompress(seed[idx].cpu().numpy().view(np.uint32), exp[idx].cpu().numpy(),
                             q[idx].cpu().numpy(), Ks, Ps)
    assert np.array_equal(W1.view(-1, 8)[idx].cpu().numpy().view(np.uint32), ref_w.view(np.uint32))
    del W1
    torch.cuda.empty_cache()
    # decode-GEMV, three sampled rows against the oracle in fp64
    x = torch.randn(ncols, device="cuda", generator=g)
    y = sq.gemv_stream(w, rungs, nrows, ncols, x, rob).cpu().numpy()
    xn = x.cpu().numpy()
    G = ncols // 8
    for r in (0, nrows // 2, nrows - 1):
        sl = slice(r * G, (r + 1) * G)
        rr = rob[sl].cpu().numpy()
        Wr, _ = oq.decompress(seed[sl].cpu().numpy().view(np.uint32), exp[sl].cpu().numpy(),
                              q[sl].cpu().numpy(), np.array([rungs[k][0] for k in rr]),
                              np.array([rungs[k][1] for k in rr]))
        Wr = np.asarray(Wr, dtype=np.float32).reshape(1, ncols)
        ref_y = float((Wr.astype(np.float64) @ xn.astype(np.float64))[0])
        assert abs(float(y[r]) - ref_y) <= float(_gemv_bound(Wr, xn[None, :])[0, 0]), r
    del w, seed, exp, q, rob, x
    torch.cuda.empty_cache()
