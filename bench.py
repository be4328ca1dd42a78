#!/usr/bin/env python3
"""Throughput of the Seed-Q per-block seed search on one MI355X.

One step = the whole hot path over one synthetic weight matrix already resident
in HBM: rung schedule (host), basis stacks for every rung, the exhaustive seed
search of every block, and the verification decompress. The headline number is
block*seed candidates per second (sum over blocks of 2^K - 1, divided by the
step time). Prints one JSON line on stdout; progress goes to stderr.

  python bench.py [--steps K] [--warmup W] [--workload attn4096] [--gpus 1]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "block·seed candidates/sec at K=16, C=8; % MFMA roofline; 1 GPU"

# MI355X published peaks
PEAK_HBM_GBS = 8000.0
PEAK_FP16_MFMA_TFLOPS = 2500.0   # dense fp16 matrix-core peak
PEAK_FP32_MFMA_TFLOPS = 157.3    # dense fp32 matrix-core peak

PROFILE_DIR = os.path.join(ROOT, "profiles")
TRAFFIC_FILE = os.path.join(PROFILE_DIR, "search_attn4096_traffic.json")
KERNEL_SOURCES = ["seedq_search_mfma.hip", "seedq_exact.h", "seedq_internal.h"]


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


# Roofline work of the search (the least-squares projection of every block on
# every seed's basis): 2 C P flops per (block, seed) candidate, i.e. 48 at
# P = 3, priced against the dense fp16 matrix-core peak because the contraction
# the kernel issues is fp16. Two other counts are reported beside it under
# their own keys: the kernel's quadratic form over the 36 pair products of a
# block (72 flops per candidate at every P) and what it issues (the 36 pairs
# padded to 48 reduction slots: 96 flops per candidate).
def projection_flops(K: int, P: int) -> float:
    return float((1 << K) - 1) * 2 * 8 * P


QUADFORM_FLOPS_PER_CANDIDATE = 72.0
ISSUED_FLOPS_PER_CANDIDATE = 96.0


def kernel_source_hash() -> str:
    import hashlib
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2609_38477_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(workload: str):
    """HBM bytes per search launch from the committed counter summary, or None
    when it was taken on another workload or an older kernel source."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("workload") != workload or rec.get("kernel_source_sha256") != kernel_source_hash():
        return None
    return float(rec["traffic_bytes_per_launch"])


def practical_mfma_tflops(n: int = 16384, reps: int = 5) -> float:
    """fp16 matrix-core rate a vendor GEMM (torch.matmul -> hipBLASLt) reaches on
    this GPU with random N(0, 1) operands: the clock of the chip drops under
    dense random-data matrix work, so this rate, not the published peak, is what
    a matrix-core-bound kernel can approach. Measurement context only."""
    import torch
    g = torch.Generator(device="cuda").manual_seed(0)
    a = torch.randn(n, n, device="cuda", dtype=torch.float16, generator=g)
    b = torch.randn(n, n, device="cuda", dtype=torch.float16, generator=g)
    for _ in range(2):
        c = a @ b
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        c = a @ b
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / reps
    del a, b, c
    return 2.0 * n ** 3 / dt / 1e12


def cpu_baseline(W: np.ndarray, K: int, P: int, target_s: float = 15.0) -> dict:
    import oracle
    blocks = W.reshape(-1, 8)
    threads = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    pinv = oracle.cached_pinv_stack(K, P)
    # calibrate on a few blocks, then run a bounded evenly spaced sample
    cal = blocks[:: max(1, len(blocks) // 16)][:16]
    t0 = time.perf_counter()
    oracle.search(cal, K, P, threads=threads, pinv=pinv)
    rate = len(cal) * ((1 << K) - 1) / (time.perf_counter() - t0)
    n = int(min(len(blocks), max(16, target_s * rate / ((1 << K) - 1))))
    idx = np.linspace(0, len(blocks) - 1, n).astype(np.int64)
    sample = np.ascontiguousarray(blocks[idx])
    t0 = time.perf_counter()
    oracle.search(sample, K, P, threads=threads, pinv=pinv)
    dt = time.perf_counter() - t0
    cands = n * ((1 << K) - 1)
    # the same oracle on one thread, over a smaller evenly spaced sample (~3 s)
    n1 = int(min(len(blocks), max(4, 3.0 * rate / threads / ((1 << K) - 1))))
    s1 = np.ascontiguousarray(blocks[np.linspace(0, len(blocks) - 1, n1).astype(np.int64)])
    t0 = time.perf_counter()
    oracle.search(s1, K, P, threads=1, pinv=pinv)
    rate1 = n1 * ((1 << K) - 1) / (time.perf_counter() - t0)
    return {"value": cands / dt, "unit": "block·seed candidates/s", "cores": int(threads),
            "value_one_thread": rate1,
            "kind": "oracle",
            "sample": f"{n} evenly spaced blocks of the same matrix at (K={K}, P={P}), "
                      f"{cands:.3g} candidates in {dt:.1f} s; one thread: {n1} blocks; per-seed "
                      f"pseudo-inverses precomputed outside the timed region"}


def decoder_bench(args) -> int:
    """Decoder path on a searched matrix: host re-derivation of the rungs from
    the stored lambda / floor / tie count, GPU pack, parse, one-pass decode, and
    decode-GEMV against a dense GEMV of the decoded weights. Every GPU time is
    the mean over the timed repetitions of HIP events on the kernels' stream."""
    import torch

    import paper_2609_38477_amd as sq
    import synthetic

    wl = synthetic.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    rungs = list(wl.rungs)
    R = len(rungs)
    a = synthetic.importance_profile(wl.ncols)
    log(f"decoder bench on {wl.name}: {wl.note}")
    W = torch.from_numpy(synthetic.workload_weights(wl)).to(dev)
    nb = wl.nblocks
    rob, rep = sq.plan_schedule(wl.nrows, wl.ncols, rungs, wl.damage, wl.target_bpw, a)
    d_rob = torch.from_numpy(rob).to(dev) if R > 1 else None
    bases = [sq.build_bases(K, P) for K, P in rungs]
    seed, exp, q, _ = sq.compress(W, bases, d_rob)
    counts = rep["count"]
    nbytes = sq.seedq_stream_bytes(rungs, counts)
    words = torch.empty(nbytes // 4, dtype=torch.int32, device=dev)
    nws = sq.seedq_stream_workspace_bytes(wl.nrows, wl.ncols)
    ws = torch.empty(nws, dtype=torch.uint8, device=dev)
    s2 = torch.empty_like(seed)
    e2 = torch.empty_like(exp)
    q2 = torch.empty_like(q)
    W_hat = torch.empty_like(W)
    g = torch.Generator(device="cuda").manual_seed(0)
    xs = {nv: torch.randn(nv, wl.ncols, device=dev, generator=g) for nv in (1, 4, 8)}
    ys = {nv: torch.empty(nv, wl.nrows, device=dev) for nv in (1, 4, 8)}
    rung_arg = d_rob if R > 1 else None

    def timed(fn, reps):
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ev[0].record(stream)
        for _ in range(reps):
            fn()
        ev[1].record(stream)
        torch.cuda.synchronize()
        return ev[0].elapsed_time(ev[1]) / reps

    reps = max(args.steps, 5) * 4
    t0 = time.perf_counter()
    for _ in range(3):
        dec_rob = sq.derive_schedule(wl.nrows, wl.ncols, rungs, wl.damage, a, rep["lam"],
                                     rep["floor_q"], rep["tie_count"])
    derive_ms = (time.perf_counter() - t0) / 3 * 1e3
    assert np.array_equal(dec_rob, rob)
    ms = {}
    ms["pack"] = timed(lambda: sq.seedq_pack(seed, exp, q, rung_arg, rungs, wl.nrows, wl.ncols, 8,
                                             words, nbytes, ws, nws, stream), reps)
    ms["unpack"] = timed(lambda: sq.seedq_unpack(words, nbytes, rung_arg, rungs, wl.nrows, wl.ncols,
                                                 8, s2, e2, q2, ws, nws, stream), reps)
    ms["decompress_stream"] = timed(lambda: sq.seedq_decompress_stream(
        words, nbytes, rung_arg, rungs, wl.nrows, wl.ncols, 8, W_hat, ws, nws, stream), reps)
    ms["decompress_codes"] = timed(lambda: sq.seedq_decompress(
        seed, exp, q, rung_arg, rungs, wl.nrows, wl.ncols, 8, W_hat, None, stream), reps)
    for nv in (1, 4, 8):
        ms[f"gemv_stream_x{nv}"] = timed(lambda nv=nv: sq.seedq_gemv_stream(
            words, nbytes, rung_arg, rungs, wl.nrows, wl.ncols, 8, nv, xs[nv], ys[nv], ws, nws,
            stream), reps)
    # dense references on the decoded weights (vendor GEMV/GEMM, context only)
    W16 = W_hat.half()
    x16 = {nv: xs[nv].half() for nv in (1, 4, 8)}
    for nv in (1, 4, 8):
        ms[f"dense_fp16_x{nv}"] = timed(lambda nv=nv: torch.matmul(W16, x16[nv].t()), reps)
        ms[f"dense_fp32_x{nv}"] = timed(lambda nv=nv: torch.matmul(W_hat, xs[nv].t()), reps)
    assert torch.equal(s2, seed) and torch.equal(e2, exp)

    stream_b = nbytes
    rung_b = nb if R > 1 else 0
    hbm = {  # algorithmic HBM bytes per launch
        "pack": nb * (4 + 1 + 8) + rung_b + stream_b,
        "unpack": stream_b + rung_b + nb * (4 + 1 + 8),
        "decompress_stream": stream_b + rung_b + nb * 32,
        "decompress_codes": nb * (4 + 1 + 8) + rung_b + nb * 32,
    }
    for nv in (1, 4, 8):
        hbm[f"gemv_stream_x{nv}"] = stream_b + rung_b + 4 * nv * (wl.ncols + wl.nrows)
        hbm[f"dense_fp16_x{nv}"] = 2 * wl.nrows * wl.ncols + 2 * nv * (wl.ncols + wl.nrows)
        hbm[f"dense_fp32_x{nv}"] = 4 * wl.nrows * wl.ncols + 4 * nv * (wl.ncols + wl.nrows)
    kernels = {k: {"ms": v, "hbm_bytes": hbm[k], "GBps": hbm[k] / (v / 1e3) / 1e9,
                   "hbm_frac": hbm[k] / (v / 1e3) / 1e9 / PEAK_HBM_GBS} for k, v in ms.items()}
    if not args.no_cpu_baseline:
        out_cpu = decoder_cpu_baseline(seed, exp, q, rob, rungs, args.cpu_seconds)
    out = {"metric": "decoder path: decoded weights/s and HBM GB/s per kernel; 1 GPU",
           "workload": wl.name, "shape": [wl.nrows, wl.ncols], "nblocks": nb,
           "rungs": [list(r) for r in rungs], "target_bpw": wl.target_bpw,
           "payload_bytes": nbytes, "payload_bits_per_weight": 8.0 * nbytes / (8 * nb),
           "derive_schedule_host_ms": derive_ms, "kernels": kernels,
           "decoded_weights_per_s": {k: 8 * nb / (v / 1e3) for k, v in ms.items()
                                     if k.startswith(("decompress", "gemv"))},
           "data": "synthetic"}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = out_cpu
    print(json.dumps(out), flush=True)
    return 0


def decoder_cpu_baseline(seed, exp, q, rob, rungs, target_s: float) -> dict:
    """The oracle's decoder on the host: the exact reconstruction
    (C, one thread) on an evenly spaced sample of the searched codes, and the
    bit-by-bit stream parser (Python) on a short run of them."""
    import oracle
    from oracle import stream as ostream
    s_ = seed.cpu().numpy().view(np.uint32)
    e_ = exp.cpu().numpy()
    q_ = q.cpu().numpy()
    r_ = np.asarray(rob, dtype=np.uint8)
    Ks = np.array([k for k, _ in rungs], dtype=np.int64)[r_]
    Ps = np.array([p for _, p in rungs], dtype=np.int64)[r_]
    n = len(s_)
    cal = np.arange(0, n, max(1, n // 4096))[:4096]
    t0 = time.perf_counter()
    oracle.decompress(s_[cal], e_[cal], q_[cal], Ks[cal], Ps[cal])
    rate = len(cal) / (time.perf_counter() - t0)
    m = int(min(n, max(4096, 0.6 * target_s * rate)))
    idx = np.linspace(0, n - 1, m).astype(np.int64)
    t0 = time.perf_counter()
    oracle.decompress(s_[idx], e_[idx], q_[idx], Ks[idx], Ps[idx])
    dt = time.perf_counter() - t0
    nb_s = 2000
    words = ostream.pack(s_[:nb_s], e_[:nb_s], q_[:nb_s], r_[:nb_s], rungs)
    t0 = time.perf_counter()
    ostream.unpack(words, r_[:nb_s], rungs)
    dt_s = time.perf_counter() - t0
    return {"value": 8 * m / dt, "unit": "decoded weights/s", "cores": 1, "kind": "oracle",
            "stream_parse_blocks_per_s": nb_s / dt_s,
            "sample": f"exact reconstruction of {m} evenly spaced blocks of the searched codes "
                      f"in {dt:.1f} s (C, one thread); the bit-by-bit stream parser on the first "
                      f"{nb_s} blocks in {dt_s:.2f} s"}


def grid_bench(args) -> int:
    """The rung grid (every rung S in 8..16, k in 2..6) on one matrix, one
    uniform search per rung, and the oracle's exhaustive search timed on the host
    over a sample of the same blocks at every rung."""
    import torch

    import synthetic
    from paper_2609_38477_amd import grid

    wl = synthetic.WORKLOADS[args.workload]
    W = synthetic.workload_weights(wl)
    dW = torch.from_numpy(W).cuda()
    grid.build_grid(dW, rungs=((8, 2),))    # warm-up
    res = grid.build_grid(dW, rungs=grid.PAPER_GRID)
    total_c = sum(res.candidates(r) for r in res.rungs)
    total_ms = sum(res.search_ms.values())
    out = {"metric": "rung grid: block·seed candidates/s over 45 uniform searches; 1 GPU",
           "value": total_c / (total_ms / 1e3), "unit": "block·seed candidates/s",
           "workload": wl.name, "shape": [wl.nrows, wl.ncols], "nblocks": res.nblocks,
           "rungs": len(res.rungs), "search_ms_total": total_ms, "candidates_total": total_c,
           "per_rung_ms": {f"{r[0]},{r[1]}": res.search_ms[r] for r in res.rungs},
           "data": "synthetic"}
    if not args.no_cpu_baseline:
        import oracle
        threads = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
        blocks = W.reshape(-1, 8)
        nbs = 256
        sample = np.ascontiguousarray(blocks[np.linspace(0, len(blocks) - 1, nbs).astype(np.int64)])
        dt, cands = 0.0, 0
        for K, P in res.rungs:
            pinv = oracle.cached_pinv_stack(K, P)
            t0 = time.perf_counter()
            oracle.search(sample, K, P, threads=threads, pinv=pinv)
            dt += time.perf_counter() - t0
            cands += nbs * ((1 << K) - 1)
            oracle.clear_pinv_cache()
        out["cpu_baseline"] = {"value": cands / dt, "unit": "block·seed candidates/s",
                               "cores": int(threads), "kind": "oracle",
                               "sample": f"{nbs} evenly spaced blocks of the same matrix at each of "
                                         f"the {len(res.rungs)} rungs, {cands:.3g} candidates in "
                                         f"{dt:.1f} s; pseudo-inverses precomputed outside the "
                                         f"timed region"}
    print(json.dumps(out), flush=True)
    return 0


def frontend_bench(args) -> int:
    """The data-free importance of one 7B-shaped synthetic layer (a of all
    seven projections, rho, channel orders, column statistics and outlier
    columns) on the GPU, and the oracle's fp64 numpy version of the same on the
    host."""
    import torch

    import synthetic
    from paper_2609_38477_amd import frontend

    L = synthetic.synthetic_layer(4096, 11008, 32, 8, 32000)
    dW = {n: torch.from_numpy(np.ascontiguousarray(L.tensors[n])).cuda()
          for n in (*frontend.PROJECTIONS, "lm_head")}
    frontend.layer_importance(L, dW)     # warm-up
    torch.cuda.synchronize()
    reps = 3
    t0 = time.perf_counter()
    for _ in range(reps):
        imp = frontend.layer_importance(L, dW)
    torch.cuda.synchronize()
    gpu_s = (time.perf_counter() - t0) / reps
    out = {"metric": "importance front end: seconds per 7B-shaped layer; 1 GPU",
           "value": gpu_s, "unit": "s", "higher_is_better": False,
           "layer": {"d": 4096, "f": 11008, "heads": 32, "kv_heads": 8, "vocab": 32000},
           "outliers": [list(o) for o in imp.outliers], "data": "synthetic"}
    if not args.no_cpu_baseline:
        from oracle import importance as oimp
        T = L.tensors
        t0 = time.perf_counter()
        a_attn = oimp.gamma_importance(L.gains["attn"])
        a_mlp = oimp.gamma_importance(L.gains["mlp"])
        ref = {"q": a_attn, "k": a_attn, "v": a_attn, "gate": a_mlp, "up": a_mlp,
               "o": oimp.propagate_o(T["v"], a_attn.astype(np.float32), L.n_heads, L.n_kv_heads),
               "down": oimp.propagate_down(T["gate"], T["up"], a_mlp.astype(np.float32))}
        oimp.rho_from_head(T["lm_head"])
        for n in frontend.PROJECTIONS:
            oimp.channel_order(ref[n].astype(np.float32))
        names = list(frontend.PROJECTIONS)
        want = oimp.outlier_columns([T[n] for n in names], [ref[n] for n in names])
        cpu_s = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": cpu_s, "unit": "s", "cores": 1, "kind": "oracle",
                               "same_outliers": [(names[t], c) for t, c in want] ==
                                                [tuple(o) for o in imp.outliers],
                               "sample": "the whole layer (the oracle's numpy fp64 path; BLAS "
                                         "threads as numpy configures them)"}
    print(json.dumps(out), flush=True)
    return 0


def row_tiles_bench(args) -> int:
    """A layer streamed through the GPU in row tiles from pinned host memory
    (two tiles resident at a time, the copy of the next tile overlapping the
    search of this one) against one call on the whole resident matrix: the same
    rungs, bases and search, codes compared bit for bit. Times are wall clock
    between synchronisations; the streamed time includes its host-to-device
    copies."""
    import torch

    import paper_2609_38477_amd as sq
    import synthetic

    wl = synthetic.WORKLOADS[args.workload]
    log(f"row tiles on {wl.name}: {wl.note}")
    W = synthetic.workload_weights(wl)
    a = synthetic.importance_profile(wl.ncols)
    rob, rep = sq.plan_schedule(wl.nrows, wl.ncols, wl.rungs, wl.damage, wl.target_bpw, a)
    d_rob = torch.from_numpy(rob).cuda() if len(wl.rungs) > 1 else None
    bases = [sq.build_bases(K, P) for K, P in wl.rungs]
    W_host = torch.from_numpy(W).pin_memory()
    cands = sum(int(rep["count"][r]) * ((1 << K) - 1) for r, (K, P) in enumerate(wl.rungs))

    def run(fn):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        out = fn()
        torch.cuda.synchronize()
        return time.perf_counter() - t0, out

    dW = torch.from_numpy(W).cuda()
    run(lambda: sq.compress(dW, bases, rung_of_block=d_rob))            # warm-up
    t_full, ref = run(lambda: sq.compress(dW, bases, rung_of_block=d_rob))
    ref = [t.cpu() for t in ref]
    del dW
    torch.cuda.empty_cache()
    out = {"metric": "row-tiled search against one resident call; 1 GPU", "workload": wl.name,
           "shape": [wl.nrows, wl.ncols], "candidates": cands, "resident_s": t_full,
           "resident_candidates_per_s": cands / t_full, "tiles": {}}
    for tiles in args.row_tiles_list:
        t, got = run(lambda: sq.compress_row_tiles(W_host, bases, rung_of_block=d_rob,
                                                   row_tiles=tiles))
        same = all(torch.equal(x.cpu(), y) for x, y in zip(got, ref))
        out["tiles"][str(tiles)] = {"s": t, "over_resident": t / t_full, "identical_codes": same,
                                    "resident_tile_bytes": 2 * 4 * wl.ncols * (-(-wl.nrows // tiles))}
        log(f"{tiles} tiles: {t:.3f} s ({t / t_full:.3f} of resident), identical {same}")
        del got
    out["data"] = "synthetic"
    print(json.dumps(out), flush=True)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="attn4096")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-gemm-reference", action="store_true")
    ap.add_argument("--no-target-layer", action="store_true",
                    help="leave out the 4096x14336 three-rung layer timed after the headline")
    ap.add_argument("--grid", action="store_true",
                    help="time the 45-rung grid (S in 8..16, k in 2..6) with the oracle beside it")
    ap.add_argument("--frontend", action="store_true",
                    help="time the importance front end on a 7B-shaped layer with the oracle beside it")
    ap.add_argument("--decoder", action="store_true",
                    help="time the decoder path (derive, pack, parse, decode, decode-GEMV) instead")
    ap.add_argument("--row-tiles", type=str, default=None,
                    help="comma-separated tile counts: time the search streamed in row tiles "
                         "from host memory against one resident call (e.g. 2,4,8)")
    ap.add_argument("--gemm-reference-only", action="store_true",
                    help="only time the fp16 GEMM used as the practical matrix-core reference")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); blocks are "
              "independent once the rungs are planned, so the search shards by row ranges with no "
              "exchange beyond gathering the codes", file=sys.stderr)
        return 2

    import torch

    if args.gemm_reference_only:
        print(json.dumps({"gemm_reference_tflops": practical_mfma_tflops()}), flush=True)
        return 0

    import paper_2609_38477_amd as sq
    import synthetic

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    if args.decoder:
        return decoder_bench(args)
    if args.grid:
        return grid_bench(args)
    if args.frontend:
        return frontend_bench(args)
    if args.row_tiles:
        args.row_tiles_list = [int(t) for t in args.row_tiles.split(",")]
        return row_tiles_bench(args)
    torch.cuda.set_device(torch.device("cuda:0"))
    wl = synthetic.WORKLOADS[args.workload]
    out, W = run_steps(wl, args.steps, args.warmup)
    out = {"metric": METRIC, **out}
    if args.workload == "attn4096" and not args.no_target_layer:
        # the 4096 x 14336 layer with the three-rung schedule, timed the same way
        tl = synthetic.WORKLOADS["mlp_up"]
        log(f"target layer {tl.name}: {TARGET_LAYER_STEPS} timed steps")
        t_out, _ = run_steps(tl, TARGET_LAYER_STEPS, 1)
        out["target_layer"] = {k: t_out[k] for k in (
            "value", "unit", "steps", "warmup", "ms_per_step", "config", "roofline",
            "roofline_other_counts", "phases_ms", "search_candidates_per_s")}
    if not args.no_gemm_reference:
        log("timing a 16384^3 fp16 GEMM on random data as the practical matrix-core reference")
        ref = practical_mfma_tflops()
        search_s = out["phases_ms"]["search"] / 1000.0
        cands = out["config"]["candidates_per_step"]
        issued = cands * ISSUED_FLOPS_PER_CANDIDATE / search_s / 1e12
        out["mfma_practical"] = {
            "reference": "torch.matmul fp16 16384x16384x16384, N(0,1) operands (hipBLASLt)",
            "reference_tflops": ref, "search_issued_tflops": issued,
            "search_issued_over_reference": issued / ref,
            "search_roofline_work_over_reference": out["roofline"]["achieved"] / ref}
    if not args.no_cpu_baseline:
        rungs = list(wl.rungs)
        K, P = rungs[0] if len(rungs) == 1 else rungs[1]
        log("timing the CPU oracle on a bounded sample")
        out["cpu_baseline"] = cpu_baseline(W, K, P, args.cpu_seconds)
    print(json.dumps(out), flush=True)
    return 0


TARGET_LAYER_STEPS = 3


def run_steps(wl, steps: int, warmup: int):
    """Whole-path steps on one workload: W untimed, then exactly `steps` timed
    between synchronisations. Returns the result fields and the host matrix."""
    import torch

    import paper_2609_38477_amd as sq
    import synthetic

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    log(f"workload {wl.name}: {wl.note}")
    W = synthetic.workload_weights(wl)
    a = synthetic.importance_profile(wl.ncols)
    dW = torch.from_numpy(W).to(dev)
    nb = wl.nblocks
    rungs = list(wl.rungs)
    R = len(rungs)
    bases = [sq.Bases(K, P, torch.empty(sq.seedq_bases_bytes(K, P), dtype=torch.uint8, device=dev))
             for K, P in rungs]
    seed = torch.empty(nb, dtype=torch.int32, device=dev)
    exp = torch.empty(nb, dtype=torch.uint8, device=dev)
    q = torch.empty((nb, 8), dtype=torch.int8, device=dev)
    err = torch.empty(nb, dtype=torch.float32, device=dev)
    W_hat = torch.empty_like(dW)
    nws = sq.seedq_compress_workspace_bytes(wl.nrows, wl.ncols, 8, R)
    ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=dev)
    d_rob = torch.empty(nb, dtype=torch.uint8, device=dev) if R > 1 else None
    rob_host = torch.zeros(nb, dtype=torch.uint8).pin_memory()
    rob_np = rob_host.numpy()

    def events():
        return {k: torch.cuda.Event(enable_timing=True) for k in ("start", "bases", "search", "decomp")}

    plan_s = []
    rep_counts = [0] * R

    def step(ev):
        t = time.perf_counter()
        rob, rep = sq.plan_schedule(wl.nrows, wl.ncols, rungs, wl.damage, wl.target_bpw, a,
                                    out=rob_np)
        plan_s.append(time.perf_counter() - t)
        cands = int(sum(int(rep["count"][r]) * ((1 << K) - 1) for r, (K, P) in enumerate(rungs)))
        rep_counts[:] = [int(rep["count"][r]) for r in range(R)]
        ev["start"].record(stream)
        if R > 1:
            d_rob.copy_(rob_host, non_blocking=True)
        for b in bases:
            sq.seedq_build_bases(b.K, b.P, 8, b.buffer, None, None, stream)
        ev["bases"].record(stream)
        sq.seedq_compress(dW, wl.nrows, wl.ncols, 8, d_rob, bases, seed, exp, q, err, ws, nws, stream)
        ev["search"].record(stream)
        sq.seedq_decompress(seed, exp, q, d_rob, rungs, wl.nrows, wl.ncols, 8, W_hat, None, stream)
        ev["decomp"].record(stream)
        return cands

    for i in range(warmup):
        step(events())
        torch.cuda.synchronize()
        log(f"{wl.name}: warmup step {i + 1}/{warmup} done")
    # timed region: exactly `steps` steps, events recorded on the stream the
    # kernels run on, read after the closing synchronisation
    evs = [events() for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        cands = step(evs[i])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    log(f"{wl.name}: {steps} timed steps done in {t1 - t0:.3f} s")
    phase = {"bases": [e["start"].elapsed_time(e["bases"]) for e in evs],
             "search": [e["bases"].elapsed_time(e["search"]) for e in evs],
             "decomp": [e["search"].elapsed_time(e["decomp"]) for e in evs]}
    ms = (t1 - t0) * 1000.0 / steps
    value = cands / (ms / 1000.0)

    search_ms = float(np.mean(phase["search"]))
    decomp_ms = float(np.mean(phase["decomp"]))
    bases_ms = float(np.mean(phase["bases"]))
    # dominant kernel: the search (one launch per rung, or per seed chunk of a
    # K >= 17 rung), timed by the events around seedq_compress on its stream
    flops = sum(rep_counts[r] * projection_flops(K, P) for r, (K, P) in enumerate(rungs))
    achieved = flops / (search_ms / 1000.0) / 1e12
    roofline = {"bound": "mfma", "achieved": achieved, "peak": PEAK_FP16_MFMA_TFLOPS,
                "unit": "TFLOP/s", "frac": achieved / PEAK_FP16_MFMA_TFLOPS,
                "traffic": measured_traffic(wl.name),
                "work": "2*C*P flops per block-seed candidate (the least-squares projection)"}
    other = {}
    for key, per in (("quadratic_form", QUADFORM_FLOPS_PER_CANDIDATE),
                     ("issued", ISSUED_FLOPS_PER_CANDIDATE)):
        t = cands * per / (search_ms / 1000.0) / 1e12
        other[key] = {"flops_per_candidate": per, "achieved": t,
                      "frac": t / PEAK_FP16_MFMA_TFLOPS}

    # The direct design -- project every block onto every seed's pseudo-inverse
    # on fp32 matrix cores (2 C P flops per candidate), then quantise each
    # candidate -- is capped at 157.3e12 / (2 C P) candidates/s even before its
    # epilogue; the quadratic-form screen above replaces that projection.
    direct_ceiling = cands / (flops / (PEAK_FP32_MFMA_TFLOPS * 1e12))
    out = {
        "value": value, "unit": "block·seed candidates/s", "n_gpus": 1,
        "steps": steps, "warmup": warmup, "ms_per_step": ms, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f16", "data": "synthetic",
        "config": {"workload": wl.name, "shape": [wl.nrows, wl.ncols], "C": 8,
                   "rungs": [list(r) for r in rungs], "target_bpw": wl.target_bpw,
                   "nblocks": nb, "blocks_per_rung": list(rep_counts),
                   "candidates_per_step": cands, "description": wl.note},
        "roofline": roofline,
        "roofline_other_counts": other,
        "phases_ms": {"plan_host": 1000.0 * float(np.mean(plan_s[-steps:])), "bases": bases_ms,
                      "search": search_ms, "decompress": decomp_ms},
        "search_candidates_per_s": cands / (search_ms / 1000.0),
        "fp32_projection_ceiling": {
            "candidates_per_s": direct_ceiling, "flops_per_candidate": flops / cands,
            "peak_tflops": PEAK_FP32_MFMA_TFLOPS,
            "search_over_ceiling": cands / (search_ms / 1000.0) / direct_ceiling},
        "decompress_GBps": nb * (14 + 32) / (decomp_ms / 1000.0) / 1e9,
    }
    del dW, bases, seed, exp, q, err, W_hat, ws, d_rob
    torch.cuda.empty_cache()
    return out, W


if __name__ == "__main__":
    sys.exit(main())
