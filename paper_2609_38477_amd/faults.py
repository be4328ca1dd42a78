"""Single-bit fault study of the decoder path (the security analysis: one bit of
the stored code or table changes between the encoder and the decoder; its
footprint by eq. (security_metrics)).

The encoder plans the rungs, searches every block and emits the headerless
stream plus a global table (lambda, floor value, tie count, rungs, damages).
The decoder re-derives every block's rung from the table (Algorithm 2), parses
the stream and reconstructs. A fault in a block's own bits changes that block
only, because no length depends on a decoded value (appendix on encoding and
decoding). A fault in the table changes the rungs the decoder derives, so the
parse goes out of step from the first affected block to the end of the tensor
(the propagation the paper simulates); a checksum over the table, whose size is
negligible, detects it. ``table_bytes`` serialises the table and
``table_crc32`` is the standard CRC-32 (zlib) of those bytes.

    python -m paper_2609_38477_amd.faults [--workload reduced] [--rows 512]

prints one JSON line with N_flip, p_flip and eta per fault.
"""
from __future__ import annotations

import argparse
import json
import struct
import sys
import zlib

import numpy as np

from . import (SEEDQ_BLOCK, build_bases, compress, decompress_stream, derive_schedule, footprint,
               pack, plan_schedule)


def table_bytes(rungs, damage, lam: float, floor_q: float, tie_count: int, offsets=()) -> bytes:
    """Little-endian serialisation of the global table: rung count, (K, P) and
    damage per rung, lambda, floor value, tie count, per-tensor word offsets."""
    out = struct.pack("<i", len(rungs))
    dmg = [0.0] * len(rungs) if damage is None else list(damage)
    for (K, P), e in zip(rungs, dmg):
        out += struct.pack("<iid", int(K), int(P), float(e))
    out += struct.pack("<ddq", float(lam), float(floor_q), int(tie_count))
    out += struct.pack("<i", len(offsets)) + b"".join(struct.pack("<q", int(o)) for o in offsets)
    return out


def table_crc32(*args, **kw) -> int:
    return zlib.crc32(table_bytes(*args, **kw)) & 0xFFFFFFFF


def flip_double(x: float, bit: int) -> float:
    """x with bit ``bit`` (0 = least significant) of its IEEE-754 pattern flipped."""
    u = struct.unpack("<Q", struct.pack("<d", x))[0] ^ (1 << bit)
    return struct.unpack("<d", struct.pack("<Q", u))[0]


class Encoded:
    """One tensor through the encoder: codes, stream, table."""

    def __init__(self, W, rungs, damage, target_bpw, col_importance, floor_fraction=0.06):
        import torch
        self.nrows, self.ncols = W.shape
        self.rungs = [tuple(int(v) for v in r) for r in rungs]
        self.damage = damage
        self.a = np.asarray(col_importance, dtype=np.float32)
        self.rob, self.rep = plan_schedule(self.nrows, self.ncols, self.rungs, damage, target_bpw,
                                           self.a, None, floor_fraction)
        d_rob = torch.from_numpy(self.rob).to(W.device)
        bases = [build_bases(K, P) for K, P in self.rungs]
        self.seed, self.exp, self.q, self.err = compress(W, bases, d_rob)
        self.words = pack(self.seed, self.exp, self.q, self.rungs, self.nrows, self.ncols, d_rob,
                          self.rep["count"])
        self.crc = table_crc32(self.rungs, damage, self.rep["lam"], self.rep["floor_q"],
                               self.rep["tie_count"])
        bits = np.array([K + 4 + 4 * P for K, P in self.rungs], dtype=np.int64)[self.rob]
        self.block_offset = np.concatenate([[0], np.cumsum(bits)])   # stream bit of every block

    def decode(self, words=None, lam=None, floor_q=None, tie_count=None):
        """The decoder: rungs re-derived from the (possibly corrupted) table, then
        a one-pass parse and reconstruction of the (possibly corrupted) stream."""
        import torch
        lam = self.rep["lam"] if lam is None else lam
        floor_q = self.rep["floor_q"] if floor_q is None else floor_q
        tie_count = self.rep["tie_count"] if tie_count is None else tie_count
        rob = derive_schedule(self.nrows, self.ncols, self.rungs, self.damage, self.a, lam, floor_q,
                              tie_count)
        d_rob = torch.from_numpy(rob).to(self.words.device)
        return decompress_stream(self.words if words is None else words, self.rungs, self.nrows,
                                 self.ncols, d_rob)

    def flip_stream_bit(self, n: int):
        w = self.words.clone()
        v = 1 << (n % 32)
        w[n // 32] ^= v - (1 << 32) if v >= 1 << 31 else v   # the words are int32
        return w


def study(enc: Encoded, block: int | None = None) -> list:
    """Footprint of one fault of every kind against the clean decode."""
    clean = enc.decode()
    nb = enc.nrows * enc.ncols // SEEDQ_BLOCK
    b = nb // 3 if block is None else block
    K, P = enc.rungs[int(enc.rob[b])]
    o = int(enc.block_offset[b])
    rows = []

    def record(kind, corrupt, detected):
        n, p, eta = footprint(clean, corrupt)
        rows.append({"fault": kind, "N_flip": n, "p_flip": p, "eta": eta,
                     "table_checksum_detects": detected})

    record(f"seed bit 0 of block {b} (rung {K},{P})", enc.decode(enc.flip_stream_bit(o)), False)
    record(f"seed bit {K - 1} of block {b}", enc.decode(enc.flip_stream_bit(o + K - 1)), False)
    record(f"exponent bit 0 of block {b}", enc.decode(enc.flip_stream_bit(o + K)), False)
    record(f"mantissa q_0 sign bit of block {b}", enc.decode(enc.flip_stream_bit(o + K + 7)), False)
    lam, qf, T = enc.rep["lam"], enc.rep["floor_q"], enc.rep["tie_count"]
    for bit in (0, 40, 52):
        lam2 = flip_double(lam, bit)
        det = table_crc32(enc.rungs, enc.damage, lam2, qf, T) != enc.crc
        try:
            rec = enc.decode(lam=lam2)
        except Exception as exc:  # the decoder refuses the table (e.g. tie count too large)
            rows.append({"fault": f"lambda bit {bit}", "decoder_error": str(exc),
                         "table_checksum_detects": det})
            continue
        record(f"lambda bit {bit}", rec, det)
    qf2 = flip_double(qf, 52)
    record("floor value bit 52", enc.decode(floor_q=qf2),
           table_crc32(enc.rungs, enc.damage, lam, qf2, T) != enc.crc)
    if T > 0:
        record("tie count - 1", enc.decode(tie_count=T - 1),
               table_crc32(enc.rungs, enc.damage, lam, qf, T - 1) != enc.crc)
    return rows


def main(argv=None) -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="reduced")
    ap.add_argument("--rows", type=int, default=0, help="first rows only (0 = all)")
    ap.add_argument("--target-bpw", type=float, default=0.0)
    args = ap.parse_args(argv)
    import os
    import torch
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    if root not in sys.path:
        sys.path.insert(0, root)
    import synthetic
    wl = synthetic.WORKLOADS[args.workload]
    nrows = args.rows or wl.nrows
    W = synthetic.weights(nrows, wl.ncols, wl.sigma, wl.key, wl.outlier_frac)
    target = args.target_bpw or wl.target_bpw
    enc = Encoded(torch.from_numpy(W).cuda(), wl.rungs, wl.damage, target,
                  synthetic.importance_profile(wl.ncols))
    rows = study(enc)
    print(json.dumps({"workload": wl.name, "shape": [nrows, wl.ncols], "rungs": enc.rungs,
                      "target_bpw": target, "tie_count": enc.rep["tie_count"],
                      "payload_bytes": int(enc.words.numel() * 4), "faults": rows}), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
