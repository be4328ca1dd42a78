"""Oracle for the headerless variable-length code stream and the fault
footprint metrics (test infrastructure only).

Stream (Algorithm 1, the emit step: every block contributes exactly l(g_b) =
K + 4P + 4 bits of eq. (rate), with no header; appendix on encoding and
decoding: a decoder reads a tensor's blocks in order from its start). The paper fixes no
bit layout; the reading used here and by the library is:

* blocks in row-major block order b = r * (ncols / 8) + g;
* inside a block: the seed (K bits), then the exponent e (4 bits), then the
  mantissas q_0 .. q_{P-1} (4 bits each, two's complement);
* every field least-significant bit first, at increasing stream bit positions;
* stream bit n is bit (n mod 32) of 32-bit little-endian word n // 32;
* the tensor's payload is padded with zero bits to a whole word.

This module writes that definition out bit by bit (a Python list of 0/1 per
stream bit), so it is slow and meant for small tensors.

Footprint (eq. (security_metrics)): for a clean and a corrupted reconstruction,
N_flip counts the weights that differ, p_flip = N_flip / (R C), and eta is the
Frobenius norm of the difference over that of the clean reconstruction.
"""
from __future__ import annotations

import numpy as np


def block_bits(K: int, P: int) -> int:
    """l(g) of eq. (rate) with m = e = 4."""
    return K + 4 + 4 * P


def _field(value: int, width: int) -> list:
    return [(value >> i) & 1 for i in range(width)]


def pack(seed, exp, q, rung_of_block, rungs) -> np.ndarray:
    """uint32 words of the payload of one tensor. ``q`` is [nblocks, >= P] of
    signed mantissas; ``rung_of_block`` indexes ``rungs``."""
    bits: list = []
    for b in range(len(rung_of_block)):
        K, P = rungs[int(rung_of_block[b])]
        bits += _field(int(seed[b]), K)
        bits += _field(int(exp[b]), 4)
        for j in range(P):
            bits += _field(int(q[b][j]) & 0xF, 4)
    bits += [0] * (-len(bits) % 32)
    words = np.zeros(len(bits) // 32, dtype=np.uint32)
    for n, bit in enumerate(bits):
        if bit:
            words[n // 32] |= np.uint32(1 << (n % 32))
    return words


def unpack(words, rung_of_block, rungs):
    """(seed, exp, q [nblocks, 8] int8) read block by block from the start of the payload."""
    words = np.asarray(words, dtype=np.uint32)
    nbits = 32 * len(words)

    def bit(n: int) -> int:
        return int(words[n // 32] >> np.uint32(n % 32)) & 1

    def read(pos: int, width: int) -> int:
        return sum(bit(pos + i) << i for i in range(width))

    nb = len(rung_of_block)
    seed = np.zeros(nb, dtype=np.uint32)
    exp = np.zeros(nb, dtype=np.uint8)
    q = np.zeros((nb, 8), dtype=np.int8)
    pos = 0
    for b in range(nb):
        K, P = rungs[int(rung_of_block[b])]
        if pos + block_bits(K, P) > nbits:
            raise ValueError("stream too short")
        seed[b] = read(pos, K)
        pos += K
        exp[b] = read(pos, 4)
        pos += 4
        for j in range(P):
            v = read(pos, 4)
            q[b, j] = v - 16 if v >= 8 else v
            pos += 4
    return seed, exp, q


def footprint(clean, corrupt):
    """(N_flip, p_flip, eta) of eq. (security_metrics)."""
    a = np.asarray(clean, dtype=np.float64)
    d = np.asarray(corrupt, dtype=np.float64) - a
    n = int(np.count_nonzero(d != 0))
    return n, n / a.size, float(np.sqrt((d * d).sum()) / np.sqrt((a * a).sum()))
