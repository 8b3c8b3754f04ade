"""Philox4x64-10, written from its published definition.

Reference: J. K. Salmon, M. A. Moraes, R. O. Dror, D. E. Shaw, "Parallel Random
Numbers: As Easy as 1, 2, 3", SC'11, section 5 (the Philox S-box: two 64x64->128
multiplications per round, key bumped by two Weyl constants between rounds).

Part of the CPU oracle (test infrastructure).

The sampler's random stream: draw s (s = 0, 1, ...) for node v at hop h under
key K is word (s mod 4) of Philox4x64-10 applied to the counter
(1 + floor(s/4), v, h, 0) with key (K, 0).  The paper does not name a generator
(it only says neighbours are selected at random, section 2.2); this layout was
chosen so that the stream equals numpy's Philox bit generator started at
counter (0, v, h, 0), which increments counter word 0 before each block.
"""
from __future__ import annotations

import numpy as np

MASK64 = (1 << 64) - 1
# Round multipliers and key-schedule (Weyl) increments of Philox4x64.
PHILOX_M0 = 0xD2E7470EE14C6C93
PHILOX_M1 = 0xCA5A826395121157
PHILOX_W0 = 0x9E3779B97F4A7C15  # golden ratio
PHILOX_W1 = 0xBB67AE8584CAA73B  # sqrt(3) - 1
ROUNDS = 10


def philox4x64(ctr, key, rounds: int = ROUNDS):
    """Scalar Philox4x64 on Python ints: ctr = (x0, x1, x2, x3), key = (k0, k1)."""
    x0, x1, x2, x3 = (int(c) & MASK64 for c in ctr)
    k0, k1 = (int(k) & MASK64 for k in key)
    for r in range(rounds):
        if r:
            k0 = (k0 + PHILOX_W0) & MASK64
            k1 = (k1 + PHILOX_W1) & MASK64
        p0 = PHILOX_M0 * x0
        p1 = PHILOX_M1 * x2
        hi0, lo0 = p0 >> 64, p0 & MASK64
        hi1, lo1 = p1 >> 64, p1 & MASK64
        x0, x1, x2, x3 = hi1 ^ x1 ^ k0, lo1, hi0 ^ x3 ^ k1, lo0
    return (x0, x1, x2, x3)


def draw_scalar(rng_key: int, hop: int, node: int, s: int) -> int:
    """Draw s of node `node` at hop `hop` (scalar reference of the stream layout)."""
    block = philox4x64((1 + s // 4, node, hop, 0), (rng_key, 0))
    return block[s % 4]


# ---- vectorised form (numpy uint64 arrays; exact, via 32-bit halves) --------

_M32 = np.uint64(0xFFFFFFFF)
_S32 = np.uint64(32)


def _mulhilo64(a: np.ndarray, b: int):
    """(hi, lo) of the 128-bit product a*b, for a uint64 array and a 64-bit constant."""
    a = a.astype(np.uint64)
    bh, bl = np.uint64(b >> 32), np.uint64(b & 0xFFFFFFFF)
    ah, al = a >> _S32, a & _M32
    ll = al * bl
    lh = al * bh
    hl = ah * bl
    hh = ah * bh
    mid = (ll >> _S32) + (lh & _M32) + (hl & _M32)
    hi = hh + (lh >> _S32) + (hl >> _S32) + (mid >> _S32)
    lo = a * np.uint64(b)
    return hi, lo


def philox4x64_vec(x0, x1, x2, x3, k0: int, k1: int, rounds: int = ROUNDS):
    """Philox4x64 on uint64 arrays (the counters); key words are scalars."""
    with np.errstate(over="ignore"):
        x0, x1, x2, x3 = (np.asarray(x, dtype=np.uint64) for x in (x0, x1, x2, x3))
        kk0, kk1 = k0 & MASK64, k1 & MASK64
        for r in range(rounds):
            if r:
                kk0 = (kk0 + PHILOX_W0) & MASK64
                kk1 = (kk1 + PHILOX_W1) & MASK64
            hi0, lo0 = _mulhilo64(x0, PHILOX_M0)
            hi1, lo1 = _mulhilo64(x2, PHILOX_M1)
            x0, x1, x2, x3 = (hi1 ^ x1 ^ np.uint64(kk0), lo1,
                              hi0 ^ x3 ^ np.uint64(kk1), lo0)
    return x0, x1, x2, x3


def draws(rng_key: int, hop: int, nodes: np.ndarray, count: int) -> np.ndarray:
    """Draws 0..count-1 for every node in `nodes` at hop `hop`: uint64 [len(nodes) x count]."""
    nodes = np.asarray(nodes, dtype=np.uint64)
    n = nodes.shape[0]
    nblk = (count + 3) // 4
    out = np.empty((n, nblk * 4), dtype=np.uint64)
    zeros = np.zeros(n, dtype=np.uint64)
    hops = np.full(n, hop, dtype=np.uint64)
    for b in range(nblk):
        ctr0 = np.full(n, 1 + b, dtype=np.uint64)
        y = philox4x64_vec(ctr0, nodes, hops, zeros, rng_key, 0)
        for w in range(4):
            out[:, 4 * b + w] = y[w]
    return out[:, :count]
