"""Philox counter-based generators -- TEST INFRASTRUCTURE ONLY.

Written from the published definition (J. K. Salmon, M. A. Moraes, R. O. Dror,
D. E. Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC 2011, Section
4.2).  The paper on butterfly partial sums draws the uniform of each token
inside its draw procedure without naming a generator; the fused-RNG draw uses
Philox4x32-10, and this module is the reference it is checked against.

Philox-4xW-R on a counter (x0, x1, x2, x3) and key (k0, k1) of W-bit words:
R rounds, each
    (hi0, lo0) = M0 * x0   (the high and low W bits of the 2W-bit product)
    (hi1, lo1) = M1 * x2
    (x0, x1, x2, x3) <- (hi1 ^ x1 ^ k0, lo1, hi0 ^ x3 ^ k1, lo0)
with the key advanced by the Weyl increments (k0 += C0, k1 += C1, mod 2^W)
between rounds (not before the first).  Plain Python integers: slow, exact.

Uniform of token n in sweep s under a 64-bit seed (the convention of the
fused draw): Philox4x32-10 with key (seed mod 2^32, seed >> 32) and counter
(n mod 2^32, n >> 32, s, 0); u = (x0 >> 8) * 2^-24, the top 24 bits of the
first output word, exact in fp32 and in [0, 1).
"""
from __future__ import annotations

import numpy as np

# Multipliers and Weyl increments of the published definition.
PARAMS = {
    32: dict(M=(0xD2511F53, 0xCD9E8D57), C=(0x9E3779B9, 0xBB67AE85)),
    64: dict(M=(0xD2E7470EE14C6C93, 0xCA5A826395121157),
             C=(0x9E3779B97F4A7C15, 0xBB67AE8584CAA73B)),
}


def philox4(counter, key, width: int = 32, rounds: int = 10) -> tuple[int, int, int, int]:
    """Philox-4x``width``-``rounds`` of one counter (4 words) and key (2 words)."""
    mask = (1 << width) - 1
    M0, M1 = PARAMS[width]["M"]
    C0, C1 = PARAMS[width]["C"]
    x0, x1, x2, x3 = (int(v) & mask for v in counter)
    k0, k1 = (int(v) & mask for v in key)
    for r in range(rounds):
        if r:
            k0, k1 = (k0 + C0) & mask, (k1 + C1) & mask
        p0, p1 = M0 * x0, M1 * x2
        hi0, lo0 = p0 >> width, p0 & mask
        hi1, lo1 = p1 >> width, p1 & mask
        x0, x1, x2, x3 = hi1 ^ x1 ^ k0, lo1, hi0 ^ x3 ^ k1, lo0
    return x0, x1, x2, x3


def philox4x32_np(c0, c1, c2, c3, k0, k1, rounds: int = 10):
    """Philox4x32 over arrays of counters (uint32 arrays, broadcast), in numpy
    uint64 arithmetic: the 64-bit product of two 32-bit words is exact."""
    M0, M1 = (np.uint64(m) for m in PARAMS[32]["M"])
    C0, C1 = (np.uint64(c) for c in PARAMS[32]["C"])
    m32 = np.uint64(0xFFFFFFFF)
    s32 = np.uint64(32)
    x0, x1, x2, x3 = (np.asarray(v, np.uint64) & m32 for v in (c0, c1, c2, c3))
    k0 = np.uint64(int(k0) & 0xFFFFFFFF)
    k1 = np.uint64(int(k1) & 0xFFFFFFFF)
    for r in range(rounds):
        if r:
            k0, k1 = (k0 + C0) & m32, (k1 + C1) & m32
        p0, p1 = M0 * x0, M1 * x2
        x0, x1, x2, x3 = ((p1 >> s32) ^ x1 ^ k0, p1 & m32,
                          (p0 >> s32) ^ x3 ^ k1, p0 & m32)
    return tuple(v.astype(np.uint32) for v in (x0, x1, x2, x3))


def token_uniforms(seed: int, sweep: int, first: int, count: int) -> np.ndarray:
    """u of tokens first .. first + count - 1 (float32), by the convention in
    the module docstring."""
    n = np.arange(first, first + count, dtype=np.uint64)
    seed = int(seed) & ((1 << 64) - 1)
    x0, _, _, _ = philox4x32_np(n & np.uint64(0xFFFFFFFF), n >> np.uint64(32),
                                np.uint64(int(sweep) & 0xFFFFFFFF), np.uint64(0),
                                seed & 0xFFFFFFFF, seed >> 32)
    return ((x0 >> np.uint32(8)).astype(np.float64) * 2.0 ** -24).astype(np.float32)
