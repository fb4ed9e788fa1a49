"""The butterfly-patterned table of partial sums (Section 4) -- TEST
INFRASTRUCTURE ONLY.

Notation: W lanes (threads) each own one token; a block holds W consecutive
topics; Z(t, v, w) is the sum of thread t's products over block topics v..w.
A table is indexed [row][column]: row = topic within the block, column = lane.

Three independent formulations, which the tests check against each other and
against the worked examples the paper prints (Figs. 1 and 2, the replacement
schedule and the search tree of thread 5):

  closed_form(i, j)        the entry at row i, column j after all replacement
                           sets (the formula stated after Algorithm 10);
  replacement_schedule(W)  the sets of 2x2 replacements R[i,j;k,l]; applying
  apply_replacements(...)  them to the transposed products builds the table;
  table_fp64(a, W)         the whole per-lane table p[K] of W tokens (leading
                           remnant untransposed, then butterfly blocks whose last
                           row is the full prefix), from the closed form;
  search_sim(...)          the search of Algorithms 9 and 10 over that table,
                           with all W lanes as one numpy vector (shuffle and
                           shuffleXor are gathers across the vector).

The alternative replacement the paper mentions in Section 4, [a b; c d] ->
[a c; a+b c+d], has its own closed form (closed_form_alt), table
(table_alt_fp64) and search (search_alt_sim): every entry of its table is the
sum over the left half of an aligned range of topics, so the search is a
descent from the whole block down a binary tree.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


def log2_exact(W: int) -> int:
    if W < 1 or W & (W - 1):
        raise ValueError("W must be a power of two")
    return W.bit_length() - 1


def closed_form(i: int, j: int) -> tuple[int, int, int]:
    """(thread, first, last) of the entry at block row i, column j: with
    m = i xor (i+1) and k = floor(m/2), the thread is (i & ~m) + (j & m) and the
    range is (j & ~k) .. (j & ~k) + k."""
    m = i ^ (i + 1)
    k = m >> 1
    thread = (i & ~m) + (j & m)
    v = j & ~k
    return thread, v, v + k


@dataclass(frozen=True)
class Z:
    """Symbolic sum of one thread's products over block topics lo..hi."""

    thread: int
    lo: int
    hi: int

    def __add__(self, other: "Z") -> "Z":
        if self.thread != other.thread:
            raise ValueError(f"adding sums of different threads: {self} + {other}")
        if other.lo == self.hi + 1:
            return Z(self.thread, self.lo, other.hi)
        if self.lo == other.hi + 1:
            return Z(self.thread, other.lo, self.hi)
        raise ValueError(f"non-adjacent ranges: {self} + {other}")

    def __str__(self) -> str:
        return f"{self.thread}:{self.lo}:{self.hi}"


def replacement_schedule(W: int) -> list[list[tuple[int, int, int, int]]]:
    """log2(W) sets of replacements R[i, j; k, l].  Set b (bit = 2**b) pairs
    rows d and d + bit for d = 2*bit*t + bit - 1, t < W/(2*bit), with column
    pairs (c, c + bit) for every c whose bit b is clear."""
    sets = []
    for b in range(log2_exact(W)):
        bit = 1 << b
        rows = [(2 * bit * t + bit - 1, 2 * bit * t + 2 * bit - 1)
                for t in range(W // (2 * bit))]
        cols = [(c, c + bit) for c in range(W) if not c & bit]
        sets.append([(i, j, k, l) for (i, j) in rows for (k, l) in cols])
    return sets


def apply_replacement(tab, i, j, k, l) -> None:
    """[a b; c d] at rows (i, j), columns (k, l) becomes [a d; a+b c+d]."""
    a, b, c, d = tab[i][k], tab[i][l], tab[j][k], tab[j][l]
    tab[i][k], tab[i][l] = a, d
    tab[j][k], tab[j][l] = a + b, c + d


def apply_replacement_alt(tab, i, j, k, l) -> None:
    """The alternative rule: [a b; c d] at rows (i, j), columns (k, l)
    becomes [a c; a+b c+d]."""
    a, b, c, d = tab[i][k], tab[i][l], tab[j][k], tab[j][l]
    tab[i][k], tab[i][l] = a, c
    tab[j][k], tab[j][l] = a + b, c + d


def apply_replacements(tab, schedule, upto: int | None = None, alt: bool = False):
    """Apply the first ``upto`` sets (all if None) in order, with the paper's
    rule or (``alt``) the alternative one; returns ``tab``."""
    rule = apply_replacement_alt if alt else apply_replacement
    for s in schedule[:upto]:
        for (i, j, k, l) in s:
            rule(tab, i, j, k, l)
    return tab


def closed_form_alt(i: int, j: int) -> tuple[int, int, int]:
    """(thread, first, last) of the entry at block row i, column j of the
    alternative table: with m = i xor (i+1) and k = floor(m/2), the thread is
    (i & ~m) + (j & m), as in the paper's table, and the range is
    (j & ~m) .. (j & ~m) + k: the left half of the aligned range of m + 1
    topics that holds topic j."""
    m = i ^ (i + 1)
    k = m >> 1
    thread = (i & ~m) + (j & m)
    v = j & ~m
    return thread, v, v + k


def transposed_products(W: int) -> list[list[Z]]:
    """Symbolic block before any replacement: row t, column c holds thread t's
    product at topic c."""
    return [[Z(t, c, c) for c in range(W)] for t in range(W)]


def table_fp64(a: np.ndarray, W: int) -> np.ndarray:
    """Per-lane table p of W tokens, shape [W lanes][K], in fp64.

    ``a[t][k]`` is thread t's product at topic k (exact fp64 products).  The
    first K mod W topics (the remnant) hold the full prefix of the lane's own
    token; each following block of W rows holds the closed-form entries in
    rows 0..W-2 and the lane's full prefix at the block's end in row W-1.
    """
    a = np.asarray(a, np.float64)
    Wt, K = a.shape
    assert Wt == W
    R = K % W
    S = np.cumsum(a, axis=1)
    p = np.empty((W, K), np.float64)
    p[:, :R] = S[:, :R]
    for base in range(R, K, W):
        for i in range(W - 1):
            for j in range(W):
                t, v, w = closed_form(i, j)
                p[j, base + i] = a[t, base + v: base + w + 1].sum()
        p[:, base + W - 1] = S[:, base + W - 1]
    return p


def table_alt_fp64(a: np.ndarray, W: int) -> np.ndarray:
    """As table_fp64, with the alternative table in rows 0..W-2 of each
    block."""
    a = np.asarray(a, np.float64)
    Wt, K = a.shape
    assert Wt == W
    R = K % W
    S = np.cumsum(a, axis=1)
    p = np.empty((W, K), np.float64)
    p[:, :R] = S[:, :R]
    for base in range(R, K, W):
        for i in range(W - 1):
            for j in range(W):
                t, v, w = closed_form_alt(i, j)
                p[j, base + i] = a[t, base + v: base + w + 1].sum()
        p[:, base + W - 1] = S[:, base + W - 1]
    return p


def search_alt_sim(p: np.ndarray, u: np.ndarray, W: int) -> np.ndarray:
    """z of each lane over the alternative table ``p`` ([W][K]): the block
    search of Algorithm 9, then a descent inside the block.  Lane r, at the
    node of 2**(s+1) topics starting at b, reads the sum over the left half,
    which the table keeps at row (r & ~(2**(s+1)-1)) + 2**s - 1 of column
    (r & (2**(s+1)-1)) + b; it goes left if stop < low + that sum, else right
    with low increased by it.  A lane that finds no entry above its stop value
    gets K - 1."""
    p = np.asarray(p, np.float64)
    Wl, K = p.shape
    assert Wl == W
    lg = log2_exact(W)
    r = np.arange(W)
    R, NB = K % W, K // W
    stop = p[:, K - 1] * np.asarray(u, np.float64)
    j = np.full(W, K - 1, np.int64)
    if K >= W:
        ends = p[:, R + W - 1::W]                       # [W][NB] block ends
        blk = np.minimum((ends <= stop[:, None]).sum(axis=1), NB - 1)
        base = R + blk * W
        low = np.where(base > 0, p[r, np.maximum(base - 1, 0)], 0.0)
        b = np.zeros(W, np.int64)
        for s in range(lg - 1, -1, -1):
            span, node = 1 << s, 2 << s
            row = (r & ~(node - 1)) + span - 1
            col = (r & (node - 1)) + b
            # column col of the table holds, in lane r's block, r's own sum
            cmp = low + p[col, base + row]
            left = stop < cmp
            low = np.where(left, low, cmp)
            b = np.where(left, b, b + span)
        j = base + b
        in_rem = (base > 0) & (stop < p[r, np.maximum(base - 1, 0)])
    else:
        in_rem = np.ones(W, bool)
    for lane in np.nonzero(in_rem)[0]:
        for i in range(R):
            if stop[lane] < p[lane, i]:
                j[lane] = i
                break
    return j.astype(np.int32)


def search_sim(p: np.ndarray, u: np.ndarray, W: int) -> np.ndarray:
    """z of each lane by the search of Algorithms 9 and 10 over table ``p``
    ([W][K]); every step is a vector operation over the W lanes.

    Readings: the block-search result j is the output variable; a lane that
    finds no entry above its stop value gets K - 1.
    """
    p = np.asarray(p, np.float64)
    Wl, K = p.shape
    assert Wl == W
    lg = log2_exact(W)
    r = np.arange(W)
    R, NB = K % W, K // W
    total = p[:, K - 1]
    stop = total * np.asarray(u, np.float64)

    # Binary search over the last row of each block.
    lo = np.zeros(W, np.int64)
    hi = np.full(W, NB - 1, np.int64)
    search_base = R + W - 1
    while (lo < hi).any():
        act = lo < hi
        mid = (lo + hi) // 2
        val = p[r, np.clip(mid * W + search_base, 0, K - 1)]
        go_low = stop < val
        hi = np.where(act & go_low, mid, hi)
        lo = np.where(act & ~go_low, mid + 1, lo)
    block_base = R + lo * W
    j = np.full(W, K - 1, np.int64)

    if K >= W:
        low = np.where(block_base > 0, p[r, np.maximum(block_base - 1, 0)], 0.0)
        high = p[r, block_base + W - 1]
        flip = np.zeros(W, np.int64)
        for b in range(lg):
            bit = 1 << (lg - 1 - b)
            mask = ((W - 1) * (2 * bit)) & (W - 1)
            y = np.zeros(W)
            for i in range(W // (2 * bit)):
                d = (bit - 1) + 2 * bit * i
                him = (d & mask) + (r & ~mask)
                his_base = block_base[him]              # shuffle(blockBase, him)
                offered = p[r, his_base + d]            # each lane's p[...]
                t = offered[r ^ flip]                   # shuffleXor(..., flip)
                y = np.where(((r ^ d) & mask) == 0, t, y)
            cmp = np.where(r & bit, high - y, low + y)
            below = stop < cmp
            high = np.where(below, cmp, high)
            low = np.where(below, low, cmp)
            flip = np.where(below, flip ^ (bit & r), flip ^ (bit & ~r))
        j = block_base + (flip ^ r)

    # Remnant: only when the stop value lies before the searched block.
    in_rem = (block_base > 0) & (stop < p[r, np.maximum(block_base - 1, 0)])
    for lane in np.nonzero(in_rem)[0]:
        for i in range(R):
            if stop[lane] < p[lane, i]:
                j[lane] = i
                break
    return j.astype(np.int32)


def table_symbolic(W: int, K: int) -> list[list[tuple[int, int, int]]]:
    """The per-lane table of Fig. 1 (right) as (thread, first, last) with
    global topic indices, indexed [row k][column j]: remnant rows and each
    block's last row hold the full prefix (j, 0, k); the other block rows hold
    the closed-form entries shifted by the block's first topic."""
    R = K % W
    tab = [[(j, 0, k) for j in range(W)] for k in range(K)]
    for base in range(R, K, W):
        for i in range(W - 1):
            for j in range(W):
                t, v, w = closed_form(i, j)
                tab[base + i][j] = (t, base + v, base + w)
    return tab


def search_nodes(tab, W: int, K: int, lane: int, block: int):
    """Table entries lane ``lane`` can read at each level of the in-block
    search of Algorithm 10 when every lane searches block ``block``, over all
    comparison outcomes.  Returns (lowValue, highValue, [set per level]).
    Entries come from the search-assist selection: at level b the lane keeps
    the entry offered by lane (lane xor flip) for the row d whose bits above
    ``bit`` match the lane's."""
    lg = log2_exact(W)
    R = K % W
    base = R + block * W
    low = tab[base - 1][lane] if base > 0 else None
    high = tab[base + W - 1][lane]
    levels = []
    flips = {0}
    for b in range(lg):
        bit = 1 << (lg - 1 - b)
        mask = ((W - 1) * (2 * bit)) & (W - 1)
        nodes, nxt = set(), set()
        for flip in flips:
            for i in range(W // (2 * bit)):
                d = (bit - 1) + 2 * bit * i
                if ((lane ^ d) & mask) == 0:
                    nodes.add(tab[base + d][lane ^ flip])
            nxt.add(flip ^ (bit & lane))
            nxt.add(flip ^ (bit & ~lane))
        levels.append(nodes)
        flips = nxt
    return low, high, levels
