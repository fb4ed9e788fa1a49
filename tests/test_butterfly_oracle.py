"""Pins of the butterfly-table formulations in the oracle (Section 4) against
the worked examples the paper prints for W = 8, K = 19, and against each
other for W up to 64."""
import os

import numpy as np
import pytest

import oracle
from oracle import butterfly as bf
from conftest import GOLDEN


def _entries(line):
    return [tuple(int(x) for x in e.split(":")) for e in line.split()]


def _read(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return [ln.rstrip("\n") for ln in f if ln.strip() and not ln.startswith("#")]


def test_schedule_matches_paper_w8():
    gold = [[tuple(int(x) for x in e.split(",")) for e in ln.split()]
            for ln in _read("replacement_schedule_W8.txt")]
    assert bf.replacement_schedule(8) == gold


def test_replacement_snapshots_match_fig2():
    lines = _read("fig2_snapshots_W8.txt")
    panels, cur = [], None
    for ln in lines:
        if ln.startswith("panel"):
            cur = []
            panels.append(cur)
        else:
            cur.append(_entries(ln))
    assert len(panels) == 4
    sched = bf.replacement_schedule(8)
    for n, gold in enumerate(panels):
        tab = bf.apply_replacements(bf.transposed_products(8), sched, upto=n)
        got = [[(z.thread, z.lo, z.hi) for z in row] for row in tab]
        assert got == gold, f"panel {n}"


@pytest.mark.parametrize("W", [2, 4, 8, 16, 32, 64])
def test_closed_form_equals_replacement_process(W):
    tab = bf.apply_replacements(bf.transposed_products(W),
                                bf.replacement_schedule(W))
    for i in range(W):
        for j in range(W):
            z = tab[i][j]
            assert (z.thread, z.lo, z.hi) == bf.closed_form(i, j)
    # the last row holds every lane's own block total
    assert all(bf.closed_form(W - 1, j) == (j, 0, W - 1) for j in range(W))


def test_symbolic_table_matches_fig1_right():
    gold = [_entries(ln) for ln in _read("fig1_right_W8_K19.txt")]
    assert bf.table_symbolic(8, 19) == gold


def test_full_prefix_table_matches_fig1_left():
    gold = [_entries(ln) for ln in _read("fig1_left_W8_K19.txt")]
    assert gold == [[(j, 0, k) for j in range(8)] for k in range(19)]
    # the remnant rows and each block's last row agree between the two tables
    right = [_entries(ln) for ln in _read("fig1_right_W8_K19.txt")]
    for k in (0, 1, 2, 10, 18):
        assert right[k] == gold[k]


def test_thread5_search_tree():
    lines = _read("thread5_tree_W8_K19.txt")
    start = _entries(lines[0].split(None, 1)[1])
    levels = [set(_entries(ln.split(None, 2)[2])) for ln in lines[1:]]
    tab = bf.table_symbolic(8, 19)
    low, high, got = bf.search_nodes(tab, 8, 19, lane=5, block=0)
    assert [low, high] == start
    assert got == levels


@pytest.mark.parametrize("W", [8, 16, 64])
@pytest.mark.parametrize("K_extra", [0, 3, 5])
def test_numeric_table_equals_replacement(W, K_extra):
    """table_fp64 (closed form, global offsets) equals the replacement process
    run on the numbers of each block, with the running prefix in the last row."""
    rng = np.random.default_rng(W + K_extra)
    K = 3 * W + K_extra
    a = rng.random((W, K))
    p = bf.table_fp64(a, W)
    R = K % W
    S = np.cumsum(a, axis=1)
    assert np.allclose(p[:, :R], S[:, :R], rtol=0, atol=0)
    for base in range(R, K, W):
        blk = [[a[t, base + c] for c in range(W)] for t in range(W)]
        tab = bf.apply_replacements(blk, bf.replacement_schedule(W))
        for i in range(W - 1):
            for j in range(W):
                assert abs(tab[i][j] - p[j, base + i]) <= 1e-12 * (1 + abs(p[j, base + i]))
        assert np.allclose(p[:, base + W - 1], S[:, base + W - 1], rtol=1e-15)


@pytest.mark.parametrize("W", [2, 4, 8, 16, 32, 64])
def test_search_over_butterfly_table_equals_definition(W):
    """Algorithms 9 and 10 run over the butterfly table give the plain
    definition's z, outside the (fp64) rounding band, for K with and without
    a remnant, below W, and with ordered and shuffled documents."""
    rng = np.random.default_rng(100 + W)
    for K in sorted({1, 3, max(1, W - 1), W, W + 1, 19, 2 * W, 2 * W + 3, 5 * W + 7}):
        for rep in range(3):
            th = rng.random((W, K)).astype(np.float32)
            ph = rng.random((W, K)).astype(np.float32)
            th[rng.random((W, K)) < 0.3] = 0
            if rep == 2:
                th[0] = 0      # one lane with S = 0: clamps to K - 1
            u = (rng.integers(0, 1 << 24, W) * 2.0 ** -24).astype(np.float32)
            a = th.astype(np.float64) * ph.astype(np.float64)
            z_sim = bf.search_sim(bf.table_fp64(a, W), u, W)
            ids = np.arange(W, dtype=np.int32)
            z_def, band = oracle.draw_np(th, ph, ids, ids, u, band_rel=1e-12)
            assert ((z_sim == z_def) | band).all(), (W, K, z_sim, z_def)


# ---------------------------------------------------------------------------
# The alternative replacement [a b; c d] -> [a c; a+b c+d] (Section 4, the
# rule the paper says also works but costs more instructions on its GPU).

@pytest.mark.parametrize("W", [2, 4, 8, 16, 32, 64])
def test_alt_closed_form_equals_replacement_process(W):
    tab = bf.apply_replacements(bf.transposed_products(W),
                                bf.replacement_schedule(W), alt=True)
    for i in range(W):
        for j in range(W):
            z = tab[i][j]
            assert (z.thread, z.lo, z.hi) == bf.closed_form_alt(i, j)
    assert all(bf.closed_form_alt(W - 1, j) == (j, 0, W - 1) for j in range(W))


@pytest.mark.parametrize("W", [2, 4, 8, 16, 32, 64])
def test_alt_entries_are_left_halves_of_aligned_ranges(W):
    """Every entry above the last row sums the left half of an aligned range
    of 2**(s+1) topics (s = trailing ones of the row), and every thread finds
    each left half it can descend through exactly once."""
    seen = {}
    for i in range(W - 1):
        for j in range(W):
            t, lo, hi = bf.closed_form_alt(i, j)
            size = hi - lo + 1
            assert size & (size - 1) == 0 and lo % (2 * size) == 0
            assert ((i + 1) & ~i) == size      # row i has s trailing ones
            seen.setdefault(t, []).append((lo, hi))
    for t in range(W):
        want = sorted((lo, lo + size - 1) for size in (1 << s for s in range(W.bit_length() - 1))
                      for lo in range(0, W, 2 * size))
        assert sorted(seen[t]) == want


def test_alt_w2_holds_each_lanes_own_prefix():
    """With two lanes the alternative table is the untransposed prefix table:
    column j holds thread j's sums over topics 0..0 and 0..1."""
    for j in range(2):
        assert [bf.closed_form_alt(i, j) for i in range(2)] == [(j, 0, 0), (j, 0, 1)]
    assert bf.closed_form(0, 1) == (1, 1, 1)        # the paper's rule does not


@pytest.mark.parametrize("W", [8, 16, 64])
@pytest.mark.parametrize("K_extra", [0, 3])
def test_alt_numeric_table_equals_replacement(W, K_extra):
    rng = np.random.default_rng(7 * W + K_extra)
    K = 3 * W + K_extra
    a = rng.random((W, K))
    p = bf.table_alt_fp64(a, W)
    R = K % W
    for base in range(R, K, W):
        blk = [[a[t, base + c] for c in range(W)] for t in range(W)]
        tab = bf.apply_replacements(blk, bf.replacement_schedule(W), alt=True)
        for i in range(W - 1):
            for j in range(W):
                assert abs(tab[i][j] - p[j, base + i]) <= 1e-12 * (1 + abs(p[j, base + i]))


@pytest.mark.parametrize("W", [2, 4, 8, 16, 32, 64])
def test_alt_search_equals_definition(W):
    rng = np.random.default_rng(300 + W)
    for K in sorted({1, 3, max(1, W - 1), W, W + 1, 19, 2 * W, 2 * W + 3, 5 * W + 7}):
        for rep in range(3):
            th = rng.random((W, K)).astype(np.float32)
            ph = rng.random((W, K)).astype(np.float32)
            th[rng.random((W, K)) < 0.3] = 0
            if rep == 2:
                th[0] = 0
            u = (rng.integers(0, 1 << 24, W) * 2.0 ** -24).astype(np.float32)
            a = th.astype(np.float64) * ph.astype(np.float64)
            z_alt = bf.search_alt_sim(bf.table_alt_fp64(a, W), u, W)
            ids = np.arange(W, dtype=np.int32)
            z_def, band = oracle.draw_np(th, ph, ids, ids, u, band_rel=1e-12)
            assert ((z_alt == z_def) | band).all(), (W, K, z_alt, z_def)


def test_alt_search_needs_the_alt_table():
    """Run over the paper's table, the descent draws wrong topics: the two
    tables differ, so the pins above are not vacuous."""
    W, K = 8, 24
    rng = np.random.default_rng(1)
    a = rng.random((W, K))
    u = rng.random(W)
    ids = np.arange(W, dtype=np.int32)
    wrong = 0
    for rep in range(20):
        u = rng.random(W).astype(np.float32)
        a32 = rng.random((W, K)).astype(np.float32)
        a = a32.astype(np.float64)
        z_def, _ = oracle.draw_np(a32, np.ones((W, K), np.float32), ids, ids, u)
        wrong += (bf.search_alt_sim(bf.table_fp64(a, W), u, W) != z_def).sum()
        assert (bf.search_alt_sim(bf.table_alt_fp64(a, W), u, W) == z_def).all()
    assert wrong > 0
