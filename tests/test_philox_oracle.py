"""Pins of the oracle's Philox generators (the uniforms of the fused-RNG
draw) against the generator's published known-answer vectors and against
numpy's independent Philox4x64-10."""
import os

import numpy as np
import pytest

from conftest import GOLDEN
from oracle import philox as px


def _kat():
    rows = []
    with open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")) as f:
        for ln in f:
            if ln.strip() and not ln.startswith("#"):
                v = [int(x, 16) for x in ln.split()]
                rows.append((tuple(v[:4]), tuple(v[4:6]), tuple(v[6:10])))
    return rows


def test_philox4x32_known_answers():
    rows = _kat()
    assert len(rows) == 3
    for ctr, key, out in rows:
        assert px.philox4(ctr, key, 32) == out


def test_philox4x32_vector_form_known_answers():
    for ctr, key, out in _kat():
        got = px.philox4x32_np(*(np.array([c], np.uint32) for c in ctr), *key)
        assert tuple(int(g[0]) for g in got) == out


def test_fewer_rounds_differ():
    """The round count matters (the pins above are not vacuous)."""
    ctr, key, out = _kat()[2]
    assert px.philox4(ctr, key, 32, rounds=9) != out
    assert px.philox4(ctr, key, 32, rounds=10) == out


@pytest.mark.parametrize("seed", [0, 1, 20150513])
def test_philox4x64_equals_numpy(seed):
    """The same round structure with 64-bit words equals numpy's Philox
    (which advances its counter by one before each block)."""
    rng = np.random.default_rng(seed)
    for _ in range(20):
        key = tuple(int(k) for k in rng.integers(0, 2 ** 63, 2, dtype=np.uint64) * 2
                    + rng.integers(0, 2, 2, dtype=np.uint64))
        ctr = [int(c) for c in rng.integers(0, 2 ** 63, 4, dtype=np.uint64)]
        if _ % 4 == 0:
            ctr[0] = 2 ** 64 - 1          # the increment carries into word 1
        bg = np.random.Philox(counter=np.array(ctr, np.uint64),
                              key=np.array(key, np.uint64))
        raw = tuple(int(x) for x in bg.random_raw(4))
        nxt = list(ctr)
        nxt[0] = (nxt[0] + 1) % 2 ** 64
        if nxt[0] == 0:
            nxt[1] = (nxt[1] + 1) % 2 ** 64
        assert px.philox4(nxt, key, 64) == raw


def test_vector_form_equals_scalar_form():
    rng = np.random.default_rng(3)
    c = rng.integers(0, 2 ** 32, (4, 200), dtype=np.uint64).astype(np.uint32)
    k0, k1 = (int(x) for x in rng.integers(0, 2 ** 32, 2))
    vec = px.philox4x32_np(c[0], c[1], c[2], c[3], k0, k1)
    for i in range(0, 200, 7):
        assert tuple(int(v[i]) for v in vec) == px.philox4(c[:, i], (k0, k1), 32)


def test_token_uniforms_convention():
    """u of token n = top 24 bits of word 0 of Philox4x32-10 at counter
    (n lo, n hi, sweep, 0) and key (seed lo, seed hi), times 2^-24."""
    seed, sweep = 0x0123456789ABCDEF, 7
    first = 2 ** 32 - 5                    # tokens across the 2^32 boundary
    u = px.token_uniforms(seed, sweep, first, 10)
    for i in range(10):
        n = first + i
        y0 = px.philox4((n & 0xFFFFFFFF, n >> 32, sweep, 0),
                        (seed & 0xFFFFFFFF, seed >> 32), 32)[0]
        assert u[i] == np.float32((y0 >> 8) * 2.0 ** -24)


def test_token_uniforms_are_uniform_24_bit():
    u = px.token_uniforms(20150513, 0, 0, 1 << 20).astype(np.float64)
    assert u.min() >= 0.0 and u.max() < 1.0
    assert (u * 2 ** 24 == np.floor(u * 2 ** 24)).all()
    from scipy import stats
    counts = np.bincount((u * 64).astype(int), minlength=64)
    assert stats.chisquare(counts).pvalue > 1e-4
    # streams of other sweeps and seeds differ
    assert (px.token_uniforms(20150513, 1, 0, 1000) != u[:1000]).mean() > 0.99
    assert (px.token_uniforms(20150514, 0, 0, 1000) != u[:1000]).mean() > 0.99
