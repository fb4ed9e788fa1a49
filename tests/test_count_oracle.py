"""Pins of the oracle's topic counts (the statistics the update of theta and
phi consumes after the draw; Section 1 and the uncollapsed sampler of
Section 2).

The counts are integer and exact, so the pins are a hand-counted fixture
(``tests/golden/counts_hand_M3_V4_K3.txt``), the identities every count table
satisfies (totals, document lengths, word frequencies, topic totals), brute
force over every cell on tiny inputs, and the rule for tokens out of range.
``MUTANTS`` plants plausible mistakes in copies of the counting and checks
that each fails at least one pin.
"""
import os

import numpy as np
import pytest

import oracle
from conftest import GOLDEN


def load_hand_fixture():
    toks, ndk, nwk = [], {}, {}
    with open(os.path.join(GOLDEN, "counts_hand_M3_V4_K3.txt")) as f:
        for ln in f:
            ln = ln.strip()
            if not ln or ln.startswith("#"):
                continue
            head, _, rest = ln.partition(" ")
            if head == "token":
                toks.append([int(x) for x in rest.split()])
            else:
                row, _, vals = rest.partition(":")
                (ndk if head == "ndk" else nwk)[int(row)] = [int(x) for x in vals.split()]
    t = np.array(toks, np.int32)
    return (t[:, 0], t[:, 1], t[:, 2],
            np.array([ndk[d] for d in sorted(ndk)], np.int32),
            np.array([nwk[w] for w in sorted(nwk)], np.int32))


def c_counts(d, w, z, M, V, K):
    return oracle.counts(d, w, z, M, V, K)


def np_counts(d, w, z, M, V, K):
    return oracle.counts_np(d, w, z, M, V, K)


# Plausible mistakes, each in a copy of the counting (never in the oracle).
def _mut_transposed(d, w, z, M, V, K):        # cells laid out [k][d], read as [d][k]
    ndk, nwk = oracle.counts_np(d, w, z, M, V, K)
    return (np.ascontiguousarray(ndk.T).reshape(M, K),
            np.ascontiguousarray(nwk.T).reshape(V, K))


def _mut_swapped(d, w, z, M, V, K):           # documents and words exchanged
    ndk, nwk = oracle.counts_np(np.minimum(w, M - 1), np.minimum(d, V - 1), z, M, V, K)
    return ndk, nwk


def _mut_topic_off_by_one(d, w, z, M, V, K):  # topic k counted in cell k + 1 (mod K)
    return oracle.counts_np(d, w, (np.asarray(z) + 1) % K, M, V, K)


def _mut_not_cleared(d, w, z, M, V, K):       # counts added onto a previous table
    ndk, nwk = oracle.counts_np(d, w, z, M, V, K)
    return ndk + 1, nwk + 1


def _mut_presence(d, w, z, M, V, K):          # a cell counts 1 however many tokens
    ndk, nwk = oracle.counts_np(d, w, z, M, V, K)
    return (ndk > 0).astype(np.int32), (nwk > 0).astype(np.int32)


def _mut_drops_last(d, w, z, M, V, K):        # last token not counted
    return oracle.counts_np(d[:-1], w[:-1], z[:-1], M, V, K)


def _mut_counts_out_of_range(d, w, z, M, V, K):  # topic K folded into K - 1
    return oracle.counts_np(d, w, np.minimum(z, K - 1), M, V, K)


MUTANTS = [_mut_transposed, _mut_swapped, _mut_topic_off_by_one, _mut_not_cleared,
           _mut_presence, _mut_drops_last, _mut_counts_out_of_range]


def _random_case(seed, N, M, V, K, bad=0):
    rng = np.random.default_rng(seed)
    d = rng.integers(0, M, N).astype(np.int32)
    w = rng.integers(0, V, N).astype(np.int32)
    z = rng.integers(0, K, N).astype(np.int32)
    if bad:
        i = rng.choice(N, bad, replace=False)
        d[i[0::3]] = -1
        z[i[1::3]] = K
        w[i[2::3]] = V
    return d, w, z


# ---------------------------------------------------------------------------
# the pins, as functions of a counting function (so that mutants can be run
# through them)
def pin_hand_fixture(fn):
    d, w, z, ndk, nwk = load_hand_fixture()
    a, b = fn(d, w, z, 3, 4, 3)
    return np.array_equal(a, ndk) and np.array_equal(b, nwk)


def pin_identities(fn):
    for seed, (N, M, V, K) in enumerate([(1000, 7, 13, 5), (5000, 40, 300, 64),
                                         (777, 3, 2, 1), (0, 4, 5, 6)]):
        d, w, z = _random_case(seed, N, M, V, K)
        ndk, nwk = fn(d, w, z, M, V, K)
        if ndk.shape != (M, K) or nwk.shape != (V, K):
            return False
        if ndk.sum() != N or nwk.sum() != N:
            return False
        if not np.array_equal(ndk.sum(1), np.bincount(d, minlength=M)):
            return False                     # a document's tokens: its length
        if not np.array_equal(nwk.sum(1), np.bincount(w, minlength=V)):
            return False                     # a word's tokens: its frequency
        topic = np.bincount(z, minlength=K)
        if not (np.array_equal(ndk.sum(0), topic) and np.array_equal(nwk.sum(0), topic)):
            return False                     # both tables give the topic totals
        if (ndk < 0).any() or (nwk < 0).any():
            return False
    return True


def pin_brute_force(fn):
    for seed, (N, M, V, K) in enumerate([(40, 3, 4, 3), (64, 2, 5, 7), (9, 4, 3, 2)]):
        d, w, z = _random_case(100 + seed, N, M, V, K)
        ndk, nwk = fn(d, w, z, M, V, K)
        for m in range(M):
            for k in range(K):
                if ndk[m, k] != sum(1 for n in range(N) if d[n] == m and z[n] == k):
                    return False
        for v in range(V):
            for k in range(K):
                if nwk[v, k] != sum(1 for n in range(N) if w[n] == v and z[n] == k):
                    return False
    return True


def pin_out_of_range(fn):
    """Tokens whose document, word or topic is out of range are not counted;
    the others are."""
    d = np.array([0, -1, 1, 1, 0, 2], np.int32)
    w = np.array([1, 1, 4, 0, 0, 1], np.int32)
    z = np.array([2, 0, 1, 3, 0, 1], np.int32)
    M, V, K = 2, 4, 3                       # tokens 1 (d), 2 (w), 3 (z), 5 (d) out
    ndk, nwk = fn(d, w, z, M, V, K)
    e_ndk = np.zeros((M, K), np.int32)
    e_nwk = np.zeros((V, K), np.int32)
    for n in (0, 4):
        e_ndk[d[n], z[n]] += 1
        e_nwk[w[n], z[n]] += 1
    return np.array_equal(ndk, e_ndk) and np.array_equal(nwk, e_nwk)


PINS = [pin_hand_fixture, pin_identities, pin_brute_force, pin_out_of_range]


@pytest.mark.parametrize("fn", [c_counts, np_counts], ids=["c", "numpy"])
@pytest.mark.parametrize("pin", PINS, ids=lambda p: p.__name__)
def test_oracle_counts_pinned(fn, pin):
    assert pin(fn)


@pytest.mark.parametrize("mutant", MUTANTS, ids=lambda m: m.__name__)
def test_every_mutant_fails_a_pin(mutant):
    assert not all(pin(mutant) for pin in PINS), mutant.__name__


@pytest.mark.parametrize("shape", [(20000, 50, 700, 33), (4096, 64, 1024, 32),
                                   (30000, 9, 20, 256)])
def test_c_equals_numpy_twin(shape):
    N, M, V, K = shape
    d, w, z = _random_case(sum(shape), N, M, V, K, bad=30)
    a = oracle.counts(d, w, z, M, V, K)
    b = oracle.counts_np(d, w, z, M, V, K)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_counts_of_oracle_draws_on_tiny_config():
    """The counts of the oracle's own draws on the tiny workload: the
    identities hold, and every document and word has exactly its tokens."""
    from paper_1505_03851_amd.inputs import make_corpus
    c = make_corpus("tiny-K32")
    z = oracle.draw(c.theta, c.phi, c.doc_id, c.word_id, c.u, with_band=False)
    ndk, nwk = oracle.counts(c.doc_id, c.word_id, z, c.M, c.V, c.K)
    assert ndk.sum() == c.N == nwk.sum()
    assert np.array_equal(ndk.sum(1), np.bincount(c.doc_id, minlength=c.M))
    assert np.array_equal(ndk.sum(0), nwk.sum(0))
    # a topic of zero weight for a token's document is never that token's draw
    assert (ndk[c.theta == 0] == 0).all()
