"""Seeded synthetic LDA corpora for the per-token topic draw.

This module only draws inputs.  It holds none of the draw's arithmetic (no
products, sums or searches), so both the HIP path and the CPU oracle can take
their inputs from it without sharing any of the method.

Shapes follow the problem statement of Section 2 of the paper: theta is an
M x K row-major matrix of document-topic weights (rows are distributions),
phi is a V x K word-major matrix of topic-word weights (columns are
distributions), and the corpus is flattened to one (doc_id, word_id) pair per
token.  The uniform variate of step 3 of the draw is an input here (the paper
leaves the generator unspecified): u = i * 2**-24 with i uniform on
[0, 2**24), so every u is exact in fp32 and strictly below 1.

Distributions (synthetic stand-ins for the paper's Wikipedia corpus, which is
not used):
  * theta rows ~ Dirichlet(alpha), phi columns ~ Dirichlet(beta) over V, both by
    gamma-normalise in fp64 and then rounded to fp32;
  * word ids ~ finite Zipf(s) over ranks 1..V (word_id = rank - 1, so the
    vocabulary is frequency sorted);
  * doc ids sequential (tokens of one document are contiguous), with fixed or
    Poisson document lengths.
"""
from __future__ import annotations

import dataclasses
import hashlib
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

BASE_SEED = 20150513


@dataclasses.dataclass(frozen=True)
class CorpusConfig:
    """One synthetic workload.  ``doc_len`` is the fixed length of every
    document, or ``None`` with ``poisson_mean`` set for Poisson lengths."""

    name: str
    index: int
    M: int
    V: int
    K: int
    alpha: float
    beta: float
    zipf_s: float
    doc_len: int | None = None
    poisson_mean: float | None = None
    # lognormal document lengths rescaled to exactly `total_tokens` tokens and
    # clipped to [1, max_doc_len] (used for the corpus shaped like the paper's)
    lognormal_sigma: float | None = None
    total_tokens: int | None = None
    max_doc_len: int | None = None

    @property
    def nominal_tokens(self) -> int:
        if self.doc_len is not None:
            return self.M * self.doc_len
        if self.total_tokens is not None:
            return self.total_tokens
        return int(round(self.M * self.poisson_mean))


# The five workloads: sizes, Dirichlet parameters and Zipf exponents.
CONFIGS: dict[str, CorpusConfig] = {
    c.name: c
    for c in (
        CorpusConfig("tiny-K32", 0, M=64, V=1024, K=32, alpha=0.1, beta=0.01,
                     zipf_s=1.0, doc_len=64),
        CorpusConfig("corpus1M-K64", 1, M=8192, V=32768, K=64, alpha=0.1,
                     beta=0.01, zipf_s=1.0, doc_len=128),
        CorpusConfig("corpus1M-K256", 2, M=8192, V=32768, K=256, alpha=0.1,
                     beta=0.01, zipf_s=1.0, doc_len=128),
        CorpusConfig("corpus16M-K1024", 3, M=65536, V=100_000, K=1024,
                     alpha=0.1, beta=0.01, zipf_s=1.05, doc_len=256),
        CorpusConfig("poisson300-K2048", 4, M=32768, V=50_000, K=2048,
                     alpha=0.05, beta=0.01, zipf_s=1.0, poisson_mean=300.0),
    )
}


@dataclasses.dataclass
class Corpus:
    """Host arrays of one workload (all C-contiguous)."""

    theta: np.ndarray    # float32 [M][K]
    phi: np.ndarray      # float32 [V][K]
    doc_id: np.ndarray   # int32 [N]
    word_id: np.ndarray  # int32 [N]
    u: np.ndarray        # float32 [N], in [0, 1)
    name: str = "custom"

    @property
    def N(self) -> int:
        return int(self.doc_id.shape[0])

    @property
    def M(self) -> int:
        return int(self.theta.shape[0])

    @property
    def V(self) -> int:
        return int(self.phi.shape[0])

    @property
    def K(self) -> int:
        return int(self.theta.shape[1])


# Corpus shaped like the one the paper's evaluation (Section 5) describes:
# 43,556 documents, 37,286 distinct words, 3,072,662 tokens, at most 307 tokens
# per document.  Only these four counts come from the paper; the length
# distribution (lognormal, sigma 0.8), the Zipf exponent and the Dirichlet
# parameters are this generator's assumptions.  No text of any corpus is used.
WIKI_SHAPE = dict(M=43_556, V=37_286, total_tokens=3_072_662, max_doc_len=307,
                  lognormal_sigma=0.8, zipf_s=1.0, alpha=0.1, beta=0.01)
# K = 32 k + 16, 0 <= k <= 7: the topic counts of the paper's measurements.
WIKI_K = tuple(32 * k + 16 for k in range(8))


def wiki_shaped(K: int) -> CorpusConfig:
    """The paper-shaped corpus at K topics (index 100 + K selects its seeds)."""
    return CorpusConfig(f"wiki-shaped-K{K}", 100 + K, K=K, **WIKI_SHAPE)


for _K in WIKI_K:
    CONFIGS[f"wiki-shaped-K{_K}"] = wiki_shaped(_K)


def corpus16M_at(K: int) -> CorpusConfig:
    """The 16.8M-token corpus (65,536 documents of 256 tokens, V = 100,000,
    Zipf s = 1.05) at another topic count K (index 200 + K selects its
    seeds); used to measure where routing the tokens to the XCDs pays."""
    base = CONFIGS["corpus16M-K1024"]
    return dataclasses.replace(base, name=f"corpus16M-sweep-K{K}", index=200 + K, K=K)


def _lognormal_lengths(seed, M: int, sigma: float, total: int,
                       max_len: int) -> np.ndarray:
    """M lengths in [1, max_len] summing to exactly `total`: lognormal draws
    scaled to the target mean, clipped, then adjusted one token at a time on
    the documents with room (deterministic given the seed)."""
    g = np.random.Generator(np.random.PCG64(seed))
    x = g.lognormal(0.0, sigma, size=M)
    x *= total / x.sum()
    n = np.clip(np.rint(x), 1, max_len).astype(np.int64)
    order = g.permutation(M)
    i = 0
    while n.sum() != total:
        j = order[i % M]
        if n.sum() < total and n[j] < max_len:
            n[j] += 1
        elif n.sum() > total and n[j] > 1:
            n[j] -= 1
        i += 1
    return n


def _threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def _gamma_rows(seed: np.random.SeedSequence, shape: float, rows: int,
                cols: int, chunk_rows: int = 4096) -> np.ndarray:
    """fp64 Gamma(shape, 1) samples of size rows x cols.  Each chunk of rows has
    its own spawned seed, so the result does not depend on the thread count."""
    out = np.empty((rows, cols), dtype=np.float64)
    nchunks = (rows + chunk_rows - 1) // chunk_rows
    seeds = seed.spawn(nchunks)

    def fill(c: int) -> None:
        lo = c * chunk_rows
        hi = min(rows, lo + chunk_rows)
        g = np.random.Generator(np.random.PCG64(seeds[c]))
        out[lo:hi] = g.standard_gamma(shape, size=(hi - lo, cols))

    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(fill, range(nchunks)))
    return out


def dirichlet_rows(seed, alpha: float, rows: int, cols: int) -> np.ndarray:
    """Each row ~ Dirichlet(alpha * 1_cols), fp32.  A row whose gamma samples
    all underflow stays all-zero."""
    g = _gamma_rows(seed, alpha, rows, cols)
    s = g.sum(axis=1, keepdims=True)
    np.divide(g, s, out=g, where=s > 0)
    return g.astype(np.float32)


def dirichlet_columns(seed, beta: float, rows: int, cols: int) -> np.ndarray:
    """Each column ~ Dirichlet(beta * 1_rows), stored row-major [rows][cols]
    (word-major for phi), fp32."""
    g = _gamma_rows(seed, beta, rows, cols)
    s = g.sum(axis=0, keepdims=True)
    np.divide(g, s, out=g, where=s > 0)
    return g.astype(np.float32)


def zipf_ids(seed, s: float, V: int, N: int) -> np.ndarray:
    """N ids in [0, V) with P(id = r - 1) proportional to r**-s, r = 1..V."""
    g = np.random.Generator(np.random.PCG64(seed))
    w = np.arange(1, V + 1, dtype=np.float64) ** (-s)
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    ids = np.searchsorted(cdf, g.random(N), side="right")
    return np.minimum(ids, V - 1).astype(np.int32)


def uniforms_24bit(seed, N: int) -> np.ndarray:
    """u = i * 2**-24 with i uniform on [0, 2**24): exact in fp32, below 1."""
    g = np.random.Generator(np.random.PCG64(seed))
    i = g.integers(0, 1 << 24, size=N, dtype=np.int64)
    return (i.astype(np.float64) * 2.0 ** -24).astype(np.float32)


def _cache_path(cfg: CorpusConfig) -> str | None:
    root = os.environ.get("LDA_INPUT_CACHE")
    if not root:
        return None
    key = hashlib.sha1(repr((BASE_SEED, dataclasses.astuple(cfg))).encode())
    return os.path.join(root, f"{cfg.name}-{key.hexdigest()[:12]}.npz")


def make_corpus(cfg: CorpusConfig | str) -> Corpus:
    """Build a named workload from its fixed seed.  If ``LDA_INPUT_CACHE`` names
    a directory, the arrays are cached there as an uncompressed .npz."""
    if isinstance(cfg, str):
        cfg = CONFIGS[cfg]
    path = _cache_path(cfg)
    if path and os.path.exists(path):
        with np.load(path, allow_pickle=False) as f:
            return Corpus(f["theta"], f["phi"], f["doc_id"], f["word_id"],
                          f["u"], name=cfg.name)

    ss = np.random.SeedSequence(BASE_SEED + cfg.index)
    s_theta, s_phi, s_word, s_u, s_len = ss.spawn(5)
    if cfg.doc_len is not None:
        lengths = np.full(cfg.M, cfg.doc_len, dtype=np.int64)
    elif cfg.lognormal_sigma is not None:
        lengths = _lognormal_lengths(s_len, cfg.M, cfg.lognormal_sigma,
                                     cfg.total_tokens, cfg.max_doc_len)
    else:
        g = np.random.Generator(np.random.PCG64(s_len))
        lengths = g.poisson(cfg.poisson_mean, size=cfg.M).astype(np.int64)
    doc_id = np.repeat(np.arange(cfg.M, dtype=np.int32), lengths)
    N = int(doc_id.shape[0])
    corpus = Corpus(
        theta=dirichlet_rows(s_theta, cfg.alpha, cfg.M, cfg.K),
        phi=dirichlet_columns(s_phi, cfg.beta, cfg.V, cfg.K),
        doc_id=doc_id,
        word_id=zipf_ids(s_word, cfg.zipf_s, cfg.V, N),
        u=uniforms_24bit(s_u, N),
        name=cfg.name,
    )
    if path:
        os.makedirs(os.path.dirname(path), exist_ok=True)
        tmp = path + ".tmp.npz"
        np.savez(tmp, theta=corpus.theta, phi=corpus.phi, doc_id=corpus.doc_id,
                 word_id=corpus.word_id, u=corpus.u)
        os.replace(tmp, path)
    return corpus


def doc_offsets(doc_id: np.ndarray, M: int) -> np.ndarray:
    """The ragged (CSR) form of a corpus whose documents are contiguous:
    int64 [M + 1], document m holding tokens offsets[m] .. offsets[m+1]-1."""
    doc_id = np.asarray(doc_id)
    if doc_id.size and (np.diff(doc_id) < 0).any():
        raise ValueError("documents are not contiguous (doc_id decreases)")
    counts = np.bincount(doc_id, minlength=M).astype(np.int64)
    return np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)


def make_random(N: int, M: int, V: int, K: int, seed: int, *, alpha=0.1,
                beta=0.01, zipf_s=1.0, doc_order: str = "sequential") -> Corpus:
    """A small corpus of arbitrary shape for parity and edge-case tests.

    ``doc_order``: "sequential" (contiguous runs of near-equal length),
    "ragged" (contiguous runs of Dirichlet-multinomial lengths, many of them
    zero), "shuffled" (random doc id per token) or "single" (every token in
    doc 0).
    """
    ss = np.random.SeedSequence([BASE_SEED, 7, seed, N, M, V, K])
    s_theta, s_phi, s_word, s_u, s_doc = ss.spawn(5)
    if doc_order == "sequential":
        doc_id = (np.arange(N, dtype=np.int64) * M // max(N, 1)).astype(np.int32)
    elif doc_order == "ragged":
        g = np.random.Generator(np.random.PCG64(s_doc))
        lengths = g.multinomial(N, g.dirichlet(np.full(M, 0.3)))
        doc_id = np.repeat(np.arange(M, dtype=np.int32), lengths)
    elif doc_order == "shuffled":
        g = np.random.Generator(np.random.PCG64(s_doc))
        doc_id = g.integers(0, M, size=N, dtype=np.int64).astype(np.int32)
    elif doc_order == "single":
        doc_id = np.zeros(N, dtype=np.int32)
    else:
        raise ValueError(doc_order)
    return Corpus(
        theta=dirichlet_rows(s_theta, alpha, M, K),
        phi=dirichlet_columns(s_phi, beta, V, K),
        doc_id=doc_id,
        word_id=zipf_ids(s_word, zipf_s, V, N),
        u=uniforms_24bit(s_u, N),
        name=f"random-N{N}-M{M}-V{V}-K{K}-{doc_order}",
    )
