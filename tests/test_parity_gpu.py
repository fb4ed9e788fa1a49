"""GPU parity: every kernel against the CPU oracle, through the C ABI.

Rule: z equals the oracle's bit for bit except at tokens where
|u*S - S_k| <= 1e-5 * S for some k (fp32 rounding may move such a draw to a
neighbouring topic); the rate of such exceptions must stay below 1e-4 on the
full-size workloads.  Every workload runs the kernel on every token, the
full-size ones in the benchmark's launch configuration, and every token is
checked against the oracle.
"""
import numpy as np
import pytest

from paper_1505_03851_amd.inputs import WIKI_K, Corpus, make_random
from parity import (MAX_MISMATCH_RATE, compare, named_corpus, reference, run_kernel,
                    to_device)

pytestmark = pytest.mark.gpu

KERNELS = ["naive", "butterfly", "transposed",
           "variant-register", "variant-lds", "variant-lds_alt", "variant-leaf8", "variant-wide"]


def _check(c, kernel, idx=None, rate=True, ref=None):
    print(f"[case] {c.name} kernel={kernel} N={c.N} K={c.K}", flush=True)
    z = run_kernel(kernel, to_device(c))
    assert z.min() >= 0 and z.max() < c.K
    rep = compare(c, z, idx, ref=ref)
    print(f"[parity] {c.name} {kernel}: {rep}", flush=True)
    assert rep.hard == 0, rep.first_hard
    if rate:
        assert rep.mismatch_rate < MAX_MISMATCH_RATE, str(rep)
    return rep


def corpus(name):
    return named_corpus(name)


@pytest.mark.parametrize("kernel", KERNELS)
@pytest.mark.parametrize("name", ["tiny-K32", "corpus1M-K64", "corpus1M-K256",
                                  "corpus16M-K1024", "poisson300-K2048"])
def test_config_every_token(name, kernel):
    """Every token of each of the five workloads, in the launch configuration
    the benchmark times, against the oracle (computed once per workload)."""
    c = corpus(name)
    _check(c, kernel, rate=c.N >= 1 << 20, ref=reference(name))


@pytest.mark.parametrize("K", [260, 384, 508])
def test_corpus16M_eight_topic_leaves_every_token(K):
    """The 16.8M-token corpus (V = 100,000, Zipf 1.05) at K from 260 to 508,
    where the draw takes 64-lane groups of 8-topic leaves: every token against
    the oracle, under the band rule and the mismatch-rate bound."""
    from paper_1505_03851_amd.inputs import corpus16M_at, make_corpus
    _check(make_corpus(corpus16M_at(K)), "butterfly")


@pytest.mark.parametrize("kernel", KERNELS)
@pytest.mark.parametrize("K", WIKI_K)
def test_wiki_shaped_every_token(K, kernel):
    """The corpus shaped like the paper's evaluation corpus (3.07M tokens,
    documents of 1..307 tokens), at all eight topic counts of the paper's
    measurements (K = 32k + 16); every K here has a remnant (K mod 64 = 16
    or 48)."""
    from paper_1505_03851_amd.inputs import wiki_shaped
    name = wiki_shaped(K).name
    _check(corpus(name), kernel, ref=reference(name))


SHAPES = [
    # (N, M, V, K, doc order)
    (1, 1, 7, 64, "sequential"),
    (63, 5, 50, 1, "sequential"),
    (65, 5, 50, 2, "shuffled"),
    (64 * 9 + 17, 40, 300, 7, "shuffled"),
    (64 * 9 + 17, 40, 300, 19, "sequential"),
    (64 * 9 + 17, 40, 300, 31, "single"),
    (64 * 21 + 5, 40, 300, 32, "sequential"),
    (64 * 21 + 5, 40, 300, 33, "shuffled"),
    (64 * 21 + 5, 40, 300, 50, "sequential"),
    (64 * 21 + 5, 40, 300, 63, "shuffled"),
    (64 * 21 + 5, 40, 300, 64, "shuffled"),
    (64 * 21 + 5, 40, 300, 65, "sequential"),
    (64 * 33 + 1, 60, 500, 100, "shuffled"),
    (64 * 33 + 63, 30, 500, 128, "sequential"),
    (64 * 33 + 63, 60, 500, 200, "shuffled"),
    (64 * 33 + 63, 60, 500, 240, "single"),
    (64 * 17 + 9, 60, 500, 1000, "sequential"),
    (64 * 17 + 9, 60, 500, 2047, "shuffled"),
    # K from 1536 to 2048 divisible by 4: the leaf kernel with six to eight
    # 256-topic blocks (its second launch shape), with and without a padded
    # first block, one, two and many documents per wave
    (64 * 13 + 7, 30, 400, 1536, "sequential"),
    (64 * 10 + 1, 30, 300, 1664, "shuffled"),
    (64 * 9 + 40, 3, 100, 1792, "single"),
    (64 * 11 + 3, 20, 300, 1900, "sequential"),
    (64 * 8 + 63, 9, 200, 2048, "sequential"),
    # K not divisible by 4: the one-topic kernel, with the half-block tail
    # from 2 to 32 blocks of 64 topics (a remnant in front), and the
    # full-block rebuild above 32 blocks
    (64 * 9 + 5, 30, 400, 130, "sequential"),
    (64 * 7 + 40, 9, 300, 513, "shuffled"),
    (64 * 6 + 3, 3, 200, 1023, "single"),
    (64 * 8 + 17, 20, 300, 1535, "sequential"),
    (64 * 5 + 60, 9, 200, 1901, "sequential"),
    (64 * 4 + 9, 5, 100, 2111, "shuffled"),
    (64 * 3 + 1, 4, 100, 3001, "sequential"),
    # K divisible by 4 but not by 256: the leaf kernel with empty topics in
    # front of its first 256-topic block (one, two and many documents per wave)
    (64 * 11 + 7, 13, 300, 1000, "sequential"),
    (64 * 7 + 50, 9, 200, 516, "shuffled"),
    (64 * 6 + 1, 4, 150, 2044, "single"),
    (64 * 9 + 3, 30, 300, 1604, "sequential"),
    (64 * 5 + 30, 3, 100, 772, "sequential"),
    (64 * 5 + 3, 20, 200, 4096, "sequential"),
    # one-document wavefronts up to K = 1024 stage their theta row in LDS for
    # the rebuild: with and without empty leading topics
    (64 * 8 + 50, 2, 200, 260, "single"),
    (64 * 6 + 20, 3, 200, 768, "single"),
    (64 * 7 + 11, 2, 200, 1020, "single"),
    # K divisible by 4 up to 128: the leaf-group kernel (groups of 8, 16 or
    # 32 lanes, empty leaves in front when K is below 32, 64 or 128), with
    # every group inside one document (long documents) or not
    (64 * 5 + 9, 2, 40, 4, "sequential"),
    (64 * 6 + 1, 50, 90, 12, "shuffled"),
    (64 * 9 + 30, 4, 120, 20, "sequential"),
    (64 * 9 + 30, 90, 120, 36, "sequential"),
    (64 * 7 + 2, 1, 300, 48, "single"),
    (64 * 8 + 63, 70, 300, 84, "sequential"),
    (64 * 8 + 5, 3, 300, 96, "sequential"),
    (64 * 12 + 11, 40, 300, 124, "ragged"),
    (64, 3, 64, 128, "shuffled"),
    # documents of 17-40 tokens: groups spanning one, two or more runs of
    # documents (the leaf-group kernel's theta leaf per run, up to 2 runs per
    # group below 64 lanes and 4 for 64 lanes, else a leaf per token)
    (64 * 20 + 7, 32, 300, 64, "sequential"),
    (64 * 20 + 7, 64, 300, 128, "sequential"),
    (64 * 30 + 5, 60, 300, 200, "sequential"),
    (64 * 30 + 5, 110, 300, 256, "sequential"),
    # K divisible by 4 from 260 to 508 (multiples of 32 up to 416): groups of
    # 64 lanes with 8-topic leaves, empty topics in front below 512 (a whole
    # empty quad when K mod 8 = 4), every group in one document, in up to
    # three runs, or more; 448 and N < 64 go to the other kernels
    (64 * 9 + 5, 40, 300, 264, "sequential"),
    (64 * 12 + 3, 3, 300, 300, "single"),
    (64 * 10 + 1, 30, 200, 384, "shuffled"),
    (64 * 8 + 9, 12, 300, 416, "sequential"),
    (64 * 30 + 5, 100, 300, 352, "sequential"),
    (64 * 6 + 7, 4, 200, 508, "ragged"),
    (64 * 5, 2, 100, 500, "single"),
    (64 * 7 + 30, 9, 300, 448, "sequential"),
    (40, 3, 50, 300, "shuffled"),
    # K a multiple of 256 (the leaf kernel with 32-topic prefix rows up to 2048)
    (1, 1, 7, 256, "sequential"),
    (63, 5, 50, 512, "shuffled"),
    (65, 5, 50, 768, "sequential"),
    (64 * 7 + 5, 3, 90, 1280, "sequential"),   # waves spanning two documents
    (64 * 9, 9, 100, 2304, "single"),
    (64 * 9 + 33, 40, 100, 512, "shuffled"),
]


@pytest.mark.parametrize("kernel", KERNELS)
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "N{}-K{}-{}".format(s[0], s[3], s[4]))
def test_edge_shapes(shape, kernel):
    N, M, V, K, order = shape
    c = make_random(N, M, V, K, seed=N + K, doc_order=order)
    _check(c, kernel, rate=False)


def _corpus(theta, phi, doc, word, u, name):
    return Corpus(np.ascontiguousarray(theta, np.float32),
                  np.ascontiguousarray(phi, np.float32),
                  np.ascontiguousarray(doc, np.int32),
                  np.ascontiguousarray(word, np.int32),
                  np.ascontiguousarray(u, np.float32), name=name)


def _grid_u(N, seed):
    rng = np.random.default_rng(seed)
    u = (rng.integers(0, 1 << 24, N) * 2.0 ** -24).astype(np.float32)
    u[:4] = [0.0, 2.0 ** -24, 0.5, 1 - 2.0 ** -24]
    return u


@pytest.mark.parametrize("kernel", KERNELS)
@pytest.mark.parametrize("K", [8, 32, 64, 256, 1024, 4096])
def test_equal_power_of_two_weights_exact(K, kernel):
    """All products 2**-3: every fp32 partial sum is exact, so z = floor(u*K)
    exactly, with no rounding band."""
    import paper_1505_03851_amd as lda
    N = 64 * 37 + 11
    u = _grid_u(N, K)
    c = _corpus(np.full((3, K), 2.0 ** -3), np.ones((5, K)),
                np.arange(N) % 3, np.arange(N) % 5, u, f"pow2-K{K}")
    print(f"[case] {c.name} kernel={kernel}", flush=True)
    z = run_kernel(kernel, to_device(c))
    expect = np.floor(u.astype(np.float64) * K).astype(np.int32)
    assert (z == expect).all(), np.nonzero(z != expect)[0][:10]


@pytest.mark.parametrize("kernel", KERNELS)
@pytest.mark.parametrize("K", [20, 50, 100, 130, 144, 208, 240, 260, 300, 508, 1000, 2044,
                               2047])
def test_tiny_uniforms_with_empty_leading_topics(K, kernel):
    """Every u is 0 or a few multiples of 2**-24, at K whose kernels pad the
    front of the first block (or leaf group) with empty topics: the search
    rebuilds prefixes as low + y or high - y, and near the empty topics (true
    prefix 0) that may round above such a stop; no draw may then land on an
    empty topic (z < 0), and every mismatch must lie inside the band.  (A
    u = 0 token at K = 208 drew z = -25 before the search was bounded by the
    first real topic.)"""
    N = 64 * 40 + 7
    c = make_random(N, 30, 400, K, seed=K + 3, doc_order="sequential")
    c.u[:] = ((np.arange(N) % 8) * 2.0 ** -24).astype(np.float32)
    rep = _check(c, kernel, rate=False)
    assert rep.hard == 0


@pytest.mark.parametrize("kernel", KERNELS)
@pytest.mark.parametrize("K", [4, 8, 20, 32, 48, 64, 100, 256, 300, 1000, 1024, 2048])
def test_uniforms_just_below_one_with_empty_trailing_topics(K, kernel):
    """Every u is 1 - j 2**-24 (j = 1 ... 8), and half the words give their
    last three topics zero weight.  stop = u S then lies within a few ulps of
    S, inside the rounding band of every token, so the band rule alone would
    admit any topic; the draw must instead be a topic whose prefix range
    [S_{z-1}, S_z] comes within the band of stop (in fp64): the last topic of
    nonzero weight, a trailing empty one (rounding, or S = 0: K - 1), or one
    whose whole weight is below the band, never an earlier topic."""
    import oracle
    N = 64 * 40 + 7
    c = make_random(N, 30, 400, K, seed=K + 11, doc_order="sequential")
    c.phi[::2, max(K - 3, 1):] = 0.0
    c.u[:] = (1.0 - ((np.arange(N) % 8) + 1) * 2.0 ** -24).astype(np.float32)
    print(f"[case] near-one-K{K} kernel={kernel}", flush=True)
    z = run_kernel(kernel, to_device(c))
    assert z.min() >= 0 and z.max() < K
    S = np.cumsum(c.theta[c.doc_id].astype(np.float64) *
                  c.phi[c.word_id].astype(np.float64), axis=1)
    total = S[:, -1]
    stop = c.u.astype(np.float64) * total
    tol = oracle.BAND_REL * total
    rows = np.arange(N)
    below = np.where(z > 0, S[rows, np.maximum(z - 1, 0)], 0.0)   # S_{z-1}
    ok = (below <= stop + tol) & ((S[rows, z] >= stop - tol) | (z == K - 1))
    assert ok.all(), [(int(i), int(z[i])) for i in np.nonzero(~ok)[0][:5]]


@pytest.mark.parametrize("kernel", KERNELS)
@pytest.mark.parametrize("K", [1, 5, 32, 64, 100, 300, 508, 1000, 1024])
def test_degenerate_weights(K, kernel):
    """All-zero documents draw K-1; a one-hot document draws its topic for
    every u (including u = 0 and u = 1 - 2**-24); mixed with normal rows."""
    N = 64 * 11 + 7
    rng = np.random.default_rng(K)
    theta = rng.random((4, K)).astype(np.float32)
    theta[1] = 0.0                         # S = 0
    theta[2] = 0.0
    theta[2, K // 2] = 0.25                # one-hot
    phi = rng.random((6, K)).astype(np.float32) + 0.01
    doc = rng.integers(0, 4, N)
    word = rng.integers(0, 6, N)
    u = _grid_u(N, K + 1)
    c = _corpus(theta, phi, doc, word, u, f"degenerate-K{K}")
    rep = _check(c, kernel, rate=False)
    z = run_kernel(kernel, to_device(c))
    assert (z[doc == 1] == K - 1).all()
    assert (z[doc == 2] == K // 2).all()
    assert rep.hard == 0


# ---------------------------------------------------------------------------
# Documents as offsets (the ragged corpus of Section 2): "docs" runs the
# token-per-lane kernels, each lane finding its document in the offsets;
# "doc_lanes" is Algorithm 7's document-per-lane driver.

OFFSET_KERNELS = ["docs", "doc_lanes", "doc_lanes_cache"]


def _offset_check(c, kernel, **kw):
    """As _check; the theta cache of the document-per-lane driver takes
    K <= 256 and must refuse larger K."""
    if kernel == "doc_lanes_cache" and c.K > 256:
        import paper_1505_03851_amd as lda
        with pytest.raises(lda.LdaError) as e:
            run_kernel(kernel, to_device(c))
        assert e.value.status == lda.STATUS["LDA_ERR_UNSUPPORTED"]
        return None
    return _check(c, kernel, **kw)


@pytest.mark.parametrize("kernel", OFFSET_KERNELS)
@pytest.mark.parametrize("name", ["tiny-K32", "corpus1M-K64", "corpus1M-K256"])
def test_docs_config_every_token(name, kernel):
    c = corpus(name)
    _offset_check(c, kernel, rate=c.N >= 1 << 20)


@pytest.mark.parametrize("kernel", OFFSET_KERNELS)
@pytest.mark.parametrize("K", WIKI_K)
def test_docs_wiki_shaped_every_token(K, kernel):
    """Lognormal document lengths of 1..307 tokens: for the document-per-lane
    driver most lanes of a wavefront repeat their last token for many
    iterations."""
    from paper_1505_03851_amd.inputs import wiki_shaped
    _offset_check(corpus(wiki_shaped(K).name), kernel)


def test_docs_full_size_equals_doc_ids():
    """At full size the offsets form gives the same z as the doc-id form,
    token for token (same kernel, same arithmetic), and every token matches
    the oracle under the band rule."""
    name = "corpus16M-K1024"
    c = corpus(name)
    dev = to_device(c)
    print(f"[case] {c.name} docs vs butterfly", flush=True)
    z_docs = run_kernel("docs", dev)
    z_ids = run_kernel("butterfly", dev)
    assert (z_docs == z_ids).all(), np.nonzero(z_docs != z_ids)[0][:10]
    rep = compare(c, z_docs, ref=reference(name))
    print(f"[parity] {c.name} docs: {rep}", flush=True)
    assert rep.hard == 0, rep.first_hard
    assert rep.mismatch_rate < MAX_MISMATCH_RATE


@pytest.mark.parametrize("name", ["corpus16M-K1024", "poisson300-K2048"])
def test_doc_lanes_full_size_every_token(name):
    """The document-per-lane driver on the full-size corpora (fixed and
    Poisson(300) lengths), every token against the oracle."""
    _check(corpus(name), "doc_lanes", ref=reference(name))


RAGGED = [
    # (N, M, V, K): Dirichlet(0.3) lengths, many documents empty
    (1, 3, 7, 64),
    (63, 40, 50, 5),
    (64 * 9 + 17, 200, 300, 19),
    (64 * 21 + 5, 2000, 300, 64),     # more documents than tokens
    (64 * 21 + 5, 40, 300, 65),
    (64 * 33 + 63, 60, 500, 128),
    (64 * 33 + 63, 60, 500, 129),
    (64 * 33 + 63, 60, 500, 200),
    (64 * 9 + 33, 40, 100, 256),      # leaf kernel, one block
    (64 * 11 + 7, 50, 300, 300),      # 64-lane groups of 8-topic leaves
    (64 * 8 + 40, 9, 200, 436),
    (64 * 7 + 5, 300, 90, 1280),
    (64 * 17 + 9, 60, 500, 2047),
    (64 * 5 + 3, 20, 200, 4096),
    (64 * 40, 130, 400, 96),          # M past two full wavefronts of documents
]


@pytest.mark.parametrize("kernel", OFFSET_KERNELS)
@pytest.mark.parametrize("shape", RAGGED, ids=lambda s: "N{}-M{}-K{}".format(s[0], s[1], s[3]))
def test_docs_ragged(shape, kernel):
    N, M, V, K = shape
    c = make_random(N, M, V, K, seed=N + M + K, doc_order="ragged")
    _offset_check(c, kernel, rate=False)
    if kernel == "docs":
        # same kernel as the doc-id form: identical z
        assert (run_kernel("docs", to_device(c)) == run_kernel("butterfly", to_device(c))).all()


@pytest.mark.parametrize("kernel", OFFSET_KERNELS)
@pytest.mark.parametrize("layout", ["huge-first", "huge-last", "huge-middle", "alternating"])
@pytest.mark.parametrize("NM", [(64 * 50 + 13, 300), (64 * 400 + 13, 6000)],
                         ids=lambda s: f"N{s[0]}-M{s[1]}")
def test_docs_skewed_lengths(layout, kernel, NM):
    """Document lengths far from uniform, so that a wavefront's guess of its
    first document (token index * M / N) is far off in either direction (by
    thousands of documents at M = 6000)."""
    (N, M), V, K = NM, 400, 96
    lengths = np.zeros(M, np.int64)
    if layout == "huge-first":
        lengths[0] = N - (M - 1)
        lengths[1:] = 1
    elif layout == "huge-last":
        lengths[-1] = N - (M - 1)
        lengths[:-1] = 1
    elif layout == "huge-middle":
        lengths[:] = 1
        lengths[M // 2] = N - (M - 1)
        lengths[M // 2 + 1: M // 2 + 40] = 0
        lengths[M // 2] += 39
    else:   # empty and long documents in turn
        lengths[1::2] = 0
        lengths[0::2] = N // (M // 2)
        lengths[0] += N - lengths.sum()
    assert lengths.sum() == N and (lengths >= 0).all()
    base = make_random(N, M, V, K, seed=len(layout), doc_order="sequential")
    doc = np.repeat(np.arange(M), lengths).astype(np.int32)
    c = _corpus(base.theta, base.phi, doc, base.word_id, base.u, f"skewed-{layout}")
    _offset_check(c, kernel, rate=False)
    if kernel == "docs":
        assert (run_kernel("docs", to_device(c)) == run_kernel("butterfly", to_device(c))).all()


@pytest.mark.parametrize("kernel", OFFSET_KERNELS)
def test_docs_empty_corpus_and_empty_documents(kernel):
    """N = 0 is a no-op; documents before, between and after the tokens
    may be empty."""
    import torch
    import paper_1505_03851_amd as lda
    fn = {"docs": lda.draw_docs, "doc_lanes": lda.draw_doc_lanes,
          "doc_lanes_cache": lambda *a, **k: lda.draw_doc_lanes(*a, theta_cache=True, **k)}[kernel]
    K, V = 48, 30
    rng = np.random.default_rng(5)
    theta = torch.from_numpy(rng.random((6, K), dtype=np.float32)).cuda()
    phi = torch.from_numpy(rng.random((V, K), dtype=np.float32)).cuda()
    off = torch.tensor([0, 0, 0, 0, 0, 0, 0], dtype=torch.int64, device="cuda")
    empty_i = torch.empty(0, dtype=torch.int32, device="cuda")
    empty_f = torch.empty(0, dtype=torch.float32, device="cuda")
    assert fn(theta, phi, off, empty_i, empty_f, validate=True).numel() == 0
    N = 100
    doc = np.repeat(np.arange(6), [0, 0, 37, 0, 63, 0]).astype(np.int32)
    word = rng.integers(0, V, N).astype(np.int32)
    u = _grid_u(N, 3)
    c = _corpus(theta.cpu().numpy(), phi.cpu().numpy(), doc, word, u, "empty-docs")
    _check(c, kernel, rate=False)


@pytest.mark.parametrize("kernel", OFFSET_KERNELS)
def test_docs_rejects_bad_offsets(kernel):
    import torch
    import paper_1505_03851_amd as lda
    fn = {"docs": lda.draw_docs, "doc_lanes": lda.draw_doc_lanes,
          "doc_lanes_cache": lambda *a, **k: lda.draw_doc_lanes(*a, theta_cache=True, **k)}[kernel]
    theta = torch.ones((3, 8), device="cuda")
    phi = torch.ones((4, 8), device="cuda")
    w = torch.zeros(5, dtype=torch.int32, device="cuda")
    u = torch.zeros(5, device="cuda")
    for bad in ([0, 2, 1, 5], [1, 2, 3, 5], [0, 1, 2, 4]):
        off = torch.tensor(bad, dtype=torch.int64, device="cuda")
        with pytest.raises(ValueError):
            fn(theta, phi, off, w, u, validate=True)
    with pytest.raises(ValueError):   # M + 1 entries
        fn(theta, phi, torch.zeros(3, dtype=torch.int64, device="cuda"), w, u)


@pytest.mark.parametrize("kernel", OFFSET_KERNELS)
@pytest.mark.parametrize("K", [8, 64, 256, 1024])
def test_docs_equal_power_of_two_weights_exact(K, kernel):
    """Equal weights 2**-3 in ragged documents: z = floor(u*K) exactly."""
    N = 64 * 37 + 11
    u = _grid_u(N, K + 7)
    doc = make_random(N, 97, 5, 1, seed=K, doc_order="ragged").doc_id
    c = _corpus(np.full((97, K), 2.0 ** -3), np.ones((5, K)), doc,
                np.arange(N) % 5, u, f"pow2-ragged-K{K}")
    print(f"[case] {c.name} kernel={kernel}", flush=True)
    if kernel == "doc_lanes_cache" and K > 256:
        return
    z = run_kernel(kernel, to_device(c))
    expect = np.floor(u.astype(np.float64) * K).astype(np.int32)
    assert (z == expect).all(), np.nonzero(z != expect)[0][:10]


@pytest.mark.parametrize("K", [32, 50, 64, 83, 200, 1024])
def test_butterfly_table_matches_closed_form(K):
    """The tables the kernel builds (Fig. 1, right) equal the oracle's closed
    form evaluated on exact products, within fp32 rounding."""
    import torch
    import paper_1505_03851_amd as lda
    from oracle import butterfly as bf
    N = 64 * 5 + 23
    c = make_random(N, 9, 120, K, seed=K, doc_order="shuffled")
    dev = to_device(c)
    print(f"[case] table K={K} N={N}", flush=True)
    tab = lda.butterfly_table(dev["theta"], dev["phi"], dev["doc_id"],
                              dev["word_id"])
    torch.cuda.synchronize()
    tab = tab.cpu().numpy().astype(np.float64)
    W = lda.butterfly_width(K)
    for g0 in range(0, N, W):
        toks = np.minimum(np.arange(g0, g0 + W), N - 1)
        a = (c.theta[c.doc_id[toks]].astype(np.float64) *
             c.phi[c.word_id[toks]].astype(np.float64))
        ref = bf.table_fp64(a, W)
        valid = np.arange(g0, g0 + W) < N
        got = tab[toks[valid]]
        exp = ref[valid]
        err = np.abs(got - exp)
        tol = 2e-5 * np.abs(exp) + 1e-37
        assert (err <= tol).all(), (g0, np.argwhere(err > tol)[:5])


# One fixed distribution drawn 10^6 times on the GPU (K = 8, one topic of zero
# weight): the counts fit the normalised weights, the empty topic is never
# drawn, and with the uniforms of the oracle's own chi-square pin every draw
# agrees with the oracle under the band rule.
CHI_WEIGHTS = np.array([0.05, 0.2, 0.0, 0.1, 0.3, 0.15, 0.12, 0.08], np.float32)


def _chi_square_pvalue(z):
    from scipy import stats
    counts = np.bincount(z, minlength=CHI_WEIGHTS.size)
    assert counts[2] == 0, counts
    nz = CHI_WEIGHTS > 0
    p = CHI_WEIGHTS[nz].astype(np.float64) / CHI_WEIGHTS.astype(np.float64).sum()
    return stats.chisquare(counts[nz], z.size * p).pvalue


@pytest.mark.parametrize("kernel", KERNELS)
def test_chi_square_of_gpu_draws(kernel):
    N = 1_000_000
    c = _corpus(CHI_WEIGHTS[None, :], np.ones((1, CHI_WEIGHTS.size)), np.zeros(N),
                np.zeros(N), _grid_u(N, 20150513), "chi-square-K8")
    rep = _check(c, kernel)
    z = run_kernel(kernel, to_device(c))
    assert _chi_square_pvalue(z) >= 1e-3, rep


def test_chi_square_of_gpu_draws_with_philox_uniforms():
    """The same distribution with the uniforms generated in the kernel."""
    import torch
    import paper_1505_03851_amd as lda
    N = 1_000_000
    th = torch.from_numpy(CHI_WEIGHTS[None, :].copy()).cuda()
    ph = torch.ones((1, CHI_WEIGHTS.size), dtype=torch.float32, device="cuda")
    zeros = torch.zeros(N, dtype=torch.int32, device="cuda")
    print("[case] chi-square-K8 philox", flush=True)
    for sweep in (0, 1):
        z = lda.draw_philox(th, ph, zeros, zeros, seed=0x5EED, sweep=sweep)
        torch.cuda.synchronize()
        assert _chi_square_pvalue(z.cpu().numpy()) >= 1e-4, sweep
