"""GPU tests of the topic counts (lda_count_topics) through the C ABI.

The counts are integer work, so the bar is bit-exact: for the same doc ids,
word ids and topics, the GPU's ndk and nwk equal the oracle's counts cell for
cell.  On the five workloads the topics are the GPU draw's own z (the path a
sampler runs: draw, then count, on one stream)."""
import numpy as np
import pytest

import oracle
from paper_1505_03851_amd.inputs import make_random
from parity import named_corpus, to_device

pytestmark = pytest.mark.gpu


def _gpu_counts(d, w, z, M, V, K, ndk=None, nwk=None):
    import torch
    import paper_1505_03851_amd as lda
    dev = [torch.from_numpy(np.ascontiguousarray(a, np.int32)).cuda() for a in (d, w, z)]
    a, b = lda.count_topics(*dev, M, V, K, ndk=ndk, nwk=nwk)
    torch.cuda.synchronize()
    return a.cpu().numpy(), b.cpu().numpy()


def _same(got, want, what):
    assert got.shape == want.shape, what
    bad = np.argwhere(got != want)
    assert bad.size == 0, f"{what}: {len(bad)} cells differ, first {bad[:5].tolist()}"


@pytest.mark.parametrize("name", ["tiny-K32", "corpus1M-K64", "corpus1M-K256",
                                  "corpus16M-K1024", "poisson300-K2048"])
def test_counts_of_the_draw_every_config(name):
    """Draw with lda_draw_butterfly, then count on the same stream; the counts
    equal the oracle's counts of that z, every cell."""
    import torch
    import paper_1505_03851_amd as lda
    c = named_corpus(name)
    dev = to_device(c)
    print(f"[case] counts {name} N={c.N} M={c.M} V={c.V} K={c.K}", flush=True)
    z = lda.draw_butterfly(dev["theta"], dev["phi"], dev["doc_id"], dev["word_id"], dev["u"])
    ndk, nwk = lda.count_topics(dev["doc_id"], dev["word_id"], z, c.M, c.V, c.K)
    torch.cuda.synchronize()
    z = z.cpu().numpy()
    want = oracle.counts(c.doc_id, c.word_id, z, c.M, c.V, c.K)
    _same(ndk.cpu().numpy(), want[0], "ndk")
    _same(nwk.cpu().numpy(), want[1], "nwk")
    print(f"[counts] {name}: ndk and nwk equal the oracle's ({c.M}x{c.K} and {c.V}x{c.K} cells)",
          flush=True)


SHAPES = [
    # (N, M, V, K, doc order)
    (1, 1, 1, 1, "sequential"),
    (7, 3, 5, 2, "shuffled"),
    (2047, 20, 300, 33, "sequential"),
    (2048, 20, 300, 64, "shuffled"),
    (2049, 20, 300, 64, "ragged"),
    (64 * 1000 + 13, 500, 4000, 1000, "shuffled"),
    (300_001, 3000, 20_000, 4096, "sequential"),
    (100_000, 1, 7, 16, "single"),
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "N{}-M{}-V{}-K{}-{}".format(*s))
def test_counts_random_topics(shape):
    N, M, V, K, order = shape
    c = make_random(N, M, V, 1, seed=N + K, doc_order=order)
    z = np.random.default_rng(K).integers(0, K, N).astype(np.int32)
    print(f"[case] counts random {shape}", flush=True)
    got = _gpu_counts(c.doc_id, c.word_id, z, M, V, K)
    want = oracle.counts(c.doc_id, c.word_id, z, M, V, K)
    _same(got[0], want[0], "ndk")
    _same(got[1], want[1], "nwk")


def test_counts_one_hot_cell():
    """Every token of one word in one document on one topic: one cell
    receives all N tokens (the case aggregation exists for)."""
    N, M, V, K = 1_000_003, 4, 9, 300
    d = np.full(N, 2, np.int32)
    w = np.full(N, 5, np.int32)
    z = np.full(N, 123, np.int32)
    ndk, nwk = _gpu_counts(d, w, z, M, V, K)
    assert ndk[2, 123] == N and nwk[5, 123] == N
    assert ndk.sum() == N and nwk.sum() == N


def test_counts_out_of_range_tokens_not_counted():
    N, M, V, K = 5000, 13, 70, 40
    rng = np.random.default_rng(4)
    d = rng.integers(0, M, N).astype(np.int32)
    w = rng.integers(0, V, N).astype(np.int32)
    z = rng.integers(0, K, N).astype(np.int32)
    d[::97] = -1
    d[5::89] = M
    w[7::83] = V
    w[9::79] = -(2 ** 31)
    z[11::71] = K
    z[13::67] = -1
    got = _gpu_counts(d, w, z, M, V, K)
    want = oracle.counts(d, w, z, M, V, K)
    _same(got[0], want[0], "ndk")
    _same(got[1], want[1], "nwk")
    assert want[0].sum() < N


def test_counts_overwrite_and_unaligned_tables():
    """Outputs holding garbage are overwritten (not added to); tables that
    start 4 bytes past a 16-byte boundary are cleared and filled whole; the
    ints around them are untouched; N = 0 clears."""
    import torch
    import paper_1505_03851_amd as lda
    N, M, V, K = 70_000, 37, 501, 45
    c = make_random(N, M, V, 1, seed=9, doc_order="ragged")
    z = np.random.default_rng(2).integers(0, K, N).astype(np.int32)
    big_d = torch.full((M * K + 2,), 777, dtype=torch.int32, device="cuda")
    big_w = torch.full((V * K + 2,), -5, dtype=torch.int32, device="cuda")
    ndk = big_d[1:1 + M * K].view(M, K)
    nwk = big_w[1:1 + V * K].view(V, K)
    got = _gpu_counts(c.doc_id, c.word_id, z, M, V, K, ndk=ndk, nwk=nwk)
    want = oracle.counts(c.doc_id, c.word_id, z, M, V, K)
    _same(got[0], want[0], "ndk")
    _same(got[1], want[1], "nwk")
    assert int(big_d[0]) == 777 and int(big_d[-1]) == 777
    assert int(big_w[0]) == -5 and int(big_w[-1]) == -5
    e = torch.empty(0, dtype=torch.int32, device="cuda")
    lda.count_topics(e, e, e, M, V, K, ndk=ndk, nwk=nwk)
    torch.cuda.synchronize()
    assert int(ndk.abs().sum()) == 0 and int(nwk.abs().sum()) == 0
    assert int(big_d[0]) == 777 and int(big_w[-1]) == -5


def test_counts_captured_in_a_graph():
    """Draw and count captured in one HIP graph and replayed with new
    uniforms (eager work between the replays); every replay's counts equal
    the oracle's counts of that replay's z."""
    import torch
    import paper_1505_03851_amd as lda
    c = make_random(64 * 300 + 17, 200, 3000, 200, seed=5, doc_order="ragged")
    dev = to_device(c)
    z = torch.empty(c.N, dtype=torch.int32, device="cuda")
    ndk = torch.empty((c.M, c.K), dtype=torch.int32, device="cuda")
    nwk = torch.empty((c.V, c.K), dtype=torch.int32, device="cuda")

    def step():
        lda.draw_butterfly(dev["theta"], dev["phi"], dev["doc_id"], dev["word_id"], dev["u"],
                           out=z)
        lda.count_topics(dev["doc_id"], dev["word_id"], z, c.M, c.V, c.K, ndk=ndk, nwk=nwk)

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    rng = np.random.default_rng(3)
    for rep in range(3):
        new_u = (rng.integers(0, 1 << 24, c.N) * 2.0 ** -24).astype(np.float32)
        dev["u"].copy_(torch.from_numpy(new_u))
        g.replay()
        torch.cuda.synchronize()
        zz = z.cpu().numpy()
        want = oracle.counts(c.doc_id, c.word_id, zz, c.M, c.V, c.K)
        _same(ndk.cpu().numpy(), want[0], f"ndk replay {rep}")
        _same(nwk.cpu().numpy(), want[1], f"nwk replay {rep}")
        ndk.fill_(3)                 # eager work between the replays
        nwk.fill_(-1)


# ---------------------------------------------------------------------------
# Documents as offsets (lda_count_topics_docs): each document's row written
# whole by one wavefront.

def _offsets(doc_id, M):
    from paper_1505_03851_amd.inputs import doc_offsets
    return doc_offsets(doc_id, M)


def _gpu_counts_docs(off, w, z, V, K, ndk=None, nwk=None):
    import torch
    import paper_1505_03851_amd as lda
    o = torch.from_numpy(np.ascontiguousarray(off, np.int64)).cuda()
    wd = torch.from_numpy(np.ascontiguousarray(w, np.int32)).cuda()
    zd = torch.from_numpy(np.ascontiguousarray(z, np.int32)).cuda()
    a, b = lda.count_topics_docs(o, wd, zd, V, K, ndk=ndk, nwk=nwk, validate=True)
    torch.cuda.synchronize()
    return a.cpu().numpy(), b.cpu().numpy()


@pytest.mark.parametrize("name", ["tiny-K32", "corpus1M-K64", "corpus1M-K256",
                                  "corpus16M-K1024", "poisson300-K2048"])
def test_counts_docs_of_the_draw_every_config(name):
    import torch
    import paper_1505_03851_amd as lda
    c = named_corpus(name)
    dev = to_device(c)
    print(f"[case] counts (offsets) {name}", flush=True)
    z = lda.draw_butterfly(dev["theta"], dev["phi"], dev["doc_id"], dev["word_id"], dev["u"])
    torch.cuda.synchronize()
    z = z.cpu().numpy()
    got = _gpu_counts_docs(_offsets(c.doc_id, c.M), c.word_id, z, c.V, c.K)
    want = oracle.counts(c.doc_id, c.word_id, z, c.M, c.V, c.K)
    _same(got[0], want[0], "ndk")
    _same(got[1], want[1], "nwk")


@pytest.mark.parametrize("shape", [(1, 1, 1, 1), (7, 30, 5, 3), (2049, 20, 300, 64),
                                   (64 * 1000 + 13, 5000, 4000, 1000),
                                   (100_000, 3, 7, 4096), (70_001, 1, 500, 200)],
                         ids=lambda s: "N{}-M{}-V{}-K{}".format(*s))
def test_counts_docs_ragged(shape):
    """Ragged documents, many of them empty (and M above N), random topics;
    a few words and topics out of range."""
    N, M, V, K = shape
    c = make_random(N, M, V, 1, seed=N + M, doc_order="ragged")
    rng = np.random.default_rng(K)
    z = rng.integers(0, K, N).astype(np.int32)
    w = c.word_id.copy()
    if N > 100:
        z[::53] = K
        w[7::61] = -1
    print(f"[case] counts (offsets) ragged {shape}", flush=True)
    got = _gpu_counts_docs(_offsets(c.doc_id, M), w, z, V, K)
    want = oracle.counts(c.doc_id, w, z, M, V, K)
    _same(got[0], want[0], "ndk")
    _same(got[1], want[1], "nwk")


def test_counts_docs_overwrite_and_equal_to_doc_id_form():
    """Outputs holding garbage are overwritten; the offsets form equals the
    doc-id form cell for cell; N = 0 writes zero rows."""
    import torch
    import paper_1505_03851_amd as lda
    N, M, V, K = 90_000, 301, 777, 45
    c = make_random(N, M, V, 1, seed=3, doc_order="ragged")
    z = np.random.default_rng(1).integers(0, K, N).astype(np.int32)
    ndk = torch.full((M, K), 9, dtype=torch.int32, device="cuda")
    nwk = torch.full((V, K), -9, dtype=torch.int32, device="cuda")
    got = _gpu_counts_docs(_offsets(c.doc_id, M), c.word_id, z, V, K, ndk=ndk, nwk=nwk)
    ref = _gpu_counts(c.doc_id, c.word_id, z, M, V, K)
    _same(got[0], ref[0], "ndk")
    _same(got[1], ref[1], "nwk")
    off0 = torch.zeros(M + 1, dtype=torch.int64, device="cuda")
    e = torch.empty(0, dtype=torch.int32, device="cuda")
    lda.count_topics_docs(off0, e, e, V, K, ndk=ndk, nwk=nwk)
    torch.cuda.synchronize()
    assert int(ndk.abs().sum()) == 0 and int(nwk.abs().sum()) == 0


# ---------------------------------------------------------------------------
# The word index (lda_word_index_build) and the counts taken from it
# (lda_count_topics_indexed).  The index is checked against its definition:
# off = the exclusive prefix sum of the in-range words' token counts, and
# positions off[w] .. off[w+1] - 1 hold exactly the tokens of word w (in any
# order); the counts against the oracle, cell for cell.

def _check_index(idx, w, V):
    import torch
    torch.cuda.synchronize()
    a = {k: v.cpu().numpy() for k, v in idx.arrays().items()}
    valid = (w >= 0) & (w < V)
    hist = np.bincount(w[valid], minlength=V)
    want_off = np.concatenate([[0], np.cumsum(hist)]).astype(np.int64)
    assert np.array_equal(a["off"].astype(np.int64), want_off)
    n = int(want_off[-1])
    perm, ws = a["perm"][:n], a["wsorted"][:n]
    assert np.array_equal(np.sort(perm), np.nonzero(valid)[0])   # each in-range token once
    assert np.array_equal(w[perm], ws)                            # its own word
    assert np.all(np.diff(ws) >= 0)                               # grouped by word
    return a


def _gpu_counts_indexed(off, w, z, V, K, idx=None, ndk=None, nwk=None):
    import torch
    import paper_1505_03851_amd as lda
    o = torch.from_numpy(np.ascontiguousarray(off, np.int64)).cuda()
    wd = torch.from_numpy(np.ascontiguousarray(w, np.int32)).cuda()
    zd = torch.from_numpy(np.ascontiguousarray(z, np.int32)).cuda()
    if idx is None:
        idx = lda.word_index_build(wd, V)
    a, b = lda.count_topics_indexed(o, wd, zd, idx, K, ndk=ndk, nwk=nwk)
    torch.cuda.synchronize()
    return a.cpu().numpy(), b.cpu().numpy(), idx


@pytest.mark.parametrize("name", ["tiny-K32", "corpus1M-K64", "corpus1M-K256",
                                  "corpus16M-K1024", "poisson300-K2048"])
def test_counts_indexed_of_the_draw_every_config(name):
    """Index once, draw, count from the index: every cell equals the oracle's,
    and the index is the counting sort of the words."""
    import torch
    import paper_1505_03851_amd as lda
    c = named_corpus(name)
    dev = to_device(c)
    print(f"[case] counts indexed {name} N={c.N} M={c.M} V={c.V} K={c.K}", flush=True)
    idx = lda.word_index_build(dev["word_id"], c.V)
    _check_index(idx, c.word_id, c.V)
    off = torch.from_numpy(_offsets(c.doc_id, c.M)).cuda()
    z = lda.draw_butterfly(dev["theta"], dev["phi"], dev["doc_id"], dev["word_id"], dev["u"])
    ndk, nwk = lda.count_topics_indexed(off, dev["word_id"], z, idx, c.K)
    torch.cuda.synchronize()
    want = oracle.counts(c.doc_id, c.word_id, z.cpu().numpy(), c.M, c.V, c.K)
    _same(ndk.cpu().numpy(), want[0], "ndk")
    _same(nwk.cpu().numpy(), want[1], "nwk")
    print(f"[counts] indexed {name}: ndk and nwk equal the oracle's", flush=True)


@pytest.mark.parametrize("shape", [(1, 1, 1, 1), (7, 30, 5, 3), (2047, 20, 300, 33),
                                   (2048, 20, 300, 64), (2049, 20, 300, 64),
                                   (64013, 5000, 4000, 1000), (100_000, 3, 7, 4096),
                                   (300_001, 3000, 20_000, 200), (70_001, 1, 500, 200)],
                         ids=lambda s: "N{}-M{}-V{}-K{}".format(*s))
def test_counts_indexed_random(shape):
    """Random topics over Zipf words (a few words span many segments, many
    words a single one), ragged documents; also the index of V = 7 words for
    100,000 tokens (every word spans many segments)."""
    N, M, V, K = shape
    c = make_random(N, M, V, 1, seed=N + 3 * K, doc_order="ragged")
    z = np.random.default_rng(K + 1).integers(0, K, N).astype(np.int32)
    print(f"[case] counts indexed random {shape}", flush=True)
    off = _offsets(c.doc_id, M)
    got_d, got_w, idx = _gpu_counts_indexed(off, c.word_id, z, V, K)
    _check_index(idx, c.word_id, V)
    want = oracle.counts(c.doc_id, c.word_id, z, M, V, K)
    _same(got_d, want[0], "ndk")
    _same(got_w, want[1], "nwk")


def test_counts_indexed_out_of_range_and_reuse():
    """Words and topics out of range are neither indexed nor counted; one
    index serves several sweeps (new topics each time, outputs with garbage
    overwritten); empty words have zero rows."""
    import torch
    N, M, V, K = 50_000, 40, 3000, 70
    rng = np.random.default_rng(8)
    w = np.minimum(rng.zipf(1.3, N) - 1, V + 50).astype(np.int32)   # some past V
    w[3::101] = -7
    doc = np.sort(rng.integers(0, M, N)).astype(np.int32)
    off = _offsets(doc, M)
    idx = None
    ndk = torch.full((M, K), 9, dtype=torch.int32, device="cuda")
    nwk = torch.full((V, K), -4, dtype=torch.int32, device="cuda")
    for sweep in range(3):
        z = rng.integers(0, K, N).astype(np.int32)
        z[sweep::53] = K + sweep
        got_d, got_w, idx = _gpu_counts_indexed(off, w, z, V, K, idx=idx, ndk=ndk, nwk=nwk)
        want = oracle.counts(doc, w, z, M, V, K)
        _same(got_d, want[0], f"ndk sweep {sweep}")
        _same(got_w, want[1], f"nwk sweep {sweep}")
        ndk.fill_(9)
        nwk.fill_(-4)
    a = _check_index(idx, w, V)
    assert int(a["off"][-1]) < N                   # out-of-range words left out
    assert (np.bincount(w[(w >= 0) & (w < V)], minlength=V) == 0).any()


def test_word_index_captured_in_a_graph():
    """Build the index, draw and count from it, all captured in one HIP graph
    and replayed (eager work between the replays, the index workspace
    scribbled over): every replay's index and counts are right."""
    import torch
    import paper_1505_03851_amd as lda
    c = make_random(64 * 400 + 9, 300, 5000, 96, seed=12, doc_order="ragged")
    dev = to_device(c)
    off = torch.from_numpy(_offsets(c.doc_id, c.M)).cuda()
    z = torch.empty(c.N, dtype=torch.int32, device="cuda")
    ndk = torch.empty((c.M, c.K), dtype=torch.int32, device="cuda")
    nwk = torch.empty((c.V, c.K), dtype=torch.int32, device="cuda")
    ws = torch.empty(lda.word_index_bytes(c.N, c.V), dtype=torch.uint8, device="cuda")
    holder = {}

    def step():
        holder["idx"] = lda.word_index_build(dev["word_id"], c.V, workspace=ws)
        lda.draw_butterfly(dev["theta"], dev["phi"], dev["doc_id"], dev["word_id"], dev["u"],
                           out=z)
        lda.count_topics_indexed(off, dev["word_id"], z, holder["idx"], c.K, ndk=ndk, nwk=nwk)

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    rng = np.random.default_rng(13)
    for rep in range(3):
        new_u = (rng.integers(0, 1 << 24, c.N) * 2.0 ** -24).astype(np.float32)
        dev["u"].copy_(torch.from_numpy(new_u))
        g.replay()
        torch.cuda.synchronize()
        _check_index(holder["idx"], c.word_id, c.V)
        want = oracle.counts(c.doc_id, c.word_id, z.cpu().numpy(), c.M, c.V, c.K)
        _same(ndk.cpu().numpy(), want[0], f"ndk replay {rep}")
        _same(nwk.cpu().numpy(), want[1], f"nwk replay {rep}")
        ws.fill_(255)                # eager work between the replays
        ndk.fill_(3)
