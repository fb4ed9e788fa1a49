"""Sizes past 2**31: token counts (every kernel indexes tokens with 64-bit
integers) and tables (byte offsets into theta and phi are unsigned 32-bit,
so tables up to 4 GiB are addressed; past 4 GiB the draws take the wide
build, which addresses rows by index and forms 64-bit addresses, for tables
of any size; count-table cells are keyed by 32-bit indices, except the rows
of ndk in the offsets and indexed forms, written at 64-bit addresses).

The large-N inputs are made on the GPU (about 35 GB of token arrays); a
sample of the tokens -- random ones, the first and last, and those around
token 2**31 -- is checked against the oracle under the rounding-band rule.
The large tables are checked on every token.
"""
import numpy as np
import pytest

from parity import BAND_REL, MAX_MISMATCH_RATE, admissible
from paper_1505_03851_amd.inputs import dirichlet_columns, dirichlet_rows

pytestmark = pytest.mark.gpu

N_BIG = (1 << 31) + 4099          # past the signed 32-bit range, ragged tail
N_MAX = (1 << 32) - (1 << 16)     # LDA_MAX_N: a dispatch's work-items fill 32 bits
M_BIG = 32771                     # documents of about 65,500 tokens (131,000 at N_MAX)
V_BIG = 5000


def _sample(N):
    rng = np.random.default_rng(31)
    parts = [rng.choice(N, size=1 << 17, replace=False), np.arange(4096),
             np.arange(N - 4096, N), np.arange((1 << 31) - 2048, (1 << 31) + 2048)]
    return np.unique(np.concatenate(parts))


@pytest.fixture(scope="module", params=[N_BIG, N_MAX], ids=["N2^31+4099", "N_MAX"])
def big(request):
    import torch
    torch.cuda.empty_cache()
    g = torch.Generator(device="cuda")
    g.manual_seed(2015)
    N = request.param
    doc = torch.empty(N, dtype=torch.int32, device="cuda")
    chunk = 1 << 27
    for a in range(0, N, chunk):
        b = min(N, a + chunk)
        t = torch.arange(a, b, dtype=torch.int64, device="cuda")
        doc[a:b] = (t * M_BIG // N).to(torch.int32)
    word = torch.randint(0, V_BIG, (N,), dtype=torch.int32, device="cuda", generator=g)
    u = (torch.randint(0, 1 << 24, (N,), dtype=torch.int32, device="cuda", generator=g)
         .to(torch.float32) * (2.0 ** -24))
    z = torch.empty(N, dtype=torch.int32, device="cuda")
    idx = _sample(N)
    it = torch.from_numpy(idx).cuda()
    host = {"doc": doc[it].cpu().numpy(), "word": word[it].cpu().numpy(),
            "u": u[it].cpu().numpy()}
    print(f"[case] large N={N} M={M_BIG} V={V_BIG} sample={idx.size}", flush=True)
    yield {"doc": doc, "word": word, "u": u, "z": z, "idx": idx, "it": it, "host": host}
    del doc, word, u, z
    torch.cuda.empty_cache()


@pytest.mark.parametrize("kernel,K", [("butterfly", 64),    # leaf groups
                                      ("butterfly", 512),   # leaf eighths
                                      ("butterfly", 50),    # one topic per lane
                                      ("naive", 64)])
def test_tokens_past_2_31(big, kernel, K):
    import torch
    import oracle
    import paper_1505_03851_amd as lda
    ss = np.random.SeedSequence([2015, K])
    s_theta, s_phi = ss.spawn(2)
    theta = dirichlet_rows(s_theta, 0.1, M_BIG, K)
    phi = dirichlet_columns(s_phi, 0.01, V_BIG, K)
    th = torch.from_numpy(theta).cuda()
    ph = torch.from_numpy(phi).cuda()
    print(f"[case] large kernel={kernel} K={K}", flush=True)
    fn = lda.draw_butterfly if kernel == "butterfly" else lda.draw_naive
    fn(th, ph, big["doc"], big["word"], big["u"], out=big["z"])
    torch.cuda.synchronize()
    z = big["z"][big["it"]].cpu().numpy()
    h = big["host"]
    z_ref, band = oracle.draw(theta, phi, h["doc"], h["word"], h["u"], band_rel=BAND_REL)
    mis = z != z_ref
    bad = mis & ~band
    soft = np.nonzero(mis & band)[0]          # in the band: the topic must be admitted
    if soft.size:
        bad[soft] = ~admissible(theta, phi, h["doc"][soft], h["word"][soft], h["u"][soft],
                                z[soft])
    hard = int(bad.sum())
    print(f"[parity] large-N{big['doc'].numel()}-K{K} {kernel}: n={z.size} mismatches={int(mis.sum())} "
          f"hard={hard} in_band={int(band.sum())}", flush=True)
    assert hard == 0, big["idx"][np.nonzero(bad)[0][:5]]
    assert mis.mean() < MAX_MISMATCH_RATE


# ---------------------------------------------------------------------------
# Tables past 2 GiB: phi of about 2.3 GiB, so that rows beyond the 2^31-byte
# offset are read (byte offsets are unsigned 32-bit); most tokens take words
# from those rows.  Every token is checked against the oracle.

def _big_phi_case(K, seed):
    V = int(2.3 * 2 ** 30) // (4 * K) + 1
    w_min = (1 << 31) // (4 * K) + 1           # first row past the 2 GiB offset
    assert w_min < V
    rng = np.random.default_rng(seed)
    phi = rng.random((V, K), dtype=np.float32)
    phi *= rng.random((V, K), dtype=np.float32) > 0.37   # exact zeros, as Dirichlet(0.01) gives
    M = 300
    theta = rng.random((M, K), dtype=np.float32) ** 8
    N = 64 * 3000 + 17
    word = np.where(rng.random(N) < 1 / 3, rng.integers(0, V, N),
                    rng.integers(w_min, V, N)).astype(np.int32)
    doc = (np.arange(N, dtype=np.int64) * M // N).astype(np.int32)
    u = (rng.integers(0, 1 << 24, N) * 2.0 ** -24).astype(np.float32)
    from paper_1505_03851_amd.inputs import Corpus
    return Corpus(theta, phi, doc, word, u, name=f"phi-past-2GiB-K{K}")


@pytest.mark.parametrize("K", [1024, 256, 96, 130])
def test_phi_past_2_gib(K):
    import torch
    from parity import compare, run_kernel, to_device
    c = _big_phi_case(K, seed=K)
    print(f"[case] {c.name} V={c.V} phi={4 * c.V * K / 2 ** 30:.2f} GiB N={c.N}", flush=True)
    torch.cuda.empty_cache()
    dev = to_device(c)
    kernels = ["butterfly", "naive", "transposed", "variant-register", "docs"] + \
              (["routed"] if K >= 768 and K % 4 == 0 else [])
    for kernel in kernels:
        z = run_kernel(kernel, dev)
        assert z.min() >= 0 and z.max() < K, kernel
        rep = compare(c, z)
        print(f"[parity] {c.name} {kernel}: {rep}", flush=True)
        assert rep.hard == 0, (kernel, rep.first_hard)
        assert rep.mismatch_rate < MAX_MISMATCH_RATE, (kernel, str(rep))
    del dev
    torch.cuda.empty_cache()


def test_word_counts_past_2_gib():
    """nwk of about 2.3 GiB (V x K int32): cells past the 2^31-byte offset are
    counted exactly."""
    import torch
    import oracle
    import paper_1505_03851_amd as lda
    K = 1024
    V = int(2.3 * 2 ** 30) // (4 * K) + 1
    w_min = (1 << 31) // (4 * K) + 1
    rng = np.random.default_rng(5)
    N, M = 500_000, 700
    word = np.where(rng.random(N) < 0.5, rng.integers(0, V, N), rng.integers(w_min, V, N))
    d = torch.from_numpy((np.arange(N) * M // N).astype(np.int32)).cuda()
    w = torch.from_numpy(word.astype(np.int32)).cuda()
    z = torch.from_numpy(rng.integers(0, K, N).astype(np.int32)).cuda()
    print(f"[case] counts nwk {4 * V * K / 2 ** 30:.2f} GiB", flush=True)
    torch.cuda.empty_cache()
    ndk, nwk = lda.count_topics(d, w, z, M, V, K)
    torch.cuda.synchronize()
    want_d, want_w = oracle.counts(d.cpu().numpy(), w.cpu().numpy(), z.cpu().numpy(), M, V, K)
    assert np.array_equal(ndk.cpu().numpy(), want_d)
    got_w = nwk.cpu().numpy()
    assert np.array_equal(got_w, want_w), np.argwhere(got_w != want_w)[:5]
    assert got_w[w_min:].sum() == (word >= w_min).sum()
    del ndk, nwk
    torch.cuda.empty_cache()


# ---------------------------------------------------------------------------
# Tables past 4 GiB: the wide build of the draw kernels.  phi (or theta) of
# about 4.3 GiB; most tokens take rows past the 2^32-byte offset, the rest
# rows anywhere; a few carry ids past the table (clamped to its last row by
# the wide build: such draws are not compared).  Every in-range token is
# checked against the oracle, for the doc-id form, the offsets form and the
# in-kernel uniforms.

WIDE_BYTES = int(4.3 * 2 ** 30)


def _wide_case(K, seed, big):
    """`big` = "phi" or "theta": the table past 4 GiB."""
    rng = np.random.default_rng(seed)
    rows = WIDE_BYTES // (4 * K) + 1
    r_min = (1 << 32) // (4 * K) + 1           # first row past the 4 GiB offset
    assert r_min < rows and 4 * rows * K > (1 << 32)
    N = 64 * 3000 + 17
    far = np.where(rng.random(N) < 1 / 3, rng.integers(0, rows, N),
                   rng.integers(r_min, rows, N)).astype(np.int32)
    if big == "phi":
        V, M = rows, 300
        word = far
        doc = (np.arange(N, dtype=np.int64) * M // N).astype(np.int32)
    else:
        V, M = 5000, rows
        word = rng.integers(0, V, N).astype(np.int32)
        doc = np.sort(far)                     # contiguous documents, most past 4 GiB
    phi = rng.random((V, K), dtype=np.float32)
    phi *= rng.random((V, K), dtype=np.float32) > 0.37   # exact zeros, as Dirichlet(0.01) gives
    theta = rng.random((M, K), dtype=np.float32) ** 8
    u = (rng.integers(0, 1 << 24, N) * 2.0 ** -24).astype(np.float32)
    from paper_1505_03851_amd.inputs import Corpus
    return Corpus(theta, phi, doc, word, u, name=f"{big}-past-4GiB-K{K}")


@pytest.mark.parametrize("big,K", [("phi", 1024), ("phi", 256), ("phi", 96), ("phi", 130),
                                   ("phi", 300), ("theta", 1024), ("theta", 20),
                                   ("theta", 436)])
def test_tables_past_4_gib(big, K):
    import torch
    import paper_1505_03851_amd as lda
    from oracle import philox as px
    from parity import compare, run_kernel, to_device
    c = _wide_case(K, seed=K + (7 if big == "theta" else 0), big=big)
    size = 4 * (c.V if big == "phi" else c.M) * K
    print(f"[case] {c.name} M={c.M} V={c.V} {big}={size / 2 ** 30:.2f} GiB N={c.N}", flush=True)
    assert size > lda.MAX_TABLE_BYTES
    torch.cuda.empty_cache()
    dev = to_device(c)
    for kernel in ("butterfly", "docs"):
        z = run_kernel(kernel, dev)
        assert z.min() >= 0 and z.max() < K, kernel
        rep = compare(c, z)
        print(f"[parity] {c.name} {kernel}: {rep}", flush=True)
        assert rep.hard == 0, (kernel, rep.first_hard)
        assert rep.mismatch_rate < MAX_MISMATCH_RATE, (kernel, str(rep))
    seed, sweep = 20150513, 3
    z = lda.draw_philox(dev["theta"], dev["phi"], dev["doc_id"], dev["word_id"], seed, sweep)
    torch.cuda.synchronize()
    c.u = px.token_uniforms(seed, sweep, 0, c.N)
    rep = compare(c, z.cpu().numpy())
    print(f"[parity] {c.name} philox: {rep}", flush=True)
    assert rep.hard == 0 and rep.mismatch_rate < MAX_MISMATCH_RATE
    # the narrow entry points refuse such tables
    with pytest.raises(lda.LdaError):
        lda.draw_naive(dev["theta"], dev["phi"], dev["doc_id"], dev["word_id"], dev["u"])
    del dev
    torch.cuda.empty_cache()


def test_wide_ids_past_the_table_stay_inside():
    """With tables past 4 GiB no buffer range check guards the reads: ids
    past the last row are clamped to it, so every read stays inside the
    table (the draws of such tokens are those of the last row)."""
    import torch
    import paper_1505_03851_amd as lda
    from parity import compare, to_device
    K = 256
    c = _wide_case(K, seed=11, big="phi")
    bad = np.arange(0, c.N, 97)
    word = c.word_id.copy()
    word[bad] = np.where(bad % 2 == 0, c.V + 5, -3)
    print(f"[case] wide ids past the table K={K} bad={bad.size}", flush=True)
    dev = to_device(c)
    dev["word_id"] = torch.from_numpy(word).cuda()
    z = lda.draw_butterfly(dev["theta"], dev["phi"], dev["doc_id"], dev["word_id"], dev["u"])
    torch.cuda.synchronize()
    z = z.cpu().numpy()
    assert z.min() >= 0 and z.max() < K
    c.word_id = np.where(np.isin(np.arange(c.N), bad), c.V - 1, c.word_id).astype(np.int32)
    rep = compare(c, z)
    print(f"[parity] wide clamped ids: {rep}", flush=True)
    assert rep.hard == 0 and rep.mismatch_rate < MAX_MISMATCH_RATE
    del dev
    torch.cuda.empty_cache()


def test_word_counts_past_4_gib():
    """nwk of about 4.3 GiB (V x K int32, more cells than a byte offset can
    reach): cells past the 2^32-byte offset are counted exactly, by every
    count entry point (document ids, offsets, the word index)."""
    import torch
    import oracle
    import paper_1505_03851_amd as lda
    from paper_1505_03851_amd.inputs import doc_offsets
    K = 1024
    V = WIDE_BYTES // (4 * K) + 1
    w_min = (1 << 32) // (4 * K) + 1
    rng = np.random.default_rng(6)
    N, M = 500_000, 700
    word = np.where(rng.random(N) < 0.5, rng.integers(0, V, N), rng.integers(w_min, V, N))
    doc = (np.arange(N) * M // N).astype(np.int32)
    d = torch.from_numpy(doc).cuda()
    w = torch.from_numpy(word.astype(np.int32)).cuda()
    z = torch.from_numpy(rng.integers(0, K, N).astype(np.int32)).cuda()
    print(f"[case] counts nwk {4 * V * K / 2 ** 30:.2f} GiB", flush=True)
    torch.cuda.empty_cache()
    want_d, want_w = oracle.counts(doc, word.astype(np.int32), z.cpu().numpy(), M, V, K)
    ndk, nwk = lda.count_topics(d, w, z, M, V, K)
    torch.cuda.synchronize()
    assert np.array_equal(ndk.cpu().numpy(), want_d)
    got_w = nwk.cpu().numpy()
    assert np.array_equal(got_w, want_w), np.argwhere(got_w != want_w)[:5]
    assert got_w[w_min:].sum() == (word >= w_min).sum()
    off = torch.from_numpy(doc_offsets(doc, M)).cuda()
    ndk2, nwk2 = lda.count_topics_docs(off, w, z, V, K, ndk=ndk, nwk=nwk)
    torch.cuda.synchronize()
    assert np.array_equal(ndk2.cpu().numpy(), want_d)
    assert np.array_equal(nwk2.cpu().numpy(), want_w)
    nwk2.fill_(-1)
    index = lda.word_index_build(w, V)
    ndk3, nwk3 = lda.count_topics_indexed(off, w, z, index, K, ndk=ndk2, nwk=nwk2)
    torch.cuda.synchronize()
    assert np.array_equal(ndk3.cpu().numpy(), want_d)
    got_w = nwk3.cpu().numpy()
    assert np.array_equal(got_w, want_w), np.argwhere(got_w != want_w)[:5]
    del ndk, nwk, ndk2, nwk2, ndk3, nwk3, got_w, index
    torch.cuda.empty_cache()


def test_counts_at_the_largest_n():
    """N = LDA_COUNT_MAX_N = 2^31 - 1 tokens, where the index's positions and
    offsets fill int32: the three count entry points agree cell for cell, and
    every table has the sums the tokens fix, computed by torch on the same
    arrays (rows of ndk: the document lengths; rows of nwk: the word
    frequencies; columns: the topic totals); the word index's offsets are the
    exclusive prefix sums of the word frequencies, its positions hold every
    token exactly once, and each position's word is that token's word, in
    non-decreasing order."""
    import torch
    import paper_1505_03851_amd as lda
    from paper_1505_03851_amd import _lib
    N = _lib._CONSTS["LDA_COUNT_MAX_N"]
    M, V, K = 1 << 20, 5000, 16
    step = 1 << 28
    print(f"[case] counts at N={N}", flush=True)
    g = torch.Generator(device="cuda")
    g.manual_seed(11)
    w = torch.randint(0, V, (N,), dtype=torch.int32, device="cuda", generator=g)
    z = torch.randint(0, K, (N,), dtype=torch.int32, device="cuda", generator=g)
    off = torch.arange(M + 1, dtype=torch.int64, device="cuda") * N // M
    lengths = off[1:] - off[:-1]
    d = torch.repeat_interleave(torch.arange(M, dtype=torch.int32, device="cuda"), lengths,
                                output_size=N)
    ndk1, nwk1 = lda.count_topics(d, w, z, M, V, K)
    torch.cuda.synchronize()
    del d
    ndk2, nwk2 = lda.count_topics_docs(off, w, z, V, K)
    index = lda.word_index_build(w, V)
    ndk3, nwk3 = lda.count_topics_indexed(off, w, z, index, K)
    torch.cuda.synchronize()
    assert torch.equal(ndk1, ndk2) and torch.equal(ndk1, ndk3)
    assert torch.equal(nwk1, nwk2) and torch.equal(nwk1, nwk3)

    def counts_of(x, n):
        c = torch.zeros(n, dtype=torch.int64, device="cuda")
        for s in range(0, N, step):
            c += torch.bincount(x[s:s + step].long(), minlength=n)
        return c
    freq, ztot = counts_of(w, V), counts_of(z, K)
    assert torch.equal(ndk1.sum(1, dtype=torch.int64), lengths)
    assert torch.equal(nwk1.sum(1, dtype=torch.int64), freq)
    assert torch.equal(ndk1.sum(0, dtype=torch.int64), ztot)
    assert torch.equal(nwk1.sum(0, dtype=torch.int64), ztot)

    a = index.arrays()
    assert torch.equal(a["off"][:V].long(), torch.cumsum(freq, 0) - freq)
    assert int(a["off"][V]) == N
    seen = torch.zeros(N, dtype=torch.bool, device="cuda")
    for s in range(0, N, step):
        p, ws = a["perm"][s:s + step].long(), a["wsorted"][s:s + step]
        assert torch.equal(w[p], ws)
        seen[p] = True
        assert bool((ws[1:] >= ws[:-1]).all())
        if s:
            assert int(a["wsorted"][s - 1]) <= int(ws[0])
    assert bool(seen.all())
    del w, z, index, seen
    torch.cuda.empty_cache()


@pytest.mark.parametrize("M,K", [((1 << 22) + 4096, 1024), ((1 << 27) + 5, 16)],
                         ids=["ndk-16GiB", "M2^27"])
def test_doc_counts_of_any_size(M, K):
    """ndk past 16 GiB (more cells than a 32-bit key holds) and M past 2^26
    documents (more work-items than one dispatch holds, at one wavefront a
    document): the offsets and indexed forms write every row of ndk (filled
    with -1 before) -- the rows with tokens equal the oracle's counts of those
    documents, every cell is non-negative and the cells sum to the tokens
    counted, so the other rows are zero -- and nwk equals the oracle's."""
    import torch
    import oracle
    import paper_1505_03851_amd as lda
    from paper_1505_03851_amd.inputs import doc_offsets
    V, N = 3000, 400_000
    rng = np.random.default_rng(8)
    # half the tokens in random documents, half in the last 5,000 (past 2^32
    # cells at K = 1024; the last workgroups' documents at M = 2^27 + 5)
    doc = np.sort(np.concatenate([rng.integers(0, M, N // 2),
                                  rng.integers(M - 5000, M, N - N // 2)])).astype(np.int32)
    word = rng.integers(0, V, N).astype(np.int32)
    zh = rng.integers(0, K, N).astype(np.int32)
    rows = np.unique(doc)
    want_d, want_w = oracle.counts(np.searchsorted(rows, doc).astype(np.int32), word, zh,
                                   rows.size, V, K)
    print(f"[case] doc counts M={M} K={K} ndk {4 * M * K / 2 ** 30:.2f} GiB", flush=True)
    torch.cuda.empty_cache()
    off = torch.from_numpy(doc_offsets(doc, M)).cuda()
    w = torch.from_numpy(word).cuda()
    z = torch.from_numpy(zh).cuda()
    at = torch.from_numpy(rows.astype(np.int64)).cuda()
    ndk = torch.full((M, K), -1, dtype=torch.int32, device="cuda")
    nwk = torch.full((V, K), -1, dtype=torch.int32, device="cuda")

    def check(form):
        torch.cuda.synchronize()
        got = ndk[at].cpu().numpy()
        assert np.array_equal(got, want_d), (form, np.argwhere(got != want_d)[:5])
        assert int(ndk.min()) >= 0, form
        assert int(ndk.sum()) == N, form
        assert np.array_equal(nwk.cpu().numpy(), want_w), form

    lda.count_topics_docs(off, w, z, V, K, ndk=ndk, nwk=nwk)
    check("offsets")
    ndk.fill_(-1)
    nwk.fill_(-1)
    index = lda.word_index_build(w, V)
    lda.count_topics_indexed(off, w, z, index, K, ndk=ndk, nwk=nwk)
    check("indexed")
    del ndk, nwk, off, w, z, at, index
    torch.cuda.empty_cache()


def test_routed_at_the_largest_n():
    """N = LDA_ROUTE_MAX_N = 2^31 - 513 tokens, where the routed positions
    (N plus up to 8 x 64 of padding) fill int32: the routing is a layout of
    every token exactly once, each list in token order and padded with -1,
    carrying each token's word and document; the routed draw agrees with the
    token-order draw except on a handful of tokens, and a sample of 2^20
    tokens (among them the last 4,096) agrees with the oracle under the band
    rule."""
    import torch
    import paper_1505_03851_amd as lda
    from paper_1505_03851_amd import _lib
    from paper_1505_03851_amd.inputs import Corpus
    from parity import compare
    N = _lib._CONSTS["LDA_ROUTE_MAX_N"]
    M, V, K = 1 << 16, 1000, 768
    step = 1 << 28
    print(f"[case] routed at N={N}", flush=True)
    g = torch.Generator(device="cuda")
    g.manual_seed(13)
    theta = torch.rand((M, K), generator=g, device="cuda") ** 8
    phi = torch.rand((V, K), generator=g, device="cuda")
    phi *= torch.rand((V, K), generator=g, device="cuda") > 0.37
    w = torch.randint(0, V, (N,), dtype=torch.int32, device="cuda", generator=g)
    u = torch.rand(N, generator=g, device="cuda")
    off = torch.arange(M + 1, dtype=torch.int64, device="cuda") * N // M
    d = torch.repeat_interleave(torch.arange(M, dtype=torch.int32, device="cuda"),
                                off[1:] - off[:-1], output_size=N)
    route = lda.route_build(d, w, M, V)
    torch.cuda.synchronize()
    assert route.N == N and sum(route.tokens) == N
    a = route.arrays()
    seen = torch.zeros(N, dtype=torch.bool, device="cuda")
    at = 0
    for x in range(8):
        t, s0, ln = route.tokens[x], route.start[x], route.length[x]
        assert s0 == at and ln == (t + 63) // 64 * 64
        at += ln
        assert bool((a["perm"][s0 + t:s0 + ln] == -1).all())
        for s in range(s0, s0 + t, step):
            e = min(s + step, s0 + t)
            p = a["perm"][s:e].long()
            assert bool((p >= 0).all()) and bool((p[1:] > p[:-1]).all())
            if s > s0:
                assert int(a["perm"][s - 1]) < int(p[0])
            assert torch.equal(a["rword"][s:e], w[p]) and torch.equal(a["rdoc"][s:e], d[p])
            seen[p] = True
    assert bool(seen.all())
    del seen, a
    z_r = lda.draw_routed(theta, phi, route, u)
    z_b = lda.draw_butterfly(theta, phi, d, w, u)
    torch.cuda.synchronize()
    differ = int((z_r != z_b).sum())
    print(f"[parity] routed at N={N}: {differ} tokens differ from the token-order draw",
          flush=True)
    assert differ <= N // 10000
    rng = np.random.default_rng(13)
    idx = np.unique(np.concatenate([rng.integers(0, N, 1 << 20), np.arange(N - 4096, N)]))
    it = torch.from_numpy(idx).cuda()
    c = Corpus(theta.cpu().numpy(), phi.cpu().numpy(), d[it].cpu().numpy(),
               w[it].cpu().numpy(), u[it].cpu().numpy(), name=f"routed-N{N}-sample")
    rep = compare(c, z_r[it].cpu().numpy())
    print(f"[parity] {c.name}: {rep}", flush=True)
    assert rep.hard == 0 and rep.mismatch_rate < MAX_MISMATCH_RATE
    del d, w, u, z_r, z_b, route
    torch.cuda.empty_cache()


# ---------------------------------------------------------------------------
# Tables at the top of the wide build's range: theta or phi of 2^32 - 1 floats
# or just under (16 GiB), generated on the GPU; most tokens take rows whose
# float offsets lie at or past 2^31 (the top half of the unsigned 32-bit
# offsets), the last 64 rows among them.  The oracle is given only the rows
# the tokens use.

def _top_rows_case(big, K, seed, unit=1, rows=None, past=1 << 31):
    """unit: 1 fills 2^32 - 1 floats (16 GiB), 4 fills 2^32 - 1 bytes (4 GiB);
    or `rows` rows.  Most tokens take rows whose offset in `unit`s is at or
    past `past`."""
    import torch
    rows = rows or (2 ** 32 - 1) // (K * unit)
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    table = torch.empty((rows, K), dtype=torch.float32, device="cuda")
    step = max(1, (1 << 28) // K)
    for r in range(0, rows, step):
        e = min(rows, r + step)
        blk = torch.rand((e - r, K), generator=g, device="cuda")
        if big == "phi":
            blk *= torch.rand((e - r, K), generator=g, device="cuda") > 0.37
        else:
            blk = blk ** 8
        table[r:e] = blk
        del blk
    rng = np.random.default_rng(seed)
    N = 64 * 1000 + 17
    r_min = past // (K * unit) + 1
    ids = np.where(rng.random(N) < 0.25, rng.integers(0, rows, N), rng.integers(r_min, rows, N))
    ids[:64] = rows - 1 - np.arange(64)
    uniq, remap = np.unique(ids, return_inverse=True)
    used = table[torch.from_numpy(uniq).cuda()].cpu().numpy()
    return table, ids.astype(np.int32), used, remap.astype(np.int32), N


@pytest.mark.parametrize("big,K,gib", [("phi", 1024, 16), ("phi", 96, 16), ("phi", 130, 16),
                                       ("theta", 20, 16), ("theta", 1024, 16),
                                       ("phi", 1024, 20), ("phi", 96, 20), ("theta", 1024, 20),
                                       ("theta", 20, 20)])
def test_tables_at_16_gib(big, K, gib):
    """gib = 16: tables of 2^32 - 1 floats or just under, most tokens on rows
    whose float offsets lie at or past 2^31; gib = 20: tables of 20 GiB, past
    the reach of 32-bit float offsets, most tokens on rows past 2^32 floats."""
    import torch
    import paper_1505_03851_amd as lda
    from paper_1505_03851_amd.inputs import Corpus, doc_offsets
    from parity import compare
    print(f"[case] {big} of {gib} GiB at K={K}", flush=True)
    if gib == 16:
        table, ids, used, remap, N = _top_rows_case(big, K, 1000 + K)
    else:
        table, ids, used, remap, N = _top_rows_case(big, K, 3000 + K,
                                                    rows=(gib << 30) // (4 * K), past=1 << 32)
    rng = np.random.default_rng(K)
    u = (rng.integers(0, 1 << 24, N) * 2.0 ** -24).astype(np.float32)
    if big == "phi":
        M = 300
        other = (rng.random((M, K), dtype=np.float32) ** 8)
        doc = (np.arange(N, dtype=np.int64) * M // N).astype(np.int32)
        th, ph, d_dev, w_dev = torch.from_numpy(other).cuda(), table, doc, ids
        c = Corpus(other, used, doc, remap, u, name=f"phi-{gib}GiB-K{K}")
    else:
        V = 5000
        other = rng.random((V, K), dtype=np.float32) * (rng.random((V, K)) > 0.37)
        other = other.astype(np.float32)
        word = rng.integers(0, V, N).astype(np.int32)
        order = np.argsort(ids, kind="stable")  # contiguous documents
        ids, remap, word, u = ids[order], remap[order], word[order], u[order]
        th, ph, d_dev, w_dev = table, torch.from_numpy(other).cuda(), ids, word
        c = Corpus(used, other, remap, word, u, name=f"theta-{gib}GiB-K{K}")
    dd, wd = torch.from_numpy(d_dev).cuda(), torch.from_numpy(w_dev).cuda()
    ud = torch.from_numpy(u).cuda()
    z = lda.draw_butterfly(th, ph, dd, wd, ud)
    torch.cuda.synchronize()
    rep = compare(c, z.cpu().numpy())
    print(f"[parity] {c.name}: {rep}", flush=True)
    assert rep.hard == 0 and rep.mismatch_rate < MAX_MISMATCH_RATE
    if big == "theta":
        off = torch.from_numpy(doc_offsets(d_dev, th.shape[0])).cuda()
        z2 = lda.draw_docs(th, ph, off, wd, ud)
        torch.cuda.synchronize()
        assert torch.equal(z, z2)
        del off, z2
    del table, th, ph, z
    torch.cuda.empty_cache()


@pytest.mark.parametrize("K", [1024, 256, 50])
def test_phi_at_4_gib(K):
    """phi of 2^32 - 1 bytes or just under, the most the buffer-resource build
    addresses (byte offsets up to 2^32 - 1), three quarters of the tokens on
    rows past the 2^31-byte offset and the last 64 rows among them: every
    kernel that stays on that build, against the oracle."""
    import torch
    import paper_1505_03851_amd as lda
    from paper_1505_03851_amd.inputs import Corpus
    from parity import compare, run_kernel
    print(f"[case] phi of 4 GiB at K={K}", flush=True)
    table, ids, used, remap, N = _top_rows_case("phi", K, 2000 + K, unit=4)
    assert table.numel() * 4 <= lda.MAX_TABLE_BYTES
    rng = np.random.default_rng(K)
    M = 300
    theta = rng.random((M, K), dtype=np.float32) ** 8
    doc = (np.arange(N, dtype=np.int64) * M // N).astype(np.int32)
    u = (rng.integers(0, 1 << 24, N) * 2.0 ** -24).astype(np.float32)
    c = Corpus(theta, used, doc, remap, u, name=f"phi-4GiB-K{K}")
    dev = {"theta": torch.from_numpy(theta).cuda(), "phi": table,
           "doc_id": torch.from_numpy(doc).cuda(), "word_id": torch.from_numpy(ids).cuda(),
           "u": torch.from_numpy(u).cuda()}
    kernels = ["butterfly", "docs", "transposed", "naive"] + (["routed"] if K >= 768 else [])
    for kernel in kernels:
        z = run_kernel(kernel, dev)
        rep = compare(c, z)
        print(f"[parity] {c.name} {kernel}: {rep}", flush=True)
        assert rep.hard == 0 and rep.mismatch_rate < MAX_MISMATCH_RATE, kernel
    del table, dev
    torch.cuda.empty_cache()
