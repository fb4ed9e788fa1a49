"""GPU tests of the routing of tokens to the XCDs (route_build) and of the
routed draw (draw_routed), through the C ABI.

The routing is checked against its definition: every token exactly once, in
its original order within its list; a word class never split across lists;
the lists' token counts equal those of the greedy assignment recomputed here
from the class counts; padding repeats a list's last token.  The routed draw
is checked against the oracle under the band rule, as every other kernel."""
import numpy as np
import pytest

from paper_1505_03851_amd.inputs import make_corpus, make_random
from parity import (MAX_MISMATCH_RATE, compare, named_corpus, reference, run_kernel,
                    to_device)

pytestmark = pytest.mark.gpu


def word_class(w):
    """The routing's word class: bits 16..23 of w * 2654435761 mod 2^32."""
    return ((w.astype(np.uint64) * np.uint64(2654435761)) % np.uint64(2 ** 32) >>
            np.uint64(16)).astype(np.int64) & 255


def greedy_lists(words):
    """Tokens per list of the assignment the routing defines: classes by
    decreasing token count (ties: lower class first), each to the list with
    the fewest tokens so far (ties: lower list)."""
    counts = np.bincount(word_class(words), minlength=256)
    order = sorted(range(256), key=lambda c: (-counts[c], c))
    load = [0] * 8
    for c in order:
        x = min(range(8), key=lambda y: (load[y], y))
        load[x] += int(counts[c])
    return load


def build(c, validate=True):
    import torch
    import paper_1505_03851_amd as lda
    dev = to_device(c)
    route = lda.route_build(dev["doc_id"], dev["word_id"], c.M, c.V, validate=validate)
    torch.cuda.synchronize()
    arr = {k: v.cpu().numpy() for k, v in route.arrays().items()}
    return route, arr


def check_route(c, route, arr):
    N = c.N
    assert route.N == N and sum(route.tokens) == N
    assert route.tokens == greedy_lists(c.word_id)
    start = 0
    seen = []
    classes = []
    for x in range(8):
        t, s0, ln = route.tokens[x], route.start[x], route.length[x]
        assert s0 == start and ln == (t + 63) // 64 * 64
        start += ln
        perm = arr["perm"][s0:s0 + ln]
        real = perm[:t]
        assert (real >= 0).all() and (perm[t:] == -1).all()
        assert (np.diff(real) > 0).all(), "list not in token order"
        assert (arr["rword"][s0:s0 + t] == c.word_id[real]).all()
        assert (arr["rdoc"][s0:s0 + t] == c.doc_id[real]).all()
        if t:
            assert (arr["rword"][s0 + t:s0 + ln] == c.word_id[real[-1]]).all()
            assert (arr["rdoc"][s0 + t:s0 + ln] == c.doc_id[real[-1]]).all()
        seen.append(real)
        classes.append(set(word_class(c.word_id[real]).tolist()))
    allp = np.sort(np.concatenate(seen))
    assert (allp == np.arange(N)).all(), "not a permutation of the tokens"
    for x in range(8):
        for y in range(x + 1, 8):
            assert not (classes[x] & classes[y]), "a word class split across lists"


SHAPES = [
    # (N, M, V, K, doc order); the routed draw takes K >= 768
    (1, 1, 7, 768, "sequential"),
    (5, 2, 9, 1000, "shuffled"),
    (63, 4, 50, 772, "sequential"),
    (64, 4, 50, 1024, "single"),
    (65, 5, 50, 1000, "ragged"),
    (64 * 37 + 11, 30, 700, 1024, "sequential"),
    (64 * 37 + 11, 30, 700, 2044, "shuffled"),
    (64 * 90 + 7, 40, 2000, 2048, "ragged"),
    (64 * 90 + 7, 400, 5000, 1604, "sequential"),
    (100_000, 900, 20_000, 768, "sequential"),
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "N{}-K{}-{}".format(s[0], s[3], s[4]))
def test_route_and_draw_random(shape):
    N, M, V, K, order = shape
    c = make_random(N, M, V, K, seed=31, doc_order=order)
    print(f"[case] route {c.name}", flush=True)
    route, arr = build(c)
    check_route(c, route, arr)
    z = run_kernel("routed", to_device(c))
    assert z.min() >= 0 and z.max() < K
    rep = compare(c, z)
    print(f"[parity] {c.name} routed: {rep}", flush=True)
    assert rep.hard == 0, rep.first_hard


@pytest.mark.parametrize("name", ["corpus1M-K256", "wiki-shaped-K240", "corpus16M-K1024",
                                  "poisson300-K2048"])
def test_routed_config_every_token(name):
    """The routing of each workload is checked against its definition; the
    routed draw, on the workloads whose K it takes (K >= 768), is checked on
    every token against the oracle, and refused below."""
    import paper_1505_03851_amd as lda
    c = named_corpus(name)
    print(f"[case] routed {name}", flush=True)
    route, arr = build(c)
    check_route(c, route, arr)
    tok = route.tokens
    assert max(tok) * 8 / sum(tok) < 1.05, tok      # Zipf words: balanced lists
    if c.K < 768:
        with pytest.raises(lda.LdaError) as e:
            run_kernel("routed", to_device(c))
        assert e.value.status == lda.STATUS["LDA_ERR_UNSUPPORTED"]
        return
    z = run_kernel("routed", to_device(c))
    assert z.min() >= 0 and z.max() < c.K
    rep = compare(c, z, ref=reference(name))
    print(f"[parity] {name} routed: {rep}", flush=True)
    assert rep.hard == 0, rep.first_hard
    assert rep.mismatch_rate < MAX_MISMATCH_RATE


def test_route_reused_across_sweeps():
    """One routing, three draws with other uniforms and into a reused output."""
    import torch
    import paper_1505_03851_amd as lda
    c = make_random(64 * 50 + 3, 40, 900, 1024, seed=5)
    dev = to_device(c)
    route = lda.route_build(dev["doc_id"], dev["word_id"], c.M, c.V)
    out = torch.full_like(dev["doc_id"], -1)
    for sweep in range(3):
        u = np.random.default_rng(100 + sweep).integers(0, 1 << 24, c.N) * 2.0 ** -24
        c.u[:] = u.astype(np.float32)
        lda.draw_routed(dev["theta"], dev["phi"], route, torch.from_numpy(c.u).cuda(), out=out)
        torch.cuda.synchronize()
        rep = compare(c, out.cpu().numpy())
        print(f"[parity] reuse sweep {sweep}: {rep}", flush=True)
        assert rep.hard == 0, rep.first_hard


def test_routed_equal_power_of_two_weights_exact():
    """All products 2**-3 (every fp32 partial sum exact): z = floor(u*K)."""
    import torch
    import paper_1505_03851_amd as lda
    from paper_1505_03851_amd.inputs import Corpus
    N, K = 64 * 37 + 11, 1024
    rng = np.random.default_rng(3)
    u = (rng.integers(0, 1 << 24, N) * 2.0 ** -24).astype(np.float32)
    u[:4] = [0.0, 2.0 ** -24, 0.5, 1 - 2.0 ** -24]
    c = Corpus(np.full((3, K), 2.0 ** -3, np.float32), np.ones((5, K), np.float32),
               (np.arange(N) % 3).astype(np.int32), (np.arange(N) % 5).astype(np.int32), u)
    z = run_kernel("routed", to_device(c))
    assert (z == np.floor(u.astype(np.float64) * K).astype(np.int32)).all()


@pytest.mark.parametrize("K", [64, 256, 512, 764, 770, 2052])
def test_routed_rejects_unsupported_k(K):
    """Below K = 768 routing is measured slower than the token-order draw and
    the routed draw refuses; so it does for K not divisible by 4 and above
    2048."""
    import paper_1505_03851_amd as lda
    c = make_random(200, 5, 50, K, seed=1)
    dev = to_device(c)
    route = lda.route_build(dev["doc_id"], dev["word_id"], c.M, c.V)
    with pytest.raises(lda.LdaError) as e:
        lda.draw_routed(dev["theta"], dev["phi"], route, dev["u"])
    assert e.value.status == lda.STATUS["LDA_ERR_UNSUPPORTED"]


def test_route_counts_every_token_whatever_its_id():
    """The class count and the scatter agree on which tokens exist (index
    below N), whatever the word id: ids outside [0, V) -- negative ones here
    -- get a class like any other, every list holds exactly its counted
    tokens, and the route stays a permutation of the tokens.  (The routing
    only; no draw runs on such ids.)"""
    c = make_random(64 * 40 + 9, 20, 300, 1024, seed=9)
    c.word_id[[3, 700, 2000, c.N - 1]] = [-1, -5, -(2 ** 31), -77]
    print(f"[case] route with negative word ids {c.name}", flush=True)
    route, arr = build(c, validate=False)
    check_route(c, route, arr)


@pytest.mark.parametrize("name", ["corpus16M-K1024", "poisson300-K2048"])
def test_routed_philox(name):
    """The routed draw with in-kernel uniforms: against the oracle fed the
    oracle's own Philox uniforms of the original token indices, and equal to
    the unrouted draw_philox except inside the rounding band."""
    import torch
    import paper_1505_03851_amd as lda
    from oracle import philox as px
    seed, sweep = 0x5EED_2015_0513_0002, 5
    c = make_corpus(name)
    c.u = px.token_uniforms(seed, sweep, 0, c.N)
    print(f"[case] routed philox {name}", flush=True)
    dev = to_device(c)
    route = lda.route_build(dev["doc_id"], dev["word_id"], c.M, c.V)
    z = lda.draw_routed_philox(dev["theta"], dev["phi"], route, seed, sweep)
    z_plain = lda.draw_philox(dev["theta"], dev["phi"], dev["doc_id"], dev["word_id"], seed, sweep)
    torch.cuda.synchronize()
    z, z_plain = z.cpu().numpy(), z_plain.cpu().numpy()
    rep = compare(c, z)
    print(f"[parity] {name} routed philox: {rep}", flush=True)
    assert rep.hard == 0, rep.first_hard
    assert rep.mismatch_rate < MAX_MISMATCH_RATE
    differ = np.nonzero(z != z_plain)[0]
    assert differ.size <= max(1, c.N // 10000), differ.size
    if differ.size:
        assert compare(c, z, differ).hard == 0
