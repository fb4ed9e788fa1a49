"""The draw with in-kernel uniforms (Philox4x32-10) on the GPU: the
uniforms bit for bit against the oracle's generator, and the draw against
the oracle's definition fed those uniforms."""
import numpy as np
import pytest

import oracle
from oracle import philox as px
from paper_1505_03851_amd.inputs import make_corpus, make_random
from parity import MAX_MISMATCH_RATE, compare, to_device

pytestmark = pytest.mark.gpu

SEED = 0x5EED_2015_0513_0001


@pytest.mark.parametrize("count,first,seed,sweep", [
    (1, 0, 0, 0),
    (1000, 0, SEED, 3),
    ((1 << 20) + 77, 12345, SEED, 0),
    (5000, (1 << 32) - 2500, SEED, 1),          # across the counter's word boundary
    (300, (1 << 40) + 5, 2 ** 64 - 1, 2 ** 32 - 1),
    (301, (1 << 63) - 302, SEED, 7),            # first + count = INT64_MAX, the limit
])
def test_uniforms_bit_exact(count, first, seed, sweep):
    import torch
    import paper_1505_03851_amd as lda
    print(f"[case] uniforms count={count} first={first}", flush=True)
    u = lda.philox_uniforms(count, seed, sweep, first=first)
    torch.cuda.synchronize()
    ref = px.token_uniforms(seed, sweep, first, count)
    got = u.cpu().numpy()
    assert got.dtype == np.float32
    assert (got.view(np.uint32) == ref.view(np.uint32)).all(), np.nonzero(got != ref)[0][:10]


def _z_philox(c, seed, sweep):
    import torch
    import paper_1505_03851_amd as lda
    dev = to_device(c)
    z = lda.draw_philox(dev["theta"], dev["phi"], dev["doc_id"], dev["word_id"], seed, sweep)
    torch.cuda.synchronize()
    return z.cpu().numpy()


def _with_u(c, seed, sweep):
    c.u = px.token_uniforms(seed, sweep, 0, c.N)
    return c


@pytest.mark.parametrize("name", ["tiny-K32", "corpus1M-K64", "corpus1M-K256", "wiki-shaped-K80",
                                  "wiki-shaped-K240"])
def test_philox_draw_every_token(name):
    c = _with_u(make_corpus(name), SEED, 7)
    print(f"[case] philox {name}", flush=True)
    z = _z_philox(c, SEED, 7)
    rep = compare(c, z)
    print(f"[parity] {name} philox: {rep}", flush=True)
    assert rep.hard == 0, rep.first_hard
    if c.N >= 1 << 20:
        assert rep.mismatch_rate < MAX_MISMATCH_RATE


@pytest.mark.parametrize("name", ["corpus16M-K1024", "poisson300-K2048"])
def test_philox_draw_full_size_every_token(name):
    c = _with_u(make_corpus(name), SEED, 0)
    print(f"[case] philox {name}", flush=True)
    z = _z_philox(c, SEED, 0)
    rep = compare(c, z)
    print(f"[parity] {name} philox: {rep}", flush=True)
    assert rep.hard == 0 and rep.mismatch_rate < MAX_MISMATCH_RATE, str(rep)


@pytest.mark.parametrize("N,K", [(1, 5), (63, 64), (64 * 9 + 17, 19), (64 * 21 + 5, 256),
                                 (64 * 13 + 3, 300), (64 * 17 + 9, 1000)])
def test_philox_draw_equals_draw_with_written_uniforms(N, K):
    """Same kernel, same uniforms: identical z to the draw given the
    uniforms lda_philox_uniforms writes."""
    import torch
    import paper_1505_03851_amd as lda
    c = make_random(N, 13, 200, K, seed=N * K, doc_order="shuffled")
    dev = to_device(c)
    u = lda.philox_uniforms(N, SEED, 11)
    z1 = lda.draw_butterfly(dev["theta"], dev["phi"], dev["doc_id"], dev["word_id"], u)
    z2 = lda.draw_philox(dev["theta"], dev["phi"], dev["doc_id"], dev["word_id"], SEED, 11)
    torch.cuda.synchronize()
    assert (z1.cpu().numpy() == z2.cpu().numpy()).all()
    c.u = px.token_uniforms(SEED, 11, 0, N)
    rep = compare(c, z2.cpu().numpy())
    assert rep.hard == 0, rep.first_hard


def test_sweeps_draw_different_topics():
    """Two sweeps differ where the oracle's draws with the two sweeps'
    uniforms differ (16% of the tokens of this corpus)."""
    c = make_corpus("tiny-K32")
    z0, z1 = _z_philox(c, SEED, 0), _z_philox(c, SEED, 1)
    r0, _ = oracle.draw(c.theta, c.phi, c.doc_id, c.word_id, px.token_uniforms(SEED, 0, 0, c.N))
    r1, _ = oracle.draw(c.theta, c.phi, c.doc_id, c.word_id, px.token_uniforms(SEED, 1, 0, c.N))
    assert (r0 != r1).mean() > 0.1
    assert abs((z0 != z1).mean() - (r0 != r1).mean()) < 0.01
