"""The C ABI on a non-default stream and inside a captured HIP graph: the
entry points enqueue kernels only (no allocation, no memset), so a graph
replays them; every replay is checked against an eager call."""
import numpy as np
import pytest

from paper_1505_03851_amd.inputs import make_corpus, make_random
from parity import compare, to_device

pytestmark = pytest.mark.gpu


def test_side_stream_orders_with_events():
    import torch
    import paper_1505_03851_amd as lda
    c = make_corpus("corpus1M-K64")
    dev = to_device(c)
    print("[case] side stream corpus1M-K64", flush=True)
    ref = lda.draw_butterfly(dev["theta"], dev["phi"], dev["doc_id"], dev["word_id"], dev["u"])
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        z = torch.empty_like(ref)
        lda.draw_butterfly(dev["theta"], dev["phi"], dev["doc_id"], dev["word_id"], dev["u"],
                           out=z, stream=side)
    torch.cuda.current_stream().wait_stream(side)
    assert (z.cpu() == ref.cpu()).all()


@pytest.mark.parametrize("kernel", ["butterfly", "docs", "philox", "routed"])
def test_graph_capture_and_replay(kernel):
    """Capture one draw, then replay it three times with new uniforms (or a
    new seed in the captured seed's place: the philox draw's uniforms are
    fixed by the capture, so its replays must repeat); each replay equals an
    eager draw on the same inputs, with eager work between the replays.  The
    routed draw's routing is built before the capture (its build waits on
    the stream and cannot be captured)."""
    import torch
    import paper_1505_03851_amd as lda
    from paper_1505_03851_amd.inputs import doc_offsets
    K = 1000 if kernel == "routed" else 200   # (the routed draw takes K >= 768)
    c = make_random(64 * 300 + 17, 200, 3000, K, seed=5, doc_order="ragged")
    dev = to_device(c)
    off = torch.from_numpy(doc_offsets(c.doc_id, c.M)).cuda()
    route = lda.route_build(dev["doc_id"], dev["word_id"], c.M, c.V) if kernel == "routed" else None
    z = torch.empty(c.N, dtype=torch.int32, device="cuda")

    def launch(out, stream=None):
        if kernel == "butterfly":
            return lda.draw_butterfly(dev["theta"], dev["phi"], dev["doc_id"], dev["word_id"],
                                      dev["u"], out=out, stream=stream)
        if kernel == "docs":
            return lda.draw_docs(dev["theta"], dev["phi"], off, dev["word_id"], dev["u"],
                                 out=out, stream=stream)
        if kernel == "routed":
            return lda.draw_routed(dev["theta"], dev["phi"], route, dev["u"], out=out,
                                   stream=stream)
        return lda.draw_philox(dev["theta"], dev["phi"], dev["doc_id"], dev["word_id"],
                               1234, 7, out=out, stream=stream)

    print(f"[case] graph {kernel}", flush=True)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        launch(z)                      # warm-up outside the capture
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        launch(z)
    rng = np.random.default_rng(9)
    for rep in range(3):
        if kernel != "philox":
            new_u = (rng.integers(0, 1 << 24, c.N) * 2.0 ** -24).astype(np.float32)
            dev["u"].copy_(torch.from_numpy(new_u))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = z.clone()
        eager = launch(torch.empty_like(z))
        torch.cuda.synchronize()
        assert (got.cpu() == eager.cpu()).all(), rep
        if kernel != "philox":
            c.u = new_u
            rep_ = compare(c, got.cpu().numpy())
            assert rep_.hard == 0, rep_.first_hard
