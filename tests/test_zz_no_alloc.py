"""The routed draw with the library's own scratch array
(lda_draw_routed_scratch), called through the C ABI: on two calls in a row
(the second with fewer tokens, so a stale routing in the array would show),
its z equals that of lda_route_build + lda_draw_routed with a caller's
workspace token for token (the same kernels and arithmetic), and the
oracle's under the rounding-band rule; sizes whose routing does not fit the
array are refused before any HIP call."""
import ctypes

import numpy as np
import pytest

from paper_1505_03851_amd.inputs import make_random
from parity import compare, to_device

pytestmark = pytest.mark.gpu


def _scratch_draw(dev, c, out):
    import torch
    from paper_1505_03851_amd import _lib
    st = _lib.load().lda_draw_routed_scratch(
        dev["theta"].data_ptr(), dev["phi"].data_ptr(), dev["doc_id"].data_ptr(),
        dev["word_id"].data_ptr(), dev["u"].data_ptr(), out.data_ptr(), c.N, c.M, c.V, c.K,
        ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == 0, _lib.status_string(st)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def _workspace_draw(dev, c):
    import torch
    import paper_1505_03851_amd as lda
    route = lda.route_build(dev["doc_id"], dev["word_id"], c.M, c.V)
    z = lda.draw_routed(dev["theta"], dev["phi"], route, dev["u"])
    torch.cuda.synchronize()
    return z.cpu().numpy()


def test_scratch_routed_draw_two_calls():
    import torch
    cases = [make_random(64 * 6000 + 17, 1500, 20_000, 1024, seed=41, doc_order="sequential"),
             make_random(64 * 700 + 5, 90, 3000, 768, seed=42, doc_order="ragged")]
    for c in cases:
        print(f"[case] scratch routed draw {c.name}", flush=True)
        dev = to_device(c)
        out = torch.full((c.N,), -1, dtype=torch.int32, device="cuda")
        z = _scratch_draw(dev, c, out)
        z_ws = _workspace_draw(dev, c)
        diff = np.nonzero(z != z_ws)[0]
        assert diff.size == 0, (diff.size, diff[:5])
        rep = compare(c, z)
        print(f"[parity] {c.name} routed scratch: {rep}", flush=True)
        assert rep.hard == 0, rep.first_hard


def test_scratch_routed_draw_at_its_largest_n():
    """The largest N whose routing fits the array (about 5.4M tokens): the
    whole array in use, the same z as with a caller's workspace."""
    import torch
    import paper_1505_03851_amd as lda
    from paper_1505_03851_amd import _lib
    cap = _lib.ROUTED_SCRATCH_BYTES
    lo, hi = 1, 1 << 24              # route_workspace_bytes(lo) <= cap < ...(hi)
    while hi - lo > 1:
        mid = (lo + hi) // 2
        lo, hi = (mid, hi) if lda.route_workspace_bytes(mid) <= cap else (lo, mid)
    c = make_random(lo, 4000, 5000, 768, seed=43, doc_order="sequential")
    print(f"[case] scratch routed draw at its largest N={c.N}", flush=True)
    dev = to_device(c)
    out = torch.full((c.N,), -1, dtype=torch.int32, device="cuda")
    z = _scratch_draw(dev, c, out)
    z_ws = _workspace_draw(dev, c)
    diff = np.nonzero(z != z_ws)[0]
    assert diff.size == 0, (diff.size, diff[:5])
    rep = compare(c, z)
    print(f"[parity] {c.name} routed scratch: {rep}", flush=True)
    assert rep.hard == 0 and rep.mismatch_rate < 1e-4, rep.first_hard


def test_scratch_refuses_what_does_not_fit():
    """Rejected on the host (no kernel runs): a routing larger than the
    array, K below the routed draw's range, and bad shapes."""
    import paper_1505_03851_amd as lda
    from paper_1505_03851_amd import _lib
    lib = _lib.load()
    cap = _lib.ROUTED_SCRATCH_BYTES
    fits = max(n for n in range(5_000_000, 6_000_000, 1024)
               if lda.route_workspace_bytes(n) <= cap)
    too_big = next(n for n in range(fits, fits + 4096) if lda.route_workspace_bytes(n) > cap)
    A = 4096       # a stand-in pointer: never dereferenced by a rejected call
    run = lambda N, K=1024: lib.lda_draw_routed_scratch(A, A, A, A, A, A, N, 5, 7, K, None)
    assert run(too_big) == _lib.STATUS["LDA_ERR_UNSUPPORTED"]
    assert run(1000, K=512) == _lib.STATUS["LDA_ERR_UNSUPPORTED"]
    assert run(-1) == _lib.STATUS["LDA_ERR_SHAPE"]
    assert run(0) == 0
