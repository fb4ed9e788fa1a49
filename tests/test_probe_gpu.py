"""GPU checks of the measurement probes (liblda_probe.so): the streaming read
reads every byte it is given the stated number of times, and the draw floor
writes every token's output slot."""
import numpy as np
import pytest

from paper_1505_03851_amd.inputs import make_random
from parity import to_device

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("floats,passes", [(4, 1), (1 << 20, 3), ((1 << 22) + 4, 2)])
def test_read_probe_reads_everything(floats, passes):
    import torch
    from paper_1505_03851_amd import probe
    buf = torch.ones(floats, dtype=torch.float32, device="cuda")
    out = torch.empty(probe.READ_OUT_FLOATS, dtype=torch.float32, device="cuda")
    print(f"[case] read probe floats={floats} passes={passes}", flush=True)
    probe.read(buf, passes, out)
    torch.cuda.synchronize()
    # every lane's sum is an integer below 2^24: exact in fp32
    assert int(out.double().sum()) == floats * passes


@pytest.mark.parametrize("K,wpg,wpc", [(32, 2, 0), (64, 2, 12), (128, 2, 0), (208, 2, 12),
                                       (256, 2, 0), (1000, 4, 8), (1024, 4, 0), (2048, 2, 16)])
def test_floor_probe_writes_every_token(K, wpg, wpc):
    import torch
    from paper_1505_03851_amd import probe
    c = make_random(64 * 40 + 9, 30, 500, K, seed=K, doc_order="sequential")
    dev = to_device(c)
    out = torch.full((c.N,), -1, dtype=torch.int32, device="cuda")
    print(f"[case] floor probe K={K} wpg={wpg} wpc={wpc}", flush=True)
    for window in (8, 16):
        out.fill_(-1)
        probe.draw_floor(dev["theta"], dev["phi"], dev["doc_id"], dev["word_id"], dev["u"], out,
                         window=window, waves_per_group=wpg, waves_per_cu=wpc)
        torch.cuda.synchronize()
        # each slot holds the bits of a positive float sum: never -1
        assert (out.cpu().numpy() != -1).all()
