"""Token counts past 2**31: every kernel indexes tokens with 64-bit integers.

The inputs are made on the GPU (about 35 GB of token arrays); a sample of the
tokens -- random ones, the first and last, and those around token 2**31 --
is checked against the oracle under the rounding-band rule.
"""
import numpy as np
import pytest

from parity import BAND_REL, MAX_MISMATCH_RATE
from paper_1505_03851_amd.inputs import dirichlet_columns, dirichlet_rows

pytestmark = pytest.mark.gpu

N_BIG = (1 << 31) + 4099          # past the signed 32-bit range, ragged tail
M_BIG = 32771                     # documents of about 65,500 tokens
V_BIG = 5000


def _sample(N):
    rng = np.random.default_rng(31)
    parts = [rng.choice(N, size=1 << 17, replace=False), np.arange(4096),
             np.arange(N - 4096, N), np.arange((1 << 31) - 2048, (1 << 31) + 2048)]
    return np.unique(np.concatenate(parts))


@pytest.fixture(scope="module")
def big():
    import torch
    torch.cuda.empty_cache()
    g = torch.Generator(device="cuda")
    g.manual_seed(2015)
    N = N_BIG
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
    hard = int((mis & ~band).sum())
    print(f"[parity] large-N{N_BIG}-K{K} {kernel}: n={z.size} mismatches={int(mis.sum())} "
          f"hard={hard} in_band={int(band.sum())}", flush=True)
    assert hard == 0, big["idx"][np.nonzero(mis & ~band)[0][:5]]
    assert mis.mean() < MAX_MISMATCH_RATE
