"""Shared helpers of the GPU parity tests: upload a corpus, run a kernel
through the C ABI, and compare with the oracle under the band rule."""
from __future__ import annotations

import dataclasses

import numpy as np

import oracle

BAND_REL = 1e-5          # |u*S - S_k| <= 1e-5 * S marks a token as in-band
MAX_MISMATCH_RATE = 1e-4  # mismatches (all in-band) per token


@dataclasses.dataclass
class ParityReport:
    n: int
    mismatches: int
    hard: int            # mismatches outside the band, or inside it at a topic
                         # the band does not admit (see ``admissible``)
    in_band: int         # tokens inside the band (a property of the data)
    first_hard: list

    @property
    def mismatch_rate(self) -> float:
        return self.mismatches / max(self.n, 1)

    def __str__(self):
        return (f"n={self.n} mismatches={self.mismatches} "
                f"({self.mismatch_rate:.2e}) hard={self.hard} "
                f"in_band={self.in_band} ({self.in_band / max(self.n, 1):.2e})")


def admissible(theta, phi, d, w, u, z) -> np.ndarray:
    """For tokens (documents d, words w, uniforms u) drawn as topics z: whether
    each z is a topic the rounding band admits.  In the band several topics
    are correct, but only those whose fp64 prefix range [S_{z-1}, S_z] comes
    within 1e-5 S of stop = u S (z = K - 1 also when stop lies past S_{K-1});
    with S = 0 only K - 1 (no prefix exceeds stop)."""
    K = theta.shape[1]
    ok = np.empty(len(z), bool)
    for i in range(len(z)):
        S = oracle.prefix_np(theta[d[i]], phi[w[i]])
        total = S[-1]
        k = int(z[i])
        if total == 0.0:
            ok[i] = k == K - 1
            continue
        stop = float(u[i]) * total
        tol = BAND_REL * total
        below = S[k - 1] if k > 0 else 0.0
        ok[i] = below <= stop + tol and (S[k] >= stop - tol or k == K - 1)
    return ok


def to_device(c, device="cuda"):
    import torch
    return dict(
        theta=torch.from_numpy(c.theta).to(device),
        phi=torch.from_numpy(c.phi).to(device),
        doc_id=torch.from_numpy(c.doc_id).to(device),
        word_id=torch.from_numpy(c.word_id).to(device),
        u=torch.from_numpy(c.u).to(device),
    )


def run_kernel(kernel: str, dev: dict):
    """z by ``kernel``; "docs", "doc_lanes" and "doc_lanes_cache" hand the
    documents over as offsets (the corpus's documents must be contiguous); "variant-<name>" is the
    butterfly kernel with the named block table; "routed" routes the tokens to
    the XCDs (route_build) and draws them with draw_routed."""
    import torch
    import paper_1505_03851_amd as lda
    if kernel in ("docs", "doc_lanes", "doc_lanes_cache"):
        from paper_1505_03851_amd.inputs import doc_offsets
        off = doc_offsets(dev["doc_id"].cpu().numpy(), dev["theta"].shape[0])
        off = torch.from_numpy(off).to(dev["theta"].device)
        args = (dev["theta"], dev["phi"], off, dev["word_id"], dev["u"])
        if kernel == "docs":
            z = lda.draw_docs(*args, validate=True)
        else:
            z = lda.draw_doc_lanes(*args, theta_cache=kernel == "doc_lanes_cache",
                                   validate=True)
        torch.cuda.synchronize()
        return z.cpu().numpy()
    if kernel == "routed":
        M, V = dev["theta"].shape[0], dev["phi"].shape[0]
        route = lda.route_build(dev["doc_id"], dev["word_id"], M, V, validate=True)
        z = lda.draw_routed(dev["theta"], dev["phi"], route, dev["u"])
        torch.cuda.synchronize()
        return z.cpu().numpy()
    if kernel.startswith("variant-"):
        z = lda.draw_variant(dev["theta"], dev["phi"], dev["doc_id"], dev["word_id"],
                             dev["u"], variant=kernel[len("variant-"):])
        torch.cuda.synchronize()
        return z.cpu().numpy()
    fn = {"naive": lda.draw_naive, "butterfly": lda.draw_butterfly,
          "transposed": lda.draw_transposed}[kernel]
    z = fn(dev["theta"], dev["phi"], dev["doc_id"], dev["word_id"], dev["u"])
    torch.cuda.synchronize()
    return z.cpu().numpy()


_NAMED = {}


def named_corpus(name):
    """A named workload, kept (with its oracle result, see ``reference``)
    until another name is asked for: one full-size corpus in memory at a
    time."""
    from paper_1505_03851_amd.inputs import make_corpus
    if name not in _NAMED:
        _NAMED.clear()
        _NAMED[name] = {"corpus": make_corpus(name)}
    return _NAMED[name]["corpus"]


def reference(name):
    """The oracle's z and band flags for every token of the named workload
    (computed once, then reused by every kernel compared with it)."""
    c = named_corpus(name)
    ent = _NAMED[name]
    if "ref" not in ent:
        ent["ref"] = oracle.draw(c.theta, c.phi, c.doc_id, c.word_id, c.u,
                                 band_rel=BAND_REL)
    return ent["ref"]


def compare(c, z_gpu, idx=None, ref=None) -> ParityReport:
    """Oracle on tokens ``idx`` (all if None) against the GPU's z there.
    ``ref``: the oracle's (z, band) for every token of ``c``, if already
    computed (``reference``)."""
    if idx is None:
        d, w, u, zg = c.doc_id, c.word_id, c.u, z_gpu
    else:
        d, w, u, zg = c.doc_id[idx], c.word_id[idx], c.u[idx], z_gpu[idx]
    if ref is not None:
        z_ref, band = ref if idx is None else (ref[0][idx], ref[1][idx])
    else:
        z_ref, band = oracle.draw(c.theta, c.phi, d, w, u, band_rel=BAND_REL)
    mis = zg != z_ref
    hard = mis & ~band
    soft = np.nonzero(mis & band)[0]          # in the band: check the topic is admitted
    if soft.size:
        hard[soft] = ~admissible(c.theta, c.phi, d[soft], w[soft], u[soft], zg[soft])
    where = np.nonzero(hard)[0][:5]
    first = [(int(i if idx is None else idx[i]), int(zg[i]), int(z_ref[i]))
             for i in where]
    return ParityReport(int(zg.size), int(mis.sum()), int(hard.sum()),
                        int(band.sum()), first)
