"""CPU oracle for the per-token LDA topic draw -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the HIP library
and never imports it.

Contents
  draw / draw_np        the plain definition of the draw (Section 2, Algorithm
                        1 with the searches of Algorithms 2/3), fp64; ``draw``
                        runs the C file ``lda_oracle.c``, ``draw_np`` is a numpy
                        twin for small inputs.
  prefix_np             the full table of partial sums of one token (Fig. 1,
                        left).
  counts / counts_np    the per-document and per-word topic counts of a set of
                        draws (the statistics the update of theta and phi
                        consumes, Section 1), integer and exact; ``counts``
                        runs the C file, ``counts_np`` is a numpy twin.
  butterfly             the butterfly-patterned table of Section 4, three ways:
                        its closed form, the replacement process that builds it,
                        and a lane-vector simulation of the search over it
                        (Algorithms 9 and 10), and the table and descent search
                        of the alternative replacement rule.
  philox                Philox4x32-10 / 4x64-10 from their published definition
                        and the per-token uniforms of the fused-RNG draw.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import butterfly  # noqa: F401  (re-exported)
from . import philox  # noqa: F401  (re-exported)

BAND_REL = 1e-5  # width of the rounding band, relative to the token's total

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liblda_oracle.so")
_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    src = os.path.join(_HERE, "lda_oracle.c")
    if (not os.path.exists(_LIB_PATH)
            or os.path.getmtime(_LIB_PATH) < os.path.getmtime(src)):
        from .build import build
        build()
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    lib.oracle_draw.argtypes = [P, P, P, P, P, ctypes.c_int64, ctypes.c_int32,
                                P, P, ctypes.c_double]
    lib.oracle_draw.restype = ctypes.c_int
    lib.oracle_num_threads.restype = ctypes.c_int
    lib.oracle_set_num_threads.argtypes = [ctypes.c_int]
    lib.oracle_set_num_threads.restype = None
    lib.oracle_counts.argtypes = [P, P, P, ctypes.c_int64, ctypes.c_int32,
                                  ctypes.c_int32, ctypes.c_int32, P, P]
    lib.oracle_counts.restype = ctypes.c_int64
    _lib = lib
    return lib


def num_threads() -> int:
    """OpenMP threads the C oracle uses."""
    return int(_load().oracle_num_threads())


def set_num_threads(n: int) -> None:
    """OpenMP threads for the following draws (timing only)."""
    _load().oracle_set_num_threads(int(n))


def _as(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a


def draw(theta, phi, doc_id, word_id, u, *, with_band: bool = True,
         band_rel: float = BAND_REL):
    """z[n] (int32) and, if ``with_band``, in_band[n] (bool) for every token.

    z[n] = min{k : u[n] * S_n < S_{n,k}} with S_{n,k} the fp64 sequential
    prefix of theta[doc_id[n]] * phi[word_id[n]] and S_n = S_{n,K-1}; K - 1
    when no k qualifies.
    """
    theta = _as(theta, np.float32)
    phi = _as(phi, np.float32)
    doc_id = _as(doc_id, np.int32)
    word_id = _as(word_id, np.int32)
    u = _as(u, np.float32)
    N = doc_id.shape[0]
    K = theta.shape[1]
    assert phi.shape[1] == K and word_id.shape[0] == N and u.shape[0] == N
    assert K >= 1
    if N:
        assert 0 <= doc_id.min() and doc_id.max() < theta.shape[0]
        assert 0 <= word_id.min() and word_id.max() < phi.shape[0]
    z = np.empty(N, dtype=np.int32)
    band = np.empty(N, dtype=np.uint8) if with_band else None
    lib = _load()
    rc = lib.oracle_draw(theta.ctypes.data, phi.ctypes.data,
                         doc_id.ctypes.data, word_id.ctypes.data,
                         u.ctypes.data, N, K, z.ctypes.data,
                         band.ctypes.data if with_band else None,
                         float(band_rel))
    if rc != 0:
        raise MemoryError("oracle_draw could not allocate its scratch row")
    return (z, band.astype(bool)) if with_band else z


def prefix_np(theta_row, phi_row) -> np.ndarray:
    """S_k of one token: sequential fp64 sum of the exact fp64 products."""
    a = np.asarray(theta_row, np.float32).astype(np.float64) * \
        np.asarray(phi_row, np.float32).astype(np.float64)
    return np.cumsum(a)


def draw_np(theta, phi, doc_id, word_id, u, band_rel: float = BAND_REL):
    """Numpy twin of ``draw`` (N x K fp64 work array: small inputs only)."""
    theta = np.asarray(theta, np.float32)
    phi = np.asarray(phi, np.float32)
    a = theta[np.asarray(doc_id)].astype(np.float64) * \
        phi[np.asarray(word_id)].astype(np.float64)
    S = np.cumsum(a, axis=1)
    K = S.shape[1]
    total = S[:, -1]
    stop = np.asarray(u, np.float32).astype(np.float64) * total
    hit = stop[:, None] < S
    z = np.where(hit.any(axis=1), hit.argmax(axis=1), K - 1).astype(np.int32)
    band = (np.abs(stop[:, None] - S) <= band_rel * total[:, None]).any(axis=1)
    return z, band


def counts(doc_id, word_id, z, M: int, V: int, K: int):
    """(ndk int32 [M][K], nwk int32 [V][K]): ndk[d][k] is the number of
    tokens of document d drawn to topic k, nwk[w][k] the number of tokens of
    word w drawn to topic k.  A token with an id or topic out of range is not
    counted."""
    doc_id = _as(doc_id, np.int32)
    word_id = _as(word_id, np.int32)
    z = _as(z, np.int32)
    N = doc_id.shape[0]
    assert word_id.shape[0] == N and z.shape[0] == N
    assert M >= 1 and V >= 1 and K >= 1
    ndk = np.empty((M, K), dtype=np.int32)
    nwk = np.empty((V, K), dtype=np.int32)
    _load().oracle_counts(doc_id.ctypes.data, word_id.ctypes.data, z.ctypes.data,
                          N, M, V, K, ndk.ctypes.data, nwk.ctypes.data)
    return ndk, nwk


def counts_np(doc_id, word_id, z, M: int, V: int, K: int):
    """Numpy twin of ``counts``: a histogram of the flat cell index of every
    counted token."""
    d = np.asarray(doc_id, np.int64)
    w = np.asarray(word_id, np.int64)
    k = np.asarray(z, np.int64)
    ok = (d >= 0) & (d < M) & (w >= 0) & (w < V) & (k >= 0) & (k < K)
    d, w, k = d[ok], w[ok], k[ok]
    ndk = np.bincount(d * K + k, minlength=M * K).reshape(M, K).astype(np.int32)
    nwk = np.bincount(w * K + k, minlength=V * K).reshape(V, K).astype(np.int32)
    return ndk, nwk
