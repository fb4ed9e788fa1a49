"""ctypes binding of liblda_probe.so (include/lda_probe.h): the measurement
probes, argument marshalling only.  Used by bench.py to time the draw's
memory floor and the rates at which HBM and the MALL serve reads."""
from __future__ import annotations

import ctypes
import os

import torch

from ._lib import LdaError, _CONSTS, _check, _stream_handle

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "liblda_probe.so")
HEADER = os.path.join(os.path.dirname(_PKG), "include", "lda_probe.h")
READ_GROUPS = 2048
READ_OUT_FLOATS = READ_GROUPS * 256

_lib = None


def load() -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with "
                          "`python -c 'import __graft_entry__ as g; g.build()'`")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    lib.lda_probe_draw_floor.argtypes = [P, P, P, P, P, P, I64, I32, I32, I32, I32, I32, I32, P]
    lib.lda_probe_draw_floor.restype = ctypes.c_int
    lib.lda_probe_read.argtypes = [P, I64, I32, P, P]
    lib.lda_probe_read.restype = ctypes.c_int
    _lib = lib
    return lib


def draw_floor(theta, phi, doc_id, word_id, u, out, window: int = 16,
               waves_per_group: int = 2, waves_per_cu: int = 0, stream=None) -> None:
    """Enqueue one memory-only pass of the draw's access pattern (see
    lda_probe_draw_floor); ``out`` (int32 [N]) receives values of no
    meaning."""
    M, K = theta.shape
    V = phi.shape[0]
    N = doc_id.shape[0]
    st = load().lda_probe_draw_floor(theta.data_ptr(), phi.data_ptr(), doc_id.data_ptr(),
                                     word_id.data_ptr(), u.data_ptr(), out.data_ptr(), N, M, V,
                                     K, window, waves_per_group, waves_per_cu,
                                     _stream_handle(stream))
    _check(st)


def read(buf: torch.Tensor, passes: int, out: torch.Tensor, stream=None) -> None:
    """Enqueue ``passes`` streaming reads of ``buf`` (lda_probe_read);
    ``out``: float32 [READ_OUT_FLOATS]."""
    if out.numel() < READ_OUT_FLOATS or out.dtype != torch.float32:
        raise ValueError(f"out must hold {READ_OUT_FLOATS} float32")
    st = load().lda_probe_read(buf.data_ptr(), buf.numel() * buf.element_size(), int(passes),
                               out.data_ptr(), _stream_handle(stream))
    _check(st)


__all__ = ["draw_floor", "read", "load", "LdaError", "READ_OUT_FLOATS"]
assert _CONSTS  # the status codes come from lda_draw.h
