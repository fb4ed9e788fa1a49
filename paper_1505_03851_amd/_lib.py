"""ctypes binding of liblda_draw.so: argument marshalling only.

torch supplies device memory and the current stream; every step of the draw
runs in the HIP kernels.  There is no fallback: if the library is missing or
fails to load, every entry point raises.
"""
from __future__ import annotations

import ctypes
import os
import re

import torch  # loaded first so the library binds to torch's HIP runtime

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "liblda_draw.so")
HEADER = os.path.join(os.path.dirname(_PKG), "include", "lda_draw.h")

_lib = None


class LdaError(RuntimeError):
    """A non-zero status returned by the C ABI."""

    def __init__(self, status: int, message: str):
        super().__init__(f"lda status {status}: {message}")
        self.status = status


def _header_constants() -> dict[str, int]:
    consts = {}
    with open(HEADER) as f:
        for m in re.finditer(r"#define\s+(LDA_\w+)\s+\(?(-?\d+)\)?", f.read()):
            consts[m.group(1)] = int(m.group(2))
    return consts


_CONSTS = _header_constants()
# status codes (LDA_OK and LDA_ERR_*) and size limits from the header
STATUS = {k: v for k, v in _CONSTS.items() if k == "LDA_OK" or k.startswith("LDA_ERR_")}
MAX_K = _CONSTS["LDA_MAX_K"]
MAX_N = _CONSTS["LDA_MAX_N"]
MAX_TABLE_BYTES = _CONSTS["LDA_MAX_TABLE_BYTES"]
MAX_COUNT_TABLE_BYTES = _CONSTS["LDA_MAX_COUNT_TABLE_BYTES"]
DOC_LANES_MAX_CACHE_BYTES = _CONSTS["LDA_DOC_LANES_MAX_CACHE_BYTES"]
# table variants of lda_draw_butterfly_variant, by name
ROUTED_SCRATCH_BYTES = _CONSTS["LDA_ROUTED_SCRATCH_BYTES"]
VARIANTS = {"register": _CONSTS["LDA_VARIANT_REGISTER_TABLE"],
            "lds": _CONSTS["LDA_VARIANT_LDS_TABLE"],
            "lds_alt": _CONSTS["LDA_VARIANT_LDS_TABLE_ALT"],
            "leaf8": _CONSTS["LDA_VARIANT_LEAF8"],
            "wide": _CONSTS["LDA_VARIANT_WIDE_TABLES"]}


class RouteInfo(ctypes.Structure):
    """struct lda_route: the sizes of the eight routed lists."""
    _fields_ = [("N", ctypes.c_int64), ("tokens", ctypes.c_int64 * 8),
                ("start", ctypes.c_int64 * 8), ("length", ctypes.c_int64 * 8)]


def load() -> ctypes.CDLL:
    """Load the library (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it with "
            "`python -c 'import __graft_entry__ as g; g.build()'` "
            "(or python paper_1505_03851_amd/build.py)")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    draw_args = [P, P, P, P, P, P, I64, I32, I32, I32, P]
    for name in ("lda_draw_naive", "lda_draw_butterfly", "lda_draw_transposed"):
        getattr(lib, name).argtypes = draw_args
        getattr(lib, name).restype = ctypes.c_int
    lib.lda_draw_butterfly_variant.argtypes = draw_args[:-1] + [I32, P]
    lib.lda_draw_butterfly_variant.restype = ctypes.c_int
    lib.lda_draw_butterfly_philox.argtypes = [P, P, P, P, P, I64, I32, I32, I32,
                                              ctypes.c_uint64, ctypes.c_uint32, P]
    lib.lda_draw_butterfly_philox.restype = ctypes.c_int
    lib.lda_philox_uniforms.argtypes = [P, I64, I64, ctypes.c_uint64, ctypes.c_uint32, P]
    lib.lda_philox_uniforms.restype = ctypes.c_int
    lib.lda_draw_docs.argtypes = draw_args
    lib.lda_draw_docs.restype = ctypes.c_int
    lib.lda_draw_doc_lanes.argtypes = draw_args[:-1] + [I32, P]
    lib.lda_draw_doc_lanes.restype = ctypes.c_int
    lib.lda_butterfly_table.argtypes = [P, P, P, P, P, I64, I32, I32, I32, P]
    lib.lda_butterfly_table.restype = ctypes.c_int
    lib.lda_butterfly_width.argtypes = [I32]
    lib.lda_butterfly_width.restype = ctypes.c_int
    lib.lda_status_string.argtypes = [ctypes.c_int]
    lib.lda_status_string.restype = ctypes.c_char_p
    lib.lda_last_hip_error.restype = ctypes.c_char_p
    lib.lda_version.restype = ctypes.c_int
    lib.lda_route_workspace_bytes.argtypes = [I64]
    lib.lda_route_workspace_bytes.restype = ctypes.c_size_t
    lib.lda_route_build.argtypes = [P, P, I64, I32, I32, P, ctypes.c_size_t,
                                    ctypes.POINTER(RouteInfo), P]
    lib.lda_route_build.restype = ctypes.c_int
    lib.lda_draw_routed.argtypes = [P, P, P, ctypes.c_size_t, ctypes.POINTER(RouteInfo), P, P,
                                    I64, I32, I32, I32, P]
    lib.lda_draw_routed.restype = ctypes.c_int
    lib.lda_draw_routed_philox.argtypes = [P, P, P, ctypes.c_size_t, ctypes.POINTER(RouteInfo),
                                           P, I64, I32, I32, I32, ctypes.c_uint64,
                                           ctypes.c_uint32, P]
    lib.lda_draw_routed_philox.restype = ctypes.c_int
    lib.lda_draw_routed_scratch.argtypes = draw_args
    lib.lda_draw_routed_scratch.restype = ctypes.c_int
    lib.lda_count_topics.argtypes = [P, P, P, I64, I32, I32, I32, P, P, P]
    lib.lda_count_topics.restype = ctypes.c_int
    lib.lda_count_topics_docs.argtypes = [P, P, P, I64, I32, I32, I32, P, P, P]
    lib.lda_count_topics_docs.restype = ctypes.c_int
    lib.lda_word_index_bytes.argtypes = [I64, I32]
    lib.lda_word_index_bytes.restype = ctypes.c_size_t
    lib.lda_word_index_build.argtypes = [P, I64, I32, P, ctypes.c_size_t, P]
    lib.lda_word_index_build.restype = ctypes.c_int
    lib.lda_count_topics_indexed.argtypes = [P, P, P, I64, I32, I32, I32, P, ctypes.c_size_t,
                                             P, P, P]
    lib.lda_count_topics_indexed.restype = ctypes.c_int
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load().lda_status_string(status).decode()


def _check(status: int) -> None:
    if status != 0:
        msg = status_string(status)
        if status == STATUS["LDA_ERR_HIP"]:
            msg += ": " + load().lda_last_hip_error().decode()
        raise LdaError(status, msg)


def _stream_handle(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream)


def _require(t: torch.Tensor, name: str, dtype, ndim: int) -> None:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be on the GPU")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dimension(s)")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _shapes(theta, phi, doc_id, word_id, u=None):
    _require(theta, "theta", torch.float32, 2)
    _require(phi, "phi", torch.float32, 2)
    _require(doc_id, "doc_id", torch.int32, 1)
    _require(word_id, "word_id", torch.int32, 1)
    M, K = theta.shape
    V, K2 = phi.shape
    N = doc_id.shape[0]
    if K2 != K:
        raise ValueError(f"theta has K={K} topics but phi has {K2}")
    if word_id.shape[0] != N:
        raise ValueError("doc_id and word_id lengths differ")
    if u is not None:
        _require(u, "u", torch.float32, 1)
        if u.shape[0] != N:
            raise ValueError("u and doc_id lengths differ")
    devs = {t.device for t in (theta, phi, doc_id, word_id) + ((u,) if u is not None else ())}
    if len(devs) != 1:
        raise ValueError("all tensors must be on one device")
    return N, M, V, K


def _validate_ids(doc_id, word_id, M, V) -> None:
    if doc_id.numel():
        if int(doc_id.min()) < 0 or int(doc_id.max()) >= M:
            raise ValueError("doc_id out of range [0, M)")
        if int(word_id.min()) < 0 or int(word_id.max()) >= V:
            raise ValueError("word_id out of range [0, V)")


def _draw(fn_name, theta, phi, doc_id, word_id, u, out, stream, validate, extra=()):
    N, M, V, K = _shapes(theta, phi, doc_id, word_id, u)
    if validate:
        _validate_ids(doc_id, word_id, M, V)
    if out is None:
        out = torch.empty(N, dtype=torch.int32, device=doc_id.device)
    else:
        _require(out, "out", torch.int32, 1)
        if out.shape[0] != N or out.device != doc_id.device:
            raise ValueError("out must be int32[N] on the tensors' device")
    with torch.cuda.device(doc_id.device):
        st = getattr(load(), fn_name)(
            theta.data_ptr(), phi.data_ptr(), doc_id.data_ptr(),
            word_id.data_ptr(), u.data_ptr(), out.data_ptr(), N, M, V, K,
            *extra, _stream_handle(stream))
    _check(st)
    return out


def draw_naive(theta, phi, doc_id, word_id, u, out=None, stream=None,
               validate: bool = False) -> torch.Tensor:
    """z[N] (int32) by the one-lane-per-token kernel (Algorithms 1 + 3)."""
    return _draw("lda_draw_naive", theta, phi, doc_id, word_id, u, out,
                 stream, validate)


def draw_butterfly(theta, phi, doc_id, word_id, u, out=None, stream=None,
                   validate: bool = False) -> torch.Tensor:
    """z[N] (int32) by the butterfly kernel (Algorithms 7-10)."""
    return _draw("lda_draw_butterfly", theta, phi, doc_id, word_id, u, out,
                 stream, validate)


def draw_transposed(theta, phi, doc_id, word_id, u, out=None, stream=None,
                    validate: bool = False) -> torch.Tensor:
    """z[N] (int32) by the transposed-access kernel (Algorithms 4-6), the
    paper's design before the butterfly, for comparison."""
    return _draw("lda_draw_transposed", theta, phi, doc_id, word_id, u, out,
                 stream, validate)


def draw_variant(theta, phi, doc_id, word_id, u, variant: str = "register",
                 out=None, stream=None, validate: bool = False) -> torch.Tensor:
    """z[N] (int32) by a variant of the butterfly draw: the one-topic-per-lane
    kernel with a chosen block table, "register" (the paper's rule,
    search-assist loop), "lds" (the same table in LDS) or "lds_alt" (the
    alternative rule [a b; c d] -> [a c; a+b c+d], Section 4); "leaf8",
    the default kernels with 8-topic leaves in the leaf groups; or "wide",
    the default kernels as built for tables past 4 GiB (the same draws)."""
    if variant not in VARIANTS:
        raise ValueError(f"variant must be one of {sorted(VARIANTS)}")
    return _draw("lda_draw_butterfly_variant", theta, phi, doc_id, word_id, u,
                 out, stream, validate, extra=(VARIANTS[variant],))


def draw_philox(theta, phi, doc_id, word_id, seed: int, sweep: int = 0, out=None,
                stream=None, validate: bool = False) -> torch.Tensor:
    """z[N] (int32) by the butterfly kernel with the uniforms generated in the
    kernel (Philox4x32-10 of token index, sweep and seed; see
    ``philox_uniforms``)."""
    N, M, V, K = _shapes(theta, phi, doc_id, word_id)
    if validate:
        _validate_ids(doc_id, word_id, M, V)
    if out is None:
        out = torch.empty(N, dtype=torch.int32, device=doc_id.device)
    else:
        _require(out, "out", torch.int32, 1)
        if out.shape[0] != N or out.device != doc_id.device:
            raise ValueError("out must be int32[N] on the tensors' device")
    with torch.cuda.device(doc_id.device):
        st = load().lda_draw_butterfly_philox(
            theta.data_ptr(), phi.data_ptr(), doc_id.data_ptr(), word_id.data_ptr(),
            out.data_ptr(), N, M, V, K, int(seed) & (2 ** 64 - 1),
            int(sweep) & (2 ** 32 - 1), _stream_handle(stream))
    _check(st)
    return out


def philox_uniforms(count: int, seed: int, sweep: int = 0, first: int = 0, out=None,
                    device="cuda", stream=None) -> torch.Tensor:
    """The uniforms of tokens first .. first + count - 1 that ``draw_philox``
    uses (float32 [count] on the GPU)."""
    if out is None:
        out = torch.empty(int(count), dtype=torch.float32, device=device)
    else:
        _require(out, "out", torch.float32, 1)
        if out.shape[0] != count:
            raise ValueError("out must be float32[count]")
    with torch.cuda.device(out.device):
        st = load().lda_philox_uniforms(out.data_ptr(), int(count), int(first),
                                        int(seed) & (2 ** 64 - 1),
                                        int(sweep) & (2 ** 32 - 1), _stream_handle(stream))
    _check(st)
    return out


def draw_docs(theta, phi, doc_offsets, word_id, u, out=None, stream=None,
              validate: bool = False) -> torch.Tensor:
    """z[N] (int32) by the butterfly kernel, documents given as offsets:
    document m holds tokens doc_offsets[m] .. doc_offsets[m+1]-1 (int64
    [M+1], doc_offsets[0] = 0, doc_offsets[M] = N, non-decreasing; empty
    documents allowed), the paper's ragged corpus of Section 2."""
    return _draw_offsets("lda_draw_docs", theta, phi, doc_offsets, word_id, u,
                         out, stream, validate)


def draw_doc_lanes(theta, phi, doc_offsets, word_id, u, theta_cache: bool = False,
                   out=None, stream=None, validate: bool = False) -> torch.Tensor:
    """z[N] (int32) by the paper's document-per-lane driver (Algorithm 7:
    one document per lane, a master index over their tokens); arguments as
    ``draw_docs``.  ``theta_cache``: copy each wavefront's theta rows to LDS
    first (Algorithm 5; K <= 256)."""
    return _draw_offsets("lda_draw_doc_lanes", theta, phi, doc_offsets, word_id,
                         u, out, stream, validate, extra=(int(bool(theta_cache)),))


def _draw_offsets(fn_name, theta, phi, doc_offsets, word_id, u, out, stream, validate,
                  extra=()):
    _require(theta, "theta", torch.float32, 2)
    _require(phi, "phi", torch.float32, 2)
    _require(doc_offsets, "doc_offsets", torch.int64, 1)
    _require(word_id, "word_id", torch.int32, 1)
    _require(u, "u", torch.float32, 1)
    M, K = theta.shape
    V, K2 = phi.shape
    N = word_id.shape[0]
    if K2 != K:
        raise ValueError(f"theta has K={K} topics but phi has {K2}")
    if doc_offsets.shape[0] != M + 1:
        raise ValueError("doc_offsets must have M + 1 entries")
    if u.shape[0] != N:
        raise ValueError("u and word_id lengths differ")
    devs = {t.device for t in (theta, phi, doc_offsets, word_id, u)}
    if len(devs) != 1:
        raise ValueError("all tensors must be on one device")
    if validate:
        off = doc_offsets.cpu()
        if int(off[0]) != 0 or int(off[-1]) != N or bool((off[1:] < off[:-1]).any()):
            raise ValueError("doc_offsets must rise from 0 to N")
        if N and (int(word_id.min()) < 0 or int(word_id.max()) >= V):
            raise ValueError("word_id out of range [0, V)")
    if out is None:
        out = torch.empty(N, dtype=torch.int32, device=word_id.device)
    else:
        _require(out, "out", torch.int32, 1)
        if out.shape[0] != N or out.device != word_id.device:
            raise ValueError("out must be int32[N] on the tensors' device")
    with torch.cuda.device(word_id.device):
        st = getattr(load(), fn_name)(
            theta.data_ptr(), phi.data_ptr(), doc_offsets.data_ptr(),
            word_id.data_ptr(), u.data_ptr(), out.data_ptr(), N, M, V, K,
            *extra, _stream_handle(stream))
    _check(st)
    return out


def butterfly_table(theta, phi, doc_id, word_id, out=None, stream=None,
                    validate: bool = False) -> torch.Tensor:
    """The per-lane butterfly tables, float32 [N][K] (Fig. 1, right)."""
    N, M, V, K = _shapes(theta, phi, doc_id, word_id)
    if validate:
        _validate_ids(doc_id, word_id, M, V)
    if out is None:
        out = torch.empty((N, K), dtype=torch.float32, device=doc_id.device)
    else:
        _require(out, "out", torch.float32, 2)
        if tuple(out.shape) != (N, K) or out.device != doc_id.device:
            raise ValueError("out must be float32[N][K] on the tensors' device")
    with torch.cuda.device(doc_id.device):
        st = load().lda_butterfly_table(
            theta.data_ptr(), phi.data_ptr(), doc_id.data_ptr(),
            word_id.data_ptr(), out.data_ptr(), N, M, V, K,
            _stream_handle(stream))
    _check(st)
    return out


def count_topics(doc_id, word_id, z, M: int, V: int, K: int, ndk=None, nwk=None,
                 stream=None) -> tuple[torch.Tensor, torch.Tensor]:
    """(ndk int32 [M][K], nwk int32 [V][K]): the tokens of each document, and
    of each word, drawn to each topic (lda_count_topics).  ``ndk`` / ``nwk``:
    optional outputs to overwrite."""
    _require(doc_id, "doc_id", torch.int32, 1)
    _require(word_id, "word_id", torch.int32, 1)
    _require(z, "z", torch.int32, 1)
    N = doc_id.shape[0]
    if word_id.shape[0] != N or z.shape[0] != N:
        raise ValueError("doc_id, word_id and z lengths differ")
    dev = doc_id.device
    if word_id.device != dev or z.device != dev:
        raise ValueError("all tensors must be on one device")
    outs = []
    for t, name, rows in ((ndk, "ndk", M), (nwk, "nwk", V)):
        if t is None:
            t = torch.empty((rows, K), dtype=torch.int32, device=dev)
        else:
            _require(t, name, torch.int32, 2)
            if tuple(t.shape) != (rows, K) or t.device != dev:
                raise ValueError(f"{name} must be int32[{rows}][{K}] on the tokens' device")
        outs.append(t)
    with torch.cuda.device(dev):
        st = load().lda_count_topics(doc_id.data_ptr(), word_id.data_ptr(), z.data_ptr(), N,
                                     int(M), int(V), int(K), outs[0].data_ptr(),
                                     outs[1].data_ptr(), _stream_handle(stream))
    _check(st)
    return outs[0], outs[1]


def count_topics_docs(doc_offsets, word_id, z, V: int, K: int, ndk=None, nwk=None,
                      stream=None, validate: bool = False) -> tuple[torch.Tensor, torch.Tensor]:
    """count_topics with the documents as offsets (int64 [M + 1]; document m =
    tokens doc_offsets[m] .. doc_offsets[m+1] - 1), as draw_docs takes them
    (lda_count_topics_docs)."""
    _require(doc_offsets, "doc_offsets", torch.int64, 1)
    _require(word_id, "word_id", torch.int32, 1)
    _require(z, "z", torch.int32, 1)
    N = word_id.shape[0]
    M = doc_offsets.shape[0] - 1
    if M < 1:
        raise ValueError("doc_offsets must hold M + 1 >= 2 entries")
    if z.shape[0] != N:
        raise ValueError("word_id and z lengths differ")
    dev = word_id.device
    if z.device != dev or doc_offsets.device != dev:
        raise ValueError("all tensors must be on one device")
    if validate:
        off = doc_offsets.cpu()
        if int(off[0]) != 0 or int(off[-1]) != N or bool((off[1:] < off[:-1]).any()):
            raise ValueError("doc_offsets must be non-decreasing from 0 to N")
    outs = []
    for t, name, rows in ((ndk, "ndk", M), (nwk, "nwk", V)):
        if t is None:
            t = torch.empty((rows, K), dtype=torch.int32, device=dev)
        else:
            _require(t, name, torch.int32, 2)
            if tuple(t.shape) != (rows, K) or t.device != dev:
                raise ValueError(f"{name} must be int32[{rows}][{K}] on the tokens' device")
        outs.append(t)
    with torch.cuda.device(dev):
        st = load().lda_count_topics_docs(doc_offsets.data_ptr(), word_id.data_ptr(),
                                          z.data_ptr(), N, int(M), int(V), int(K),
                                          outs[0].data_ptr(), outs[1].data_ptr(),
                                          _stream_handle(stream))
    _check(st)
    return outs[0], outs[1]


class WordIndex:
    """The tokens grouped by word (lda_word_index_build): a uint8 device
    workspace holding off [V + 1], perm [N] and wsorted [N], for N tokens and
    V words."""

    def __init__(self, workspace: torch.Tensor, N: int, V: int):
        self.workspace, self.N, self.V = workspace, N, V

    def arrays(self) -> dict[str, torch.Tensor]:
        """Views of off (int32 [V + 1]), perm and wsorted (int32 [N])."""
        lay = word_index_layout(self.N, self.V)
        return {"off": self.workspace[lay["off"]:lay["off"] + 4 * (self.V + 1)].view(torch.int32),
                "perm": self.workspace[lay["perm"]:lay["perm"] + 4 * self.N].view(torch.int32),
                "wsorted": self.workspace[lay["wsorted"]:lay["wsorted"] + 4 * self.N]
                .view(torch.int32)}


def word_index_bytes(N: int, V: int) -> int:
    """Bytes of device workspace ``word_index_build`` needs (0: unsupported)."""
    return int(load().lda_word_index_bytes(int(N), int(V)))


def word_index_layout(N: int, V: int) -> dict[str, int]:
    """Byte offsets of the index's sections (the layout the header states)."""
    def up(b):
        return (b + 255) & ~255
    lay, at = {}, 0
    for name, b in (("off", 4 * (V + 1)), ("cursor", 4 * V * 16), ("sums", 4 * 4096),
                    ("perm", 4 * max(N, 1)), ("wsorted", 4 * max(N, 1))):
        lay[name] = at
        at += up(b)
    lay["bytes"] = at
    return lay


def word_index_build(word_id, V: int, workspace=None, stream=None) -> WordIndex:
    """Group the tokens (word_id: int32 [N] on the GPU) by word, once per
    corpus (lda_word_index_build).  ``workspace``: a uint8 tensor of at least
    ``word_index_bytes(N, V)`` bytes on the same GPU, or None to allocate one."""
    _require(word_id, "word_id", torch.int32, 1)
    N = word_id.shape[0]
    need = word_index_bytes(N, V)
    if need == 0:
        raise LdaError(STATUS["LDA_ERR_UNSUPPORTED"], status_string(STATUS["LDA_ERR_UNSUPPORTED"]))
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=word_id.device)
    else:
        _require(workspace, "workspace", torch.uint8, 1)
        if workspace.device != word_id.device:
            raise ValueError("workspace must be on word_id's device")
    with torch.cuda.device(word_id.device):
        st = load().lda_word_index_build(word_id.data_ptr(), N, int(V), workspace.data_ptr(),
                                         workspace.numel(), _stream_handle(stream))
    _check(st)
    return WordIndex(workspace, N, int(V))


def count_topics_indexed(doc_offsets, word_id, z, index: WordIndex, K: int, ndk=None, nwk=None,
                         stream=None) -> tuple[torch.Tensor, torch.Tensor]:
    """count_topics_docs with the word table counted from ``index``
    (word_index_build over the same word_id): lda_count_topics_indexed."""
    _require(doc_offsets, "doc_offsets", torch.int64, 1)
    _require(word_id, "word_id", torch.int32, 1)
    _require(z, "z", torch.int32, 1)
    N, V = word_id.shape[0], index.V
    M = doc_offsets.shape[0] - 1
    if M < 1:
        raise ValueError("doc_offsets must hold M + 1 >= 2 entries")
    if z.shape[0] != N or index.N != N:
        raise ValueError("word_id, z and the index must cover the same N tokens")
    dev = word_id.device
    if z.device != dev or doc_offsets.device != dev or index.workspace.device != dev:
        raise ValueError("all tensors must be on one device")
    outs = []
    for t, name, rows in ((ndk, "ndk", M), (nwk, "nwk", V)):
        if t is None:
            t = torch.empty((rows, K), dtype=torch.int32, device=dev)
        else:
            _require(t, name, torch.int32, 2)
            if tuple(t.shape) != (rows, K) or t.device != dev:
                raise ValueError(f"{name} must be int32[{rows}][{K}] on the tokens' device")
        outs.append(t)
    with torch.cuda.device(dev):
        st = load().lda_count_topics_indexed(doc_offsets.data_ptr(), word_id.data_ptr(),
                                             z.data_ptr(), N, int(M), int(V), int(K),
                                             index.workspace.data_ptr(), index.workspace.numel(),
                                             outs[0].data_ptr(), outs[1].data_ptr(),
                                             _stream_handle(stream))
    _check(st)
    return outs[0], outs[1]


def butterfly_width(K: int) -> int:
    w = load().lda_butterfly_width(int(K))
    _check(min(w, 0))
    return w


def version() -> int:
    return int(load().lda_version())


def route_workspace_bytes(N: int) -> int:
    """Bytes of device workspace ``route_build`` needs for N tokens."""
    return int(load().lda_route_workspace_bytes(int(N)))


def route_layout(N: int) -> dict[str, int]:
    """Byte offsets of the routing's sections in the workspace (the library's
    layout: perm, rword, rdoc int32 [N + 512] each, then the builder's
    tables, every section starting on a 256-byte boundary) and its size."""
    Np = N + 8 * 64
    nchunks = (N + 4095) // 4096
    off, out = 0, {}
    for name, nbytes in (("perm", 4 * Np), ("rword", 4 * Np), ("rdoc", 4 * Np),
                         ("chunk_off", 32 * nchunks), ("counts", 1024), ("map", 1024),
                         ("lists", 192), ("chunk_hist", 1024 * nchunks)):
        out[name] = off
        off += (nbytes + 255) & ~255
    out["bytes"] = off
    return out


class Route:
    """Tokens routed to the GPU's XCDs by word (``route_build``): the device
    workspace that holds the routing and the host copy of the list sizes.
    It belongs to one corpus (its doc and word ids) and can be reused by
    every ``draw_routed`` over that corpus."""

    def __init__(self, workspace: torch.Tensor, info: RouteInfo, M: int, V: int):
        self.workspace = workspace
        self.info = info
        self.M, self.V = M, V

    @property
    def N(self) -> int:
        return int(self.info.N)

    @property
    def tokens(self) -> list[int]:
        return list(self.info.tokens)

    @property
    def start(self) -> list[int]:
        return list(self.info.start)

    @property
    def length(self) -> list[int]:
        return list(self.info.length)

    def arrays(self) -> dict[str, torch.Tensor]:
        """Views of the routed arrays in the workspace: perm (token at each
        routed position, -1 for padding), rword and rdoc (its word and
        document), int32 [N + 512] each (positions past the lists unused)."""
        lay = route_layout(self.N)
        n = self.N + 8 * 64
        return {k: self.workspace[lay[k]:lay[k] + 4 * n].view(torch.int32)
                for k in ("perm", "rword", "rdoc")}


def route_build(doc_id, word_id, M: int, V: int, workspace=None, stream=None,
                validate: bool = False) -> Route:
    """Route the tokens (doc_id, word_id: int32 [N] on the GPU) to the eight
    XCDs by word.  ``workspace``: a uint8 tensor of at least
    ``route_workspace_bytes(N)`` bytes on the same GPU, or None to allocate
    one.  Synchronises ``stream`` once (to read back the word class counts);
    a draw on the same stream follows the rest of the build."""
    _require(doc_id, "doc_id", torch.int32, 1)
    _require(word_id, "word_id", torch.int32, 1)
    N = doc_id.shape[0]
    if word_id.shape[0] != N or word_id.device != doc_id.device:
        raise ValueError("doc_id and word_id must have one length and device")
    if validate:
        _validate_ids(doc_id, word_id, M, V)
    need = route_workspace_bytes(N)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=doc_id.device)
    else:
        _require(workspace, "workspace", torch.uint8, 1)
        if workspace.device != doc_id.device:
            raise ValueError("workspace must be on the tensors' device")
    info = RouteInfo()
    with torch.cuda.device(doc_id.device):
        st = load().lda_route_build(doc_id.data_ptr(), word_id.data_ptr(), N, int(M), int(V),
                                    workspace.data_ptr(), workspace.numel(),
                                    ctypes.byref(info), _stream_handle(stream))
    _check(st)
    return Route(workspace, info, int(M), int(V))


def _routed_args(theta, phi, route: "Route", N: int, device, out):
    _require(theta, "theta", torch.float32, 2)
    _require(phi, "phi", torch.float32, 2)
    M, K = theta.shape
    V, K2 = phi.shape
    if K2 != K:
        raise ValueError(f"theta has K={K} topics but phi has {K2}")
    if (M, V, N) != (route.M, route.V, route.N):
        raise ValueError("theta, phi and u do not match the routed corpus")
    devs = {t.device for t in (theta, phi, route.workspace)} | {device}
    if len(devs) != 1:
        raise ValueError("all tensors must be on one device")
    if out is None:
        out = torch.empty(N, dtype=torch.int32, device=device)
    else:
        _require(out, "out", torch.int32, 1)
        if out.shape[0] != N or out.device != device:
            raise ValueError("out must be int32[N] on the tensors' device")
    return M, V, K, out


def draw_routed_scratch(theta, phi, doc_id, word_id, u, out=None, stream=None,
                        validate: bool = False) -> torch.Tensor:
    """The routed draw with the routing built in the library's own scratch
    array (lda_draw_routed_scratch): no workspace, nothing allocated by the
    library; waits on the stream once; N up to about 5.4M tokens."""
    return _draw("lda_draw_routed_scratch", theta, phi, doc_id, word_id, u, out, stream,
                 validate)


def draw_routed(theta, phi, route: Route, u, out=None, stream=None) -> torch.Tensor:
    """z[N] (int32, indexed by the original token) by the leaf kernel over the
    routed tokens; u float32 [N] indexed by the original token.  K must be
    divisible by 4 with 132 <= K <= 2048."""
    _require(u, "u", torch.float32, 1)
    N = u.shape[0]
    M, V, K, out = _routed_args(theta, phi, route, N, u.device, out)
    with torch.cuda.device(u.device):
        st = load().lda_draw_routed(theta.data_ptr(), phi.data_ptr(), route.workspace.data_ptr(),
                                    route.workspace.numel(), ctypes.byref(route.info),
                                    u.data_ptr(), out.data_ptr(), N, M, V, K,
                                    _stream_handle(stream))
    _check(st)
    return out


def draw_routed_philox(theta, phi, route: Route, seed: int, sweep: int = 0, out=None,
                       stream=None) -> torch.Tensor:
    """``draw_routed`` with the uniforms of ``draw_philox`` (generated in the
    kernel from the original token index, sweep and seed)."""
    N = route.N
    M, V, K, out = _routed_args(theta, phi, route, N, route.workspace.device, out)
    with torch.cuda.device(route.workspace.device):
        st = load().lda_draw_routed_philox(
            theta.data_ptr(), phi.data_ptr(), route.workspace.data_ptr(),
            route.workspace.numel(), ctypes.byref(route.info), out.data_ptr(), N, M, V, K,
            int(seed) & (2 ** 64 - 1), int(sweep) & (2 ** 32 - 1), _stream_handle(stream))
    _check(st)
    return out
