"""The C ABI on the CPU: the library loads, exports every function the header
declares, and rejects bad arguments before touching HIP (no kernel is
launched by these tests)."""
import ctypes
import os
import re
import subprocess

import pytest

from conftest import ROOT

HEADER_DIR = os.path.join(ROOT, "include")


# each header and the library that must export what it declares
HEADER_LIBS = {"lda_draw.h": "liblda_draw.so", "lda_probe.h": "liblda_probe.so"}


def declared_functions(header=None):
    names = []
    for fn in sorted(os.listdir(HEADER_DIR)):
        if fn.endswith(".h") and (header is None or fn == header):
            src = open(os.path.join(HEADER_DIR, fn)).read()
            src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
            names += re.findall(r"^[A-Za-z_][\w\s\*]*?\b(lda_\w+)\s*\(", src,
                                flags=re.M)
    return names


@pytest.fixture(scope="module")
def lib():
    from paper_1505_03851_amd import _lib
    return _lib.load()


def test_header_declares_the_boundary():
    names = declared_functions()
    for must in ("lda_draw_naive", "lda_draw_butterfly", "lda_status_string"):
        assert must in names


def test_every_header_has_its_library():
    assert sorted(f for f in os.listdir(HEADER_DIR) if f.endswith(".h")) == sorted(HEADER_LIBS)


@pytest.mark.parametrize("header", sorted(HEADER_LIBS))
def test_every_declared_symbol_is_exported(header):
    from paper_1505_03851_amd import _lib, probe
    loaded = {"lda_draw.h": _lib.load, "lda_probe.h": probe.load}[header]()
    path = os.path.join(ROOT, "paper_1505_03851_amd", HEADER_LIBS[header])
    out = subprocess.run(["nm", "-D", "--defined-only", path],
                         capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\bT\s+(\w+)$", out, flags=re.M))
    names = declared_functions(header)
    assert names
    for name in names:
        assert name in exported, name
        assert getattr(loaded, name) is not None


def test_status_strings(lib):
    from paper_1505_03851_amd import _lib
    seen = set()
    for k, v in _lib.STATUS.items():
        s = lib.lda_status_string(v).decode()
        assert s and s != "unknown status"
        seen.add(s)
    assert len(seen) == len(_lib.STATUS)
    assert lib.lda_status_string(12345).decode() == "unknown status"
    assert lib.lda_version() >= 100


# Fake, aligned, non-null addresses: every call below must be rejected (or be
# a no-op) by the host-side checks, so none of them is dereferenced.
A = 4096


def call(lib, fn, **kw):
    args = dict(theta=A, phi=A, doc=A, word=A, u=A, z=A, N=10, M=3, V=5, K=8)
    args.update(kw)
    f = getattr(lib, fn)
    if fn == "lda_draw_butterfly_variant":
        return f(args["theta"], args["phi"], args["doc"], args["word"], args["u"],
                 args["z"], args["N"], args["M"], args["V"], args["K"],
                 args.get("variant", 2), None)
    if fn == "lda_draw_doc_lanes":
        return f(args["theta"], args["phi"], args["doc"], args["word"], args["u"],
                 args["z"], args["N"], args["M"], args["V"], args["K"],
                 args.get("theta_cache", 0), None)
    if fn == "lda_butterfly_table":
        return f(args["theta"], args["phi"], args["doc"], args["word"],
                 args["z"], args["N"], args["M"], args["V"], args["K"], None)
    return f(args["theta"], args["phi"], args["doc"], args["word"], args["u"],
             args["z"], args["N"], args["M"], args["V"], args["K"], None)


FNS = ["lda_draw_naive", "lda_draw_butterfly", "lda_draw_transposed", "lda_draw_docs",
       "lda_draw_doc_lanes", "lda_draw_butterfly_variant", "lda_butterfly_table"]
# entry points that take tables of any size (past LDA_MAX_TABLE_BYTES with the
# wide build)
WIDE_FNS = ("lda_draw_butterfly", "lda_draw_docs")


@pytest.mark.parametrize("fn", FNS)
def test_shape_errors(lib, fn):
    from paper_1505_03851_amd._lib import STATUS
    for kw in (dict(N=-1), dict(M=0), dict(V=0), dict(K=0), dict(K=-5),
               dict(M=-1)):
        assert call(lib, fn, **kw) == STATUS["LDA_ERR_SHAPE"], kw
    from paper_1505_03851_amd._lib import MAX_K, MAX_TABLE_BYTES
    assert call(lib, fn, K=MAX_K + 1) == STATUS["LDA_ERR_UNSUPPORTED"]
    # token counts past what one dispatch can hold
    from paper_1505_03851_amd._lib import MAX_N
    assert MAX_N >= 2 ** 32 - 2 ** 16
    assert call(lib, fn, N=MAX_N + 1) == STATUS["LDA_ERR_UNSUPPORTED"]
    assert call(lib, fn, N=2 ** 40) == STATUS["LDA_ERR_UNSUPPORTED"]
    # tables past the buffer resources' byte limit are rejected before any
    # HIP call, except by the entry points that take any size; every call
    # that is accepted here has N = 0, so it launches nothing and the fake
    # addresses are never read
    past_4_gib = MAX_TABLE_BYTES // (4 * 1024) + 1
    if fn in WIDE_FNS:
        for kw in (dict(V=past_4_gib), dict(M=past_4_gib), dict(V=2 ** 31 - 1),
                   dict(M=2 ** 31 - 1, V=2 ** 31 - 1)):
            assert call(lib, fn, K=1024, N=0, **kw) == 0, kw
    else:
        assert call(lib, fn, K=1024, V=past_4_gib) == STATUS["LDA_ERR_UNSUPPORTED"]
        assert call(lib, fn, K=1024, M=past_4_gib) == STATUS["LDA_ERR_UNSUPPORTED"]
        assert call(lib, fn, K=1024, V=past_4_gib - 1, M=past_4_gib - 1, N=0) == 0


@pytest.mark.parametrize("fn", FNS)
def test_null_and_alignment_errors(lib, fn):
    from paper_1505_03851_amd._lib import STATUS
    keys = ["theta", "phi", "doc", "word", "z"] + (["u"] if fn != "lda_butterfly_table" else [])
    for key in keys:
        assert call(lib, fn, **{key: None}) == STATUS["LDA_ERR_NULL"], key
        assert call(lib, fn, **{key: A + 2}) == STATUS["LDA_ERR_ALIGN"], key


@pytest.mark.parametrize("fn", FNS)
def test_empty_is_noop(lib, fn):
    # N = 0: no launch, no pointer needed
    assert call(lib, fn, N=0, theta=None, phi=None, doc=None, word=None,
                u=None, z=None) == 0


def test_variant_codes(lib):
    from paper_1505_03851_amd._lib import STATUS, VARIANTS
    assert sorted(VARIANTS.values()) == [0, 1, 2, 3, 4]
    for bad in (-1, 5, 99):
        assert call(lib, "lda_draw_butterfly_variant", variant=bad) == \
            STATUS["LDA_ERR_UNSUPPORTED"]
    # a known variant still goes through the argument checks
    assert call(lib, "lda_draw_butterfly_variant", variant=0, K=0) == STATUS["LDA_ERR_SHAPE"]
    # the wide build takes tables past 4 GiB; the others do not (N = 0: no launch)
    from paper_1505_03851_amd._lib import MAX_TABLE_BYTES
    past = MAX_TABLE_BYTES // (4 * 1024) + 1
    for name, code in VARIANTS.items():
        want = 0 if name == "wide" else STATUS["LDA_ERR_UNSUPPORTED"]
        assert call(lib, "lda_draw_butterfly_variant", variant=code, K=1024, V=past, N=0) == \
            want, name


def test_doc_lanes_theta_cache_limits(lib):
    from paper_1505_03851_amd._lib import DOC_LANES_MAX_CACHE_BYTES, STATUS
    fn = "lda_draw_doc_lanes"
    for bad in (-1, 2):
        assert call(lib, fn, theta_cache=bad) == STATUS["LDA_ERR_UNSUPPORTED"]
    # the cache holds K rounded up to 64-topic blocks, 64 lanes x 4 bytes each
    kmax = DOC_LANES_MAX_CACHE_BYTES // 256
    assert kmax == 256
    assert call(lib, fn, theta_cache=1, K=kmax + 1, N=0) == STATUS["LDA_ERR_UNSUPPORTED"]
    assert call(lib, fn, theta_cache=1, K=kmax, N=0) == 0
    assert call(lib, fn, theta_cache=0, K=4096, N=0) == 0


def test_docs_offsets_need_8_byte_alignment(lib):
    # doc_offsets is int64: 4-byte aligned is not enough
    from paper_1505_03851_amd._lib import STATUS
    for fn in ("lda_draw_docs", "lda_draw_doc_lanes"):
        assert call(lib, fn, doc=A + 4) == STATUS["LDA_ERR_ALIGN"]


def test_width(lib):
    from paper_1505_03851_amd._lib import MAX_K, STATUS
    assert lib.lda_butterfly_width(1) == 32
    assert lib.lda_butterfly_width(63) == 32
    assert lib.lda_butterfly_width(64) == 64
    assert lib.lda_butterfly_width(MAX_K) == 64
    assert lib.lda_butterfly_width(0) == STATUS["LDA_ERR_SHAPE"]
    assert lib.lda_butterfly_width(MAX_K + 1) == STATUS["LDA_ERR_UNSUPPORTED"]


def test_binding_rejects_cpu_tensors():
    import torch
    import paper_1505_03851_amd as lda
    t = torch.zeros((2, 4))
    i = torch.zeros(3, dtype=torch.int32)
    with pytest.raises(ValueError):
        lda.draw_butterfly(t, t, i, i, torch.zeros(3))


def test_philox_draw_argument_errors(lib):
    from paper_1505_03851_amd._lib import STATUS
    f = lib.lda_draw_butterfly_philox
    ok = dict(theta=A, phi=A, doc=A, word=A, z=A, N=10, M=3, V=5, K=8)

    def run(**kw):
        a = dict(ok, **kw)
        return f(a["theta"], a["phi"], a["doc"], a["word"], a["z"], a["N"], a["M"],
                 a["V"], a["K"], 123, 0, None)
    for key in ("theta", "phi", "doc", "word", "z"):
        assert run(**{key: None}) == STATUS["LDA_ERR_NULL"], key
        assert run(**{key: A + 2}) == STATUS["LDA_ERR_ALIGN"], key
    for kw in (dict(N=-1), dict(M=0), dict(V=0), dict(K=0)):
        assert run(**kw) == STATUS["LDA_ERR_SHAPE"], kw
    assert run(N=0, theta=None, phi=None, doc=None, word=None, z=None) == 0
    # tables of any size (N = 0: nothing is launched)
    from paper_1505_03851_amd._lib import MAX_TABLE_BYTES
    assert run(K=1024, V=MAX_TABLE_BYTES // 4096 + 1, M=2 ** 31 - 1, N=0) == 0


def test_philox_uniforms_argument_errors(lib):
    from paper_1505_03851_amd._lib import STATUS
    f = lib.lda_philox_uniforms
    assert f(None, 0, 0, 1, 0, None) == 0                     # no-op
    assert f(A, -1, 0, 1, 0, None) == STATUS["LDA_ERR_SHAPE"]
    assert f(A, 5, -1, 1, 0, None) == STATUS["LDA_ERR_SHAPE"]
    assert f(A, 2, 2 ** 63 - 1, 1, 0, None) == STATUS["LDA_ERR_SHAPE"]
    assert f(A, 301, 2 ** 63 - 301, 1, 0, None) == STATUS["LDA_ERR_SHAPE"]  # first + count = 2^63
    assert f(None, 5, 0, 1, 0, None) == STATUS["LDA_ERR_NULL"]
    assert f(A + 1, 5, 0, 1, 0, None) == STATUS["LDA_ERR_ALIGN"]


# ---------------------------------------------------------------------------
# Routing of tokens to the XCDs: argument checks (before any HIP call) and the
# workspace size.

def test_route_workspace_bytes(lib):
    from paper_1505_03851_amd import _lib
    f = lib.lda_route_workspace_bytes
    assert f(-1) == 0
    assert f(_lib._CONSTS["LDA_ROUTE_MAX_N"] + 1) == 0
    prev = 0
    for N in (0, 1, 63, 64, 4095, 4096, 4097, 10 ** 6, 16777216):
        b = f(N)
        assert b >= 12 * (N + 512) and b >= prev and b % 256 == 0
        assert _lib.route_layout(N)["bytes"] == b   # the binding's mirror of the layout
        prev = b


def test_route_build_argument_errors(lib):
    import ctypes
    from paper_1505_03851_amd._lib import STATUS, RouteInfo
    r = RouteInfo()
    ws = lib.lda_route_workspace_bytes(10)

    def run(doc=A, word=A, N=10, M=3, V=5, w=A, wb=ws, route=True):
        return lib.lda_route_build(doc, word, N, M, V, w, wb,
                                   ctypes.byref(r) if route else None, None)
    assert run(route=False) == STATUS["LDA_ERR_NULL"]
    for kw in (dict(N=-1), dict(M=0), dict(V=0), dict(V=-2)):
        assert run(**kw) == STATUS["LDA_ERR_SHAPE"], kw
    assert run(N=2 ** 31) == STATUS["LDA_ERR_UNSUPPORTED"]
    for key in ("doc", "word", "w"):
        assert run(**{key: None}) == STATUS["LDA_ERR_NULL"], key
    assert run(doc=A + 2) == STATUS["LDA_ERR_ALIGN"]
    assert run(word=A + 1) == STATUS["LDA_ERR_ALIGN"]
    assert run(w=A + 4) == STATUS["LDA_ERR_ALIGN"]          # the workspace holds int64
    assert run(wb=ws - 1) == STATUS["LDA_ERR_WORKSPACE"]
    r.N = 77
    assert run(N=0, doc=None, word=None, w=None) == 0        # no-op, route cleared
    assert r.N == 0 and list(r.length) == [0] * 8


@pytest.mark.parametrize("philox", [False, True])
def test_draw_routed_argument_errors(lib, philox):
    import ctypes
    from paper_1505_03851_amd._lib import STATUS, RouteInfo
    N = 1000
    ws = lib.lda_route_workspace_bytes(N)
    r = RouteInfo()
    r.N = N
    for x in range(8):          # a consistent (made-up) route of N tokens
        r.tokens[x] = N // 8
        r.length[x] = (N // 8 + 63) // 64 * 64
        r.start[x] = x * r.length[0]

    def run(theta=A, phi=A, w=A, wb=ws, route=True, u=A, z=A, n=N, M=3, V=5, K=1024):
        rp = ctypes.byref(r) if route else None
        if philox:              # no u: the uniforms come from the seed
            return lib.lda_draw_routed_philox(theta, phi, w, wb, rp, z, n, M, V, K,
                                              12345, 0, None)
        return lib.lda_draw_routed(theta, phi, w, wb, rp, u, z, n, M, V, K, None)
    assert run(route=False) == STATUS["LDA_ERR_NULL"]
    for key in ("theta", "phi", "w", "z") + (() if philox else ("u",)):
        assert run(**{key: None}) == STATUS["LDA_ERR_NULL"], key
    for kw in (dict(n=-1), dict(M=0), dict(V=0), dict(K=0)):
        assert run(**kw) == STATUS["LDA_ERR_SHAPE"], kw
    # K: divisible by 4, 768 <= K <= 2048 (routing measured slower below)
    for K in (64, 128, 130, 256, 512, 764, 766, 1023, 2052, 4096):
        assert run(K=K) == STATUS["LDA_ERR_UNSUPPORTED"], K
    assert run(w=A + 4) == STATUS["LDA_ERR_ALIGN"]
    assert run(wb=ws - 1) == STATUS["LDA_ERR_WORKSPACE"]
    assert run(n=N - 1) == STATUS["LDA_ERR_WORKSPACE"]        # route of other tokens
    r.length[3] += 1                                          # not whole wavefronts
    assert run() == STATUS["LDA_ERR_WORKSPACE"]
    r.length[3] -= 1
    r.tokens[0] += 1                                          # token counts do not add up
    assert run() == STATUS["LDA_ERR_WORKSPACE"]
    r.tokens[0] -= 1
    r.start[7] = 10 ** 9                                      # past the workspace
    assert run() == STATUS["LDA_ERR_WORKSPACE"]
    assert run(n=0, theta=None, phi=None, w=None, u=None, z=None) == 0


def test_count_topics_argument_errors(lib):
    """lda_count_topics rejects bad arguments before any HIP call (calls that
    pass every check would launch kernels, so none is made here)."""
    from paper_1505_03851_amd._lib import STATUS, _CONSTS

    def run(d=A, w=A, z=A, N=100, M=3, V=5, K=7, ndk=A, nwk=A):
        return lib.lda_count_topics(d, w, z, N, M, V, K, ndk, nwk, None)
    for kw in (dict(N=-1), dict(M=0), dict(V=-2), dict(K=0)):
        assert run(**kw) == STATUS["LDA_ERR_SHAPE"], kw
    assert run(K=_CONSTS["LDA_MAX_K"] + 1) == STATUS["LDA_ERR_UNSUPPORTED"]
    assert run(N=_CONSTS["LDA_COUNT_MAX_N"] + 1) == STATUS["LDA_ERR_UNSUPPORTED"]
    assert run(M=1 << 22, K=1024) == STATUS["LDA_ERR_UNSUPPORTED"]   # ndk of 16 GiB
    assert run(V=1 << 22, K=1024) == STATUS["LDA_ERR_UNSUPPORTED"]   # nwk of 16 GiB
    for key in ("ndk", "nwk"):
        assert run(**{key: None}) == STATUS["LDA_ERR_NULL"], key
        assert run(N=0, **{key: None}) == STATUS["LDA_ERR_NULL"], key  # tables are cleared
    for key in ("d", "w", "z"):
        assert run(**{key: None}) == STATUS["LDA_ERR_NULL"], key
        assert run(**{key: A + 2}) == STATUS["LDA_ERR_ALIGN"], key
    for key in ("ndk", "nwk"):
        assert run(**{key: A + 1}) == STATUS["LDA_ERR_ALIGN"], key


def test_probe_argument_errors():
    """The probes reject bad arguments before any HIP call."""
    from paper_1505_03851_amd import probe
    from paper_1505_03851_amd._lib import STATUS
    lib = probe.load()

    def floor(N=1000, M=3, V=5, K=64, window=16, wpg=2, wpc=0, **ptr):
        p = dict(theta=A, phi=A, d=A, w=A, u=A, z=A)
        p.update(ptr)
        return lib.lda_probe_draw_floor(p["theta"], p["phi"], p["d"], p["w"], p["u"], p["z"],
                                        N, M, V, K, window, wpg, wpc, None)
    for kw in (dict(N=-1), dict(M=0), dict(V=0), dict(K=0)):
        assert floor(**kw) == STATUS["LDA_ERR_SHAPE"], kw
    for kw in (dict(K=30), dict(K=2052), dict(N=63), dict(window=4), dict(wpg=3),
               dict(wpc=-1), dict(wpc=33), dict(M=1 << 20, K=1024)):
        assert floor(**kw) == STATUS["LDA_ERR_UNSUPPORTED"], kw
    for key in ("theta", "phi", "d", "w", "u", "z"):
        assert floor(**{key: None}) == STATUS["LDA_ERR_NULL"], key
        assert floor(**{key: A + 2}) == STATUS["LDA_ERR_ALIGN"], key
    assert lib.lda_probe_read(A, 4096, 0, A, None) == STATUS["LDA_ERR_SHAPE"]
    assert lib.lda_probe_read(A, -16, 1, A, None) == STATUS["LDA_ERR_SHAPE"]
    assert lib.lda_probe_read(A, 0, 1, None, None) == 0             # no-op
    assert lib.lda_probe_read(None, 4096, 1, A, None) == STATUS["LDA_ERR_NULL"]
    assert lib.lda_probe_read(A + 4, 4096, 1, A, None) == STATUS["LDA_ERR_ALIGN"]
    assert lib.lda_probe_read(A, 4100, 1, A, None) == STATUS["LDA_ERR_ALIGN"]


def test_routed_scratch_argument_errors(lib):
    """lda_draw_routed_scratch rejects bad arguments, K outside the routed
    range and N whose routing does not fit its scratch array before any HIP
    call."""
    from paper_1505_03851_amd import _lib
    from paper_1505_03851_amd._lib import STATUS

    def run(N=1000, M=3, V=5, K=1024, **ptr):
        p = dict(theta=A, phi=A, d=A, w=A, u=A, z=A)
        p.update(ptr)
        return lib.lda_draw_routed_scratch(p["theta"], p["phi"], p["d"], p["w"], p["u"],
                                           p["z"], N, M, V, K, None)
    for kw in (dict(N=-1), dict(M=0), dict(V=0), dict(K=0)):
        assert run(**kw) == STATUS["LDA_ERR_SHAPE"], kw
    for K in (64, 256, 764, 1023, 2052):
        assert run(K=K) == STATUS["LDA_ERR_UNSUPPORTED"], K
    n = 5_000_000
    while lib.lda_route_workspace_bytes(n) <= _lib.ROUTED_SCRATCH_BYTES:
        n += 4096
    assert run(N=n) == STATUS["LDA_ERR_UNSUPPORTED"]
    for key in ("theta", "phi", "d", "w", "u", "z"):
        assert run(**{key: None}) == STATUS["LDA_ERR_NULL"], key
    assert run(N=0) == 0


def test_count_topics_docs_argument_errors(lib):
    from paper_1505_03851_amd._lib import STATUS

    def run(off=A, w=A, z=A, N=100, M=3, V=5, K=7, ndk=A, nwk=A):
        return lib.lda_count_topics_docs(off, w, z, N, M, V, K, ndk, nwk, None)
    for kw in (dict(N=-1), dict(M=0), dict(V=-2), dict(K=0)):
        assert run(**kw) == STATUS["LDA_ERR_SHAPE"], kw
    # (ndk may be of any size: a call with a large M passes every check and
    # would launch, so none is made here)
    assert run(V=1 << 22, K=1024) == STATUS["LDA_ERR_UNSUPPORTED"]   # nwk of 16 GiB
    for key in ("off", "ndk", "nwk"):
        assert run(**{key: None}) == STATUS["LDA_ERR_NULL"], key
        assert run(N=0, **{key: None}) == STATUS["LDA_ERR_NULL"], key
    for key in ("w", "z"):
        assert run(**{key: None}) == STATUS["LDA_ERR_NULL"], key
    assert run(off=A + 4) == STATUS["LDA_ERR_ALIGN"]
    assert run(w=A + 2) == STATUS["LDA_ERR_ALIGN"]


def test_word_index_sizes_and_layout(lib):
    """lda_word_index_bytes agrees with the layout the header states (and the
    binding's views use); 0 for sizes the index does not take."""
    from paper_1505_03851_amd._lib import _CONSTS, word_index_layout
    for N, V in ((0, 1), (1, 1), (1000, 7), (2048, 300), (16_777_216, 100_000),
                 (2 ** 31 - 1, _CONSTS["LDA_WORD_INDEX_MAX_V"])):
        assert lib.lda_word_index_bytes(N, V) == word_index_layout(N, V)["bytes"], (N, V)
    for N, V in ((-1, 5), (10, 0), (2 ** 31, 5), (10, _CONSTS["LDA_WORD_INDEX_MAX_V"] + 1)):
        assert lib.lda_word_index_bytes(N, V) == 0, (N, V)


def test_word_index_argument_errors(lib):
    """The build and the indexed counts reject bad arguments before any HIP
    call (calls that pass every check launch kernels, so none is made)."""
    from paper_1505_03851_amd._lib import STATUS, _CONSTS
    ws = lib.lda_word_index_bytes(100, 5)

    def build(w=A, N=100, V=5, index=A, nbytes=ws):
        return lib.lda_word_index_build(w, N, V, index, nbytes, None)
    assert build(N=-1) == STATUS["LDA_ERR_SHAPE"]
    assert build(V=0) == STATUS["LDA_ERR_SHAPE"]
    assert build(N=2 ** 31) == STATUS["LDA_ERR_UNSUPPORTED"]
    assert build(V=_CONSTS["LDA_WORD_INDEX_MAX_V"] + 1) == STATUS["LDA_ERR_UNSUPPORTED"]
    assert build(index=None) == STATUS["LDA_ERR_NULL"]
    assert build(w=None) == STATUS["LDA_ERR_NULL"]
    assert build(index=A + 4) == STATUS["LDA_ERR_ALIGN"]
    assert build(w=A + 2) == STATUS["LDA_ERR_ALIGN"]
    assert build(nbytes=ws - 1) == STATUS["LDA_ERR_WORKSPACE"]

    def count(off=A, w=A, z=A, N=100, M=3, V=5, K=7, index=A, nbytes=ws, ndk=A, nwk=A):
        return lib.lda_count_topics_indexed(off, w, z, N, M, V, K, index, nbytes, ndk, nwk, None)
    for kw in (dict(N=-1), dict(M=0), dict(V=-2), dict(K=0)):
        assert count(**kw) == STATUS["LDA_ERR_SHAPE"], kw
    assert count(K=_CONSTS["LDA_MAX_K"] + 1) == STATUS["LDA_ERR_UNSUPPORTED"]
    assert count(V=1 << 22, K=1024) == STATUS["LDA_ERR_UNSUPPORTED"]   # nwk of 16 GiB
    assert count(nbytes=ws - 1) == STATUS["LDA_ERR_WORKSPACE"]
    assert count(N=1000) == STATUS["LDA_ERR_WORKSPACE"]                # an index of 100 tokens
    for key in ("off", "ndk", "nwk", "index", "w", "z"):
        assert count(**{key: None}) == STATUS["LDA_ERR_NULL"], key
    for key in ("w", "z", "ndk", "nwk"):
        assert count(**{key: A + 2}) == STATUS["LDA_ERR_ALIGN"], key
    assert count(off=A + 4) == STATUS["LDA_ERR_ALIGN"]
    assert count(index=A + 4) == STATUS["LDA_ERR_ALIGN"]
