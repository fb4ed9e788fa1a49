"""Build the HIP libraries in-tree for gfx950: liblda_draw.so (the draw and
its C ABI, include/lda_draw.h) and liblda_probe.so (the measurement probes,
include/lda_probe.h)."""
from __future__ import annotations

import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
# the draw library: its C ABI with the default build of the kernels, and the
# build for tables past 4 GiB (lda_draw_wide.hip)
SRC = [os.path.join(PKG, "csrc", "lda_draw.hip"), os.path.join(PKG, "csrc", "lda_draw_wide.hip")]
LIB = os.path.join(PKG, "liblda_draw.so")
PROBE_SRC = os.path.join(PKG, "csrc", "probe.hip")
PROBE_LIB = os.path.join(PKG, "liblda_probe.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    # fp32 subnormals are kept (the products of small Dirichlet weights are
    # often subnormal); a*b+c may contract to one fused multiply-add.
    "-fno-gpu-flush-denormals-to-zero",
    "-ffp-contract=fast",
    # no packed-fp32 instructions in generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
    "-I", os.path.join(ROOT, "include"),
]


def _compile(src: str | list[str], lib: str, verbose: bool, extra: list[str] | None) -> str:
    srcs = [src] if isinstance(src, str) else list(src)
    cmd = [HIPCC, *FLAGS, *(extra or []), *srcs, "-o", lib + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(lib + ".tmp", lib)
    return lib


def build(verbose: bool = False, extra: list[str] | None = None) -> str:
    """Both libraries; returns the draw library's path."""
    _compile(PROBE_SRC, PROBE_LIB, verbose, extra)
    return _compile(SRC, LIB, verbose, extra)


if __name__ == "__main__":
    print(build(verbose=True))
