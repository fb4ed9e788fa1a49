#!/usr/bin/env python3
"""Benchmark of the per-token LDA topic draw on one MI355X.

One step = one launch of the draw over every token of the workload (all inputs
resident in HBM).  The headline workload is the K=1024 corpus (N=16,777,216
tokens, M=65,536 documents x 256, V=100,000 Zipf(1.05) words); the K=256
corpus is reported beside it, and every one of the five workloads is drawn
and compared with the oracle on every token.

Prints ONE JSON line.  ``roofline`` sets the draw against the memory floor of
its own access pattern: ``achieved`` is the launch's algorithmic bytes over
its average duration (HIP events on the launch stream), ``peak`` the same
bytes over the average duration of the memory-only probe that moves them in
the same token order (lda_probe_draw_floor, best of its launch shapes, timed
in the same run), so ``frac`` = floor time / draw time.  ``traffic`` is the
bytes the launch moves past L2 (rocprofv3 request-size counters, no
calibration factor), from the committed counter record while the headline
kernel's source is unchanged since it was taken, else null.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("z draws/sec and achieved HBM GB/s (% of peak) at K=256 and K=1024, "
          "1 MI355X")
PEAK_HBM_GBPS = 8000.0            # MI355X HBM3E, published
HEADLINE = "corpus16M-K1024"
SECOND = "corpus1M-K256"
PARITY_WORKLOADS = ("tiny-K32", "corpus1M-K64", "corpus1M-K256", "corpus16M-K1024",
                    "poisson300-K2048")
PROFILES = os.path.join(ROOT, "profiles")
CSRC = os.path.join(ROOT, "paper_1505_03851_amd", "csrc")
# the device kernel lda_draw_butterfly launches on each timed workload, and
# the source files it is compiled from
DEVICE_KERNEL = {HEADLINE: "leaf_eighths_kernel", SECOND: "leaf_group_kernel"}
_COMMON_SOURCES = ("butterfly.hpp", "philox.hpp", "sources.hpp", "tile.hpp", "tuning.hpp")
KERNEL_SOURCES = {"leaf_eighths_kernel": _COMMON_SOURCES + ("leaf_eighths.hpp",),
                  "leaf_group_kernel": _COMMON_SOURCES + ("leaf_group.hpp",)}


def counters_path(workload: str) -> str:
    return os.path.join(PROFILES, f"butterfly_{workload}_counters.json")


def kernel_source_hash(device_kernel: str = "leaf_eighths_kernel") -> str:
    """sha1 of the code of the files the device kernel is compiled from (in
    the order listed), with comments removed and runs of white space made one
    space: a counter record applies while this is unchanged.  (The files hold
    no comment markers inside string literals.)"""
    h = hashlib.sha1()
    for name in KERNEL_SOURCES[device_kernel]:
        with open(os.path.join(CSRC, name), encoding="utf-8") as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()


def routable(K: int) -> bool:
    """K the routed draw takes (divisible by 4, 768 <= K <= 2048: below, the
    routed draw is refused, being measured slower than the token-order
    draw)."""
    return K % 4 == 0 and 768 <= K <= 2048


def algorithmic_bytes(c) -> int:
    """Bytes the method must move: each token's phi row (4K), its doc id,
    word id, u and z (16), and each run of one document's tokens its theta row
    once (4K)."""
    import numpy as np
    runs = 1 + int(np.count_nonzero(np.diff(c.doc_id))) if c.N else 0
    return c.N * (4 * c.K + 16) + runs * 4 * c.K


def upload(c):
    """The corpus on the GPU; documents also as offsets when they are
    contiguous (the form lda_draw_docs takes)."""
    import numpy as np
    import torch
    from paper_1505_03851_amd.inputs import doc_offsets
    dev = {k: torch.from_numpy(getattr(c, k)).cuda()
           for k in ("theta", "phi", "doc_id", "word_id", "u")}
    if c.N == 0 or (np.diff(c.doc_id) >= 0).all():
        dev["doc_offsets"] = torch.from_numpy(doc_offsets(c.doc_id, c.M)).cuda()
    return dev


# kernels bench.py can time: name -> entry point of the binding
KERNELS = ("butterfly", "naive", "transposed", "docs", "doc_lanes", "doc_lanes_cache",
           "variant-register", "variant-lds", "variant-lds_alt", "variant-leaf8", "variant-wide",
           "philox",
           "routed",
           "routed+build", "routed-philox", "floor", "count", "count-clear", "count-docs",
           "count-indexed", "word-index", "sweep")


def draw_occupancy(K: int) -> tuple[int, int]:
    """(wavefronts per workgroup, wavefronts per CU) of the kernel
    lda_draw_butterfly launches for K divisible by 4 (N >= 64), as the
    compiler's register report for gfx950 gives them: the leaf-group kernel up
    to K = 256, 2 per workgroup and, per SIMD, 6 for groups of 8 lanes (K <=
    32), 5 for 16, 4 for 32 and 3 for 64; the leaf-eighths kernel above (4 per
    workgroup and 2 per SIMD up to 1280 topics, then 2 and 4)."""
    if K <= 256:
        per_simd = 6 if K <= 32 else 5 if K <= 64 else 4 if K <= 128 else 3
        return 2, 4 * per_simd
    return (4, 8) if K <= 1280 else (2, 16)


PHILOX_SEED = 0x5EED20150513


def launcher(kernel: str, dev):
    """A function (out, stream) that launches ``kernel`` once over ``dev``.
    "routed" draws the tokens routed to the XCDs with the routing built once
    beforehand (as a sampler does once per corpus); "routed+build" builds the
    routing again in every launch (one stream synchronisation inside)."""
    import torch
    import paper_1505_03851_amd as lda
    th, ph, d, w, u = (dev["theta"], dev["phi"], dev["doc_id"], dev["word_id"], dev["u"])
    if kernel == "routed":
        if "route" not in dev:
            dev["route"] = lda.route_build(d, w, th.shape[0], ph.shape[0])
        route = dev["route"]
        return lambda out, stream: lda.draw_routed(th, ph, route, u, out=out, stream=stream)
    if kernel == "routed-philox":
        if "route" not in dev:
            dev["route"] = lda.route_build(d, w, th.shape[0], ph.shape[0])
        route = dev["route"]
        return lambda out, stream: lda.draw_routed_philox(th, ph, route, PHILOX_SEED, 0,
                                                          out=out, stream=stream)
    if kernel == "routed+build":
        if "route" not in dev:
            dev["route"] = lda.route_build(d, w, th.shape[0], ph.shape[0])
        ws = dev["route"].workspace

        def build_and_draw(out, stream):
            r = lda.route_build(d, w, th.shape[0], ph.shape[0], workspace=ws, stream=stream)
            lda.draw_routed(th, ph, r, u, out=out, stream=stream)
        return build_and_draw
    if kernel == "floor":
        from paper_1505_03851_amd import probe
        window, wpg, wpc = dev.get("floor_cfg") or (16,) + draw_occupancy(th.shape[1])
        return lambda out, stream: probe.draw_floor(th, ph, d, w, u, out, window=window,
                                                    waves_per_group=wpg, waves_per_cu=wpc,
                                                    stream=stream)
    if kernel == "word-index":          # the index build (once per corpus in a sampler)
        V = ph.shape[0]
        ws = torch.empty(lda.word_index_bytes(w.shape[0], V), dtype=torch.uint8, device=w.device)
        return lambda out, stream: lda.word_index_build(w, V, workspace=ws, stream=stream)
    if kernel == "sweep":               # one sampler sweep: the draw, then its topic counts
        M, V, K = th.shape[0], ph.shape[0], th.shape[1]
        off = dev["doc_offsets"]
        if "word_index" not in dev:
            dev["word_index"] = lda.word_index_build(w, V)
        idx = dev["word_index"]
        ndk = torch.empty((M, K), dtype=torch.int32, device=d.device)
        nwk = torch.empty((V, K), dtype=torch.int32, device=d.device)

        def draw_and_count(out, stream):
            lda.draw_butterfly(th, ph, d, w, u, out=out, stream=stream)
            lda.count_topics_indexed(off, w, out, idx, K, ndk=ndk, nwk=nwk, stream=stream)
        return draw_and_count
    if kernel in ("count", "count-clear", "count-docs", "count-indexed"):
        M, V, K = th.shape[0], ph.shape[0], th.shape[1]
        if "z_draw" not in dev:
            dev["z_draw"] = lda.draw_butterfly(th, ph, d, w, u)
            dev["ndk"] = torch.empty((M, K), dtype=torch.int32, device=d.device)
            dev["nwk"] = torch.empty((V, K), dtype=torch.int32, device=d.device)
        zd, ndk, nwk = dev["z_draw"], dev["ndk"], dev["nwk"]
        if kernel == "count-clear":     # the tables cleared, no token counted
            e = d[:0]
            return lambda out, stream: lda.count_topics(e, e, e, M, V, K, ndk=ndk, nwk=nwk,
                                                        stream=stream)
        if kernel == "count-docs":      # documents as offsets: rows of ndk written whole
            off = dev["doc_offsets"]
            return lambda out, stream: lda.count_topics_docs(off, w, zd, V, K, ndk=ndk, nwk=nwk,
                                                             stream=stream)
        if kernel == "count-indexed":   # and nwk from the word index (built once per corpus)
            off = dev["doc_offsets"]
            if "word_index" not in dev:
                dev["word_index"] = lda.word_index_build(w, V)
            idx = dev["word_index"]
            return lambda out, stream: lda.count_topics_indexed(off, w, zd, idx, K, ndk=ndk,
                                                                nwk=nwk, stream=stream)
        return lambda out, stream: lda.count_topics(d, w, zd, M, V, K, ndk=ndk, nwk=nwk,
                                                    stream=stream)
    if kernel == "philox":
        return lambda out, stream: lda.draw_philox(th, ph, d, w, PHILOX_SEED, 0, out=out,
                                                   stream=stream)
    if kernel == "docs":
        off = dev["doc_offsets"]
        return lambda out, stream: lda.draw_docs(th, ph, off, w, u, out=out, stream=stream)
    if kernel in ("doc_lanes", "doc_lanes_cache"):
        off, cache = dev["doc_offsets"], kernel == "doc_lanes_cache"
        return lambda out, stream: lda.draw_doc_lanes(th, ph, off, w, u, theta_cache=cache,
                                                      out=out, stream=stream)
    if kernel.startswith("variant-"):
        v = kernel[len("variant-"):]
        return lambda out, stream: lda.draw_variant(th, ph, d, w, u, variant=v, out=out,
                                                    stream=stream)
    fn = {"butterfly": lda.draw_butterfly, "naive": lda.draw_naive,
          "transposed": lda.draw_transposed}[kernel]
    return lambda out, stream: fn(th, ph, d, w, u, out=out, stream=stream)


def time_kernel(kernel: str, dev, steps: int, warmup: int, flush=None):
    """Warm up, then time exactly ``steps`` launches.  Returns (wall seconds of
    the timed region, per-launch milliseconds from HIP events, z).  With
    ``flush`` (a large device tensor), it is overwritten before every timed
    launch, outside the launch's event pair: a cold-cache launch."""
    import torch
    launch = launcher(kernel, dev)
    stream = torch.cuda.current_stream()
    z = torch.empty_like(dev["doc_id"])
    for _ in range(warmup):
        launch(z, stream)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True),
           torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    t0 = time.perf_counter()
    for s, e in ev:
        if flush is not None:
            flush.zero_()
        s.record(stream)
        launch(z, stream)
        e.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return wall, [s.elapsed_time(e) for s, e in ev], z


def count_bytes(c) -> int:
    """Bytes the topic counts must move: each token's doc id, word id and z
    read (12), both tables written whole (4 (M + V) K)."""
    return 12 * c.N + 4 * (c.M + c.V) * c.K


def measure(name: str, c, dev, kernel: str, steps: int, warmup: int, flush=None) -> dict:
    wall, per_ms, z = time_kernel(kernel, dev, steps, warmup, flush)
    avg_ms = sum(per_ms) / len(per_ms)
    srt = sorted(per_ms)
    med_ms = srt[len(srt) // 2]
    if kernel.startswith("count"):
        b_alg = count_bytes(c)
    elif kernel == "word-index":     # word ids read twice, perm and wsorted written
        b_alg = 16 * c.N
    elif kernel == "sweep":
        b_alg = algorithmic_bytes(c) + count_bytes(c)
    else:
        b_alg = algorithmic_bytes(c)
    gbps = b_alg / (avg_ms * 1e-3) / 1e9
    tag = " cold" if flush is not None else ""
    print(f"[bench] {name} {kernel}{tag}: {avg_ms:.3f} ms/launch "
          f"(median {med_ms:.3f}, min {srt[0]:.3f}, max {srt[-1]:.3f}), "
          f"{c.N / (avg_ms * 1e-3) / 1e9:.3f} G tokens/s, "
          f"{gbps:.0f} GB/s of algorithmic bytes", file=sys.stderr, flush=True)
    return {
        "workload": name, "kernel": kernel + ("-cold" if flush is not None else ""),
        "N": c.N, "K": c.K, "steps": steps, "wall_s": wall,
        "ms_per_launch": avg_ms, "ms_per_launch_median": med_ms,
        "ms_per_launch_min": srt[0], "ms_per_launch_max": srt[-1],
        "draws_per_s": c.N / (avg_ms * 1e-3),
        "alg_bytes_per_launch": b_alg,
        "alg_GBps": gbps,
        "z": z,
    }


MALL_PROBE_BYTES = 192 << 20   # above the 8 x 4 MiB of L2, inside the 256 MiB MALL
MALL_PROBE_PASSES = 8
HBM_PROBE_BYTES = 4 << 30     # 16x the MALL


def read_ceiling(nbytes: int, passes: int, steps: int = 10) -> tuple[float, float]:
    """(ms per launch, GB/s) of the streaming-read probe over ``nbytes``,
    ``passes`` times per launch (median of ``steps`` HIP-event-timed
    launches after two warm-up launches)."""
    import torch
    from paper_1505_03851_amd import probe
    buf = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    out = torch.empty(probe.READ_OUT_FLOATS, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    for _ in range(2):
        probe.read(buf, passes, out, stream=stream)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    for a, b in ev:
        a.record(stream)
        probe.read(buf, passes, out, stream=stream)
        b.record(stream)
    torch.cuda.synchronize()
    ms = sorted(a.elapsed_time(b) for a, b in ev)[steps // 2]
    del buf, out
    torch.cuda.empty_cache()
    return ms, nbytes * passes / (ms * 1e-3) / 1e9


def device_copy_GBps(steps: int = 10) -> float:
    """Bytes read plus bytes written per second by a plain 1 GiB device copy
    (torch's copy kernel, HIP events): the practical HBM ceiling on this machine."""
    import torch
    n = 1 << 28
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    for a, b in ev:
        a.record()
        dst.copy_(src)
        b.record()
    torch.cuda.synchronize()
    ms = sorted(a.elapsed_time(b) for a, b in ev)[steps // 2]
    del src, dst
    torch.cuda.empty_cache()
    return 2 * 4 * n / (ms * 1e-3) / 1e9


def traffic_from_counters(workload: str):
    """Bytes per launch that the headline kernel moves past L2 (read +
    written), from the committed counter record, if it was taken on the
    kernel's current source; else None."""
    try:
        with open(counters_path(workload)) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_sha1") != kernel_source_hash(rec.get("device_kernel", "")):
        return None
    return rec.get("egress_bytes_per_launch")


def _counter_means(d: str, kernel_substr: str) -> dict:
    """Mean per-dispatch value of each counter in a rocprofv3 --pmc csv
    directory, over the dispatches whose kernel name contains
    ``kernel_substr`` (per-dispatch values are summed over instances)."""
    per = {}
    for path in glob.glob(os.path.join(d, "*counter_collection.csv")):
        with open(path) as f:
            for row in csv.DictReader(f):
                if kernel_substr not in row["Kernel_Name"]:
                    continue
                key = (row["Counter_Name"], row["Dispatch_Id"])
                per[key] = per.get(key, 0.0) + float(row["Counter_Value"])
    out = {}
    for (name, _), v in per.items():
        out.setdefault(name, []).append(v)
    if not out:
        raise SystemExit(f"no dispatch of {kernel_substr!r} in {d}")
    return {k: sum(v) / len(v) for k, v in out.items()}


# rocprofv3 counter passes of one kernel (at most 4 TCC counters per pass)
PASS_READS = ("TCC_EA0_RDREQ_32B_sum", "TCC_EA0_RDREQ_64B_sum", "TCC_EA0_RDREQ_128B_sum",
              "TCC_EA0_RDREQ_sum")
PASS_DRAM = ("TCC_EA0_RDREQ_DRAM_32B_sum", "TCC_EA0_WRREQ_WRITE_DRAM_32B_sum",
             "TCC_EA0_WRREQ_sum", "TCC_EA0_WRREQ_64B_sum")
PASS_HIT = ("TCC_HIT_sum", "TCC_MISS_sum", "TCP_TCC_READ_REQ_sum", "SQ_INSTS_VMEM_RD")


def egress_record(reads: str, dram: str, kname: str, hit: str | None = None) -> dict:
    """Bytes that dispatches of ``kname`` move past L2, from the request-size
    counters: read = 32 n32 + 64 n64 + 128 n128 (the three sizes must add up
    to all read requests); written = 32 (all - n64) + 64 n64.  Cross-check:
    the DRAM-side counters count the same reads and writes in 32-byte units."""
    r = _counter_means(reads, kname)
    d = _counter_means(dram, kname)
    n32, n64, n128 = (r["TCC_EA0_RDREQ_32B_sum"], r["TCC_EA0_RDREQ_64B_sum"],
                      r["TCC_EA0_RDREQ_128B_sum"])
    rec = {
        "read_requests": {"32B": n32, "64B": n64, "128B": n128,
                          "all": r["TCC_EA0_RDREQ_sum"]},
        "read_sizes_cover_all_requests": (n32 + n64 + n128) / max(r["TCC_EA0_RDREQ_sum"], 1),
        "bytes_read": 32 * n32 + 64 * n64 + 128 * n128,
        "bytes_read_dram_side": 32 * d["TCC_EA0_RDREQ_DRAM_32B_sum"],
        "bytes_written": 32 * (d["TCC_EA0_WRREQ_sum"] - d["TCC_EA0_WRREQ_64B_sum"]) +
                         64 * d["TCC_EA0_WRREQ_64B_sum"],
        "bytes_written_dram_side": 32 * d["TCC_EA0_WRREQ_WRITE_DRAM_32B_sum"],
    }
    rec["egress_bytes_per_launch"] = rec["bytes_read"] + rec["bytes_written"]
    if hit:
        h = _counter_means(hit, kname)
        rec["tcc_hit_rate"] = h["TCC_HIT_sum"] / (h["TCC_HIT_sum"] + h["TCC_MISS_sum"])
        rec["l1_to_l2_read_requests"] = h["TCP_TCC_READ_REQ_sum"]
        rec["vector_load_instructions"] = h["SQ_INSTS_VMEM_RD"]
        rec["l2_requests_per_load"] = h["TCP_TCC_READ_REQ_sum"] / max(h["SQ_INSTS_VMEM_RD"], 1)
    return rec


def counters_summary(args) -> int:
    """The counter record of the draw on one workload (--workload), from the
    csv directories of its three counter passes (--reads, --dram, --hitmiss);
    ``traffic_from_counters`` reads it back."""
    kname = DEVICE_KERNEL[args.workload]
    rec = {"kernel": "butterfly", "device_kernel": kname, "workload": args.workload,
           "kernel_source_sha1": kernel_source_hash(kname)}
    rec.update(egress_record(args.reads, args.dram, kname, args.hitmiss))
    out = args.out or counters_path(args.workload)
    with open(out, "w") as f:
        json.dump(rec, f, indent=1)
        f.write("\n")
    print(json.dumps(rec, indent=1))
    return 0


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(c, z_gpu, sample: int) -> dict:
    """The oracle, as it stands, on the first ``sample`` tokens with all its
    OpenMP threads, and on the first ``sample // 16`` with one thread."""
    import numpy as np
    import oracle
    n = min(sample, c.N)
    d, w, u = c.doc_id[:n], c.word_id[:n], c.u[:n]
    oracle.draw(c.theta, c.phi, d[:1024], w[:1024], u[:1024], with_band=False)
    threads = oracle.num_threads()
    t0 = time.perf_counter()
    z_ref = oracle.draw(c.theta, c.phi, d, w, u, with_band=False)
    dt = time.perf_counter() - t0
    n1 = max(1, n // 16)
    oracle.set_num_threads(1)
    t1 = time.perf_counter()
    oracle.draw(c.theta, c.phi, d[:n1], w[:n1], u[:n1], with_band=False)
    dt1 = time.perf_counter() - t1
    oracle.set_num_threads(threads)
    zg = z_gpu[:n].cpu().numpy()
    # parity on the same sample (outside the timed call): every mismatch must
    # lie in the rounding band |u*S - S_k| <= 1e-5 * S
    z_chk, band = oracle.draw(c.theta, c.phi, d, w, u, with_band=True)
    mism = zg != z_chk
    return {
        "_ref": (z_chk, band),
        "value": n / dt, "unit": "draws/s", "cores": threads,
        "kind": "oracle",
        "sample": f"first {n} tokens of {c.name} (K={c.K}), fp64 oracle, "
                  f"draw only, {dt:.2f} s wall",
        "cpu": cpu_model(), "host_cpus": os.cpu_count(),
        "single_thread": {"value": n1 / dt1, "unit": "draws/s",
                          "sample": f"first {n1} tokens, 1 thread, {dt1:.2f} s wall"},
        "parity": {
            "tokens": n,
            "mismatches": int(mism.sum()),
            "mismatch_rate": float(mism.mean()),
            "mismatches_outside_band": int((mism & ~band).sum()),
            "mismatches_not_admitted": not_admitted(c, d, w, u, zg, z_chk, band),
            "in_band_rate": float(band.mean()),
        },
    }


def k_sweep(args) -> int:
    """Kernel time of the naive and butterfly draws at the paper's topic
    counts, on the synthetic corpus shaped like its evaluation corpus."""
    import torch
    from paper_1505_03851_amd.inputs import WIKI_K, make_corpus, wiki_shaped
    for K in WIKI_K:
        c = make_corpus(wiki_shaped(K))
        dev = upload(c)
        rec = {"workload": c.name, "K": K, "N": c.N}
        for kernel in ("naive", "transposed", "doc_lanes", "doc_lanes_cache", "butterfly"):
            r = measure(c.name, c, dev, kernel, args.steps, args.warmup)
            rec[kernel + "_ms"] = r["ms_per_launch"]
            rec[kernel + "_draws_per_s"] = r["draws_per_s"]
        rec["speedup"] = rec["naive_ms"] / rec["butterfly_ms"]
        rec["speedup_vs_transposed"] = rec["transposed_ms"] / rec["butterfly_ms"]
        rec["speedup_vs_doc_lanes"] = rec["doc_lanes_ms"] / rec["butterfly_ms"]
        print(json.dumps(rec), flush=True)
        del dev
        torch.cuda.empty_cache()
    return 0


def route_sweep(args) -> int:
    """Where routing the tokens to the XCDs pays: the plain draw against the
    routed draw (routing built once, and rebuilt in every launch) on the
    16.8M-token corpus at K = 256 ... 2048; one JSON line per K."""
    import torch
    from paper_1505_03851_amd.inputs import corpus16M_at, make_corpus
    for K in (256, 512, 768, 1024, 1536, 2048):
        c = make_corpus(corpus16M_at(K))
        dev = upload(c)
        rec = {"workload": c.name, "N": c.N, "V": c.V, "K": K,
               "phi_MiB": 4 * c.V * K / 2 ** 20}
        z_bf = None
        for kernel in ("butterfly", "routed", "routed+build"):
            if kernel != "butterfly" and not routable(K):
                rec[kernel + "_ms"] = None      # refused below K = 768
                continue
            r = measure(c.name, c, dev, kernel, args.steps, args.warmup)
            z = r.pop("z")
            if z_bf is None:
                z_bf = z
            else:
                rec[kernel + "_differs_from_butterfly"] = int((z != z_bf).sum())
            rec[kernel + "_ms"] = r["ms_per_launch"]
        if routable(K):
            rec["routed_speedup"] = rec["butterfly_ms"] / rec["routed_ms"]
            rec["routed_build_speedup"] = rec["butterfly_ms"] / rec["routed+build_ms"]
        print(json.dumps(rec), flush=True)
        del dev, c
        torch.cuda.empty_cache()
    return 0


FLOOR_SWEEP_K = (256, 260, 384, 512, 640, 768, 1024, 1280, 1536, 2048)


def floor_sweep(args) -> int:
    """Each draw against its own floor across K on the 16.8M-token corpus (or,
    with --wiki, on the corpus shaped like the paper's at its eight K): the
    token-order draw and the fastest launch shape of the floor probe, and
    (K >= 768) the routed draw, routing built once, and the routed order's
    floor; one JSON line per K, with each draw's fraction of its floor."""
    import torch
    from paper_1505_03851_amd.inputs import WIKI_K, corpus16M_at, make_corpus, wiki_shaped
    ks = [int(k) for k in args.floor_k.split(",")] if args.floor_k else \
        (WIKI_K if args.wiki else FLOOR_SWEEP_K)
    for K in ks:
        c = make_corpus(wiki_shaped(K) if args.wiki else corpus16M_at(K))
        dev = upload(c)
        rec = {"workload": c.name, "N": c.N, "V": c.V, "K": K}
        measure(c.name, c, dev, "butterfly", args.steps, args.warmup)  # (untimed pass)
        r = measure(c.name, c, dev, "butterfly", args.steps, args.warmup)
        r.pop("z")
        f = measure_floor(c.name, c, dev, args.steps, args.warmup)
        rec.update({"butterfly_ms": r["ms_per_launch"], "floor_ms": f["ms_per_launch"],
                    "floor_shape": f["shape"], "frac": f["ms_per_launch"] / r["ms_per_launch"]})
        if routable(K):
            r = measure(c.name, c, dev, "routed", args.steps, args.warmup)
            r.pop("z")
            f = measure_routed_floor(c.name, c, dev, args.steps, args.warmup)
            rec.update({"routed_ms": r["ms_per_launch"], "routed_floor_ms": f["ms_per_launch"],
                        "routed_floor_shape": f["shape"],
                        "routed_frac": f["ms_per_launch"] / r["ms_per_launch"]})
        print(json.dumps(rec), flush=True)
        del dev, c
        torch.cuda.empty_cache()
    return 0


def ablation(args) -> int:
    """The table variants of Section 4 (the paper's rule with the table in
    registers or LDS, the alternative rule in LDS), 8-topic leaves, the build
    for tables past 4 GiB, the offsets form of the documents, the
    document-per-lane driver, the draw with in-kernel uniforms and the default
    dispatch, on the two corpora and the corpus
    shaped like the paper's at K = 80 and 240; one JSON line per workload.
    z of every variant is compared with the default kernel's (identical
    unless a token lies in the fp32 rounding band)."""
    import torch
    from paper_1505_03851_amd.inputs import make_corpus, wiki_shaped
    names = [SECOND, HEADLINE, wiki_shaped(80).name, wiki_shaped(240).name]
    for name in names:
        c = make_corpus(name)
        dev = upload(c)
        rec = {"workload": name, "N": c.N, "K": c.K}
        z_ref = None
        kernels = ["butterfly", "variant-register", "variant-lds", "variant-lds_alt",
                   "variant-leaf8", "variant-wide", "docs", "doc_lanes"] + \
                  (["doc_lanes_cache"] if c.K <= 256 else []) + ["philox"]
        # one untimed pass first: the first kernel timed after the upload
        # otherwise runs a few percent slow (measured: docs and philox, the
        # same kernel, 1.5-4.5% faster than the butterfly timed before them)
        measure(name, c, dev, "butterfly", args.steps, args.warmup)
        for kernel in kernels:
            r = measure(name, c, dev, kernel, args.steps, args.warmup)
            z = r.pop("z")
            if z_ref is None:
                z_ref = z
            rec[kernel + "_ms"] = r["ms_per_launch"]
            if kernel != "philox":   # (other uniforms: z is not comparable)
                rec[kernel + "_differs"] = int((z != z_ref).sum())
        print(json.dumps(rec), flush=True)
        del dev
        torch.cuda.empty_cache()
    return 0


def wide_builds(args) -> int:
    """The default build of the draw kernels against the build for tables past
    4 GiB (rows addressed by index, 64-bit addresses;
    lda_draw_butterfly_variant with LDA_VARIANT_WIDE_TABLES) on the same workloads: three alternating rounds
    of each after an untimed pass, the median launch of each round, the
    fastest round kept; z of the two compared.  One JSON line per workload."""
    import torch
    from paper_1505_03851_amd.inputs import CONFIGS, make_corpus, wiki_shaped
    names = [n for n in CONFIGS if not n.startswith("wiki-shaped")] + \
            [wiki_shaped(k).name for k in (16, 48, 80, 112, 144, 176, 208, 240)]
    for name in names:
        c = make_corpus(name)
        dev = upload(c)
        time_kernel("butterfly", dev, args.steps, args.warmup)
        best = {"butterfly": float("inf"), "variant-wide": float("inf")}
        zs = {}
        for _ in range(3):
            for kernel in best:
                _, per_ms, zs[kernel] = time_kernel(kernel, dev, args.steps, args.warmup)
                best[kernel] = min(best[kernel], sorted(per_ms)[len(per_ms) // 2])
        rec = {"workload": name, "N": c.N, "K": c.K, "default_ms": best["butterfly"],
               "wide_ms": best["variant-wide"],
               "wide_over_default": best["variant-wide"] / best["butterfly"],
               "z_identical": bool(torch.equal(zs["butterfly"], zs["variant-wide"]))}
        print(json.dumps(rec), flush=True)
        del dev, zs
        torch.cuda.empty_cache()
    return 0


def permuted_ids(args) -> int:
    """Sensitivity of the draw, the routed draw, the word index build and the
    indexed counts to the order of the word ids: each workload as generated
    (ids by falling frequency, so the frequent rows of phi lie together) and
    with its ids renamed by a fixed random permutation, phi's rows moved with
    them (every token draws from the same weights).  Three alternating rounds
    after an untimed pass, the median launch of each round, the fastest round
    kept; z and the counts of the two orders compared.  One JSON line per
    workload."""
    import numpy as np
    import torch
    from paper_1505_03851_amd.inputs import Corpus, make_corpus
    for name in ("corpus1M-K64", SECOND, HEADLINE, "poisson300-K2048"):
        c = make_corpus(name)
        perm = np.random.default_rng(150503851).permutation(c.V).astype(np.int32)
        phi_p = np.empty_like(c.phi)
        phi_p[perm] = c.phi
        cp = Corpus(c.theta, phi_p, c.doc_id, perm[c.word_id], c.u, name=name + "-permuted")
        devs = {"sorted": upload(c), "permuted": upload(cp)}
        kernels = ["butterfly"] + (["routed"] if routable(c.K) else []) + \
                  ["word-index", "count-indexed"]
        for dev in devs.values():
            time_kernel("butterfly", dev, args.steps, args.warmup)
        best = {(o, k): float("inf") for o in devs for k in kernels}
        zs = {}
        for _ in range(3):
            for k in kernels:
                for o, dev in devs.items():
                    _, per_ms, zs[o, k] = time_kernel(k, dev, args.steps, args.warmup)
                    best[o, k] = min(best[o, k], sorted(per_ms)[len(per_ms) // 2])
        rec = {"workload": name, "N": c.N, "V": c.V, "K": c.K}
        for k in kernels:
            rec[k + "_sorted_ms"] = best["sorted", k]
            rec[k + "_permuted_ms"] = best["permuted", k]
            rec[k + "_permuted_over_sorted"] = best["permuted", k] / best["sorted", k]
        rec["z_identical"] = bool(torch.equal(zs["sorted", "butterfly"],
                                              zs["permuted", "butterfly"]))
        if routable(c.K):
            rec["routed_z_differs"] = int((zs["sorted", "routed"]
                                           != zs["permuted", "routed"]).sum())
        perm_t = torch.from_numpy(perm).long().cuda()
        s, p = devs["sorted"], devs["permuted"]
        rec["counts_identical"] = bool(torch.equal(s["ndk"], p["ndk"]) and
                                       torch.equal(s["nwk"], p["nwk"][perm_t]))
        print(json.dumps(rec), flush=True)
        del devs, zs, s, p
        torch.cuda.empty_cache()
    return 0


def all_configs(args) -> int:
    """Every kernel on every workload of inputs.CONFIGS but the K sweep's, warm
    and (butterfly) with a cold cache; one JSON line per workload."""
    import torch
    from paper_1505_03851_amd.inputs import CONFIGS, make_corpus
    flush = torch.empty(1 << 28, dtype=torch.float32, device="cuda")  # 1 GiB
    for name in [n for n in CONFIGS if not n.startswith("wiki-shaped")]:
        c = make_corpus(name)
        dev = upload(c)
        rec = {"workload": name, "N": c.N, "M": c.M, "V": c.V, "K": c.K,
               "alg_bytes_per_launch": algorithmic_bytes(c)}
        for kernel in ("naive", "transposed", "butterfly"):
            steps = args.steps if kernel != "naive" or c.K <= 256 else max(3, args.steps // 4)
            r = measure(name, c, dev, kernel, steps, args.warmup)
            for key in ("ms_per_launch", "ms_per_launch_median", "ms_per_launch_min",
                        "ms_per_launch_max", "draws_per_s", "alg_GBps"):
                rec[f"{kernel}_{key}"] = r[key]
        r = measure(name, c, dev, "butterfly", args.steps, args.warmup, flush=flush)
        for key in ("ms_per_launch", "ms_per_launch_median", "draws_per_s", "alg_GBps"):
            rec[f"butterfly_cold_{key}"] = r[key]
        if routable(c.K):
            z_bf = measure(name, c, dev, "butterfly", 1, 0)["z"]
            for kernel in ("routed", "routed+build", "routed-philox"):
                r = measure(name, c, dev, kernel, args.steps, args.warmup)
                for key in ("ms_per_launch", "ms_per_launch_median", "draws_per_s", "alg_GBps"):
                    rec[f"{kernel}_{key}"] = r[key]
                if kernel != "routed-philox":   # (other uniforms: z is not comparable)
                    rec[f"{kernel}_differs_from_butterfly"] = int((r["z"] != z_bf).sum())
        print(json.dumps(rec), flush=True)
        del dev
        torch.cuda.empty_cache()
    return 0


def graph_timing(args) -> int:
    """Launch overhead: ``steps`` back-to-back draws launched one by one
    against the same draws captured once in a HIP graph and replayed, on the
    small workloads where a launch costs as much as the draw; one JSON line
    per workload (per-draw time from events around all the draws)."""
    import torch
    from paper_1505_03851_amd.inputs import make_corpus
    reps = max(args.steps, 50)
    for name in ("tiny-K32", "corpus1M-K64", "corpus1M-K256"):
        c = make_corpus(name)
        dev = upload(c)
        launch = launcher("butterfly", dev)
        z = torch.empty_like(dev["doc_id"])
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            for _ in range(3):
                launch(z, s)
        torch.cuda.current_stream().wait_stream(s)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(reps):
                launch(z, torch.cuda.current_stream())
        stream = torch.cuda.current_stream()
        e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
        g.replay()
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(reps):
            launch(z, stream)
        e1.record(stream)
        g.replay()
        e2.record(stream)
        torch.cuda.synchronize()
        eager_us = 1e3 * e0.elapsed_time(e1) / reps
        graph_us = 1e3 * e1.elapsed_time(e2) / reps
        print(f"[bench] {name} butterfly x{reps}: {eager_us:.2f} us/draw launched one by one, "
              f"{graph_us:.2f} us/draw from one graph", file=sys.stderr, flush=True)
        print(json.dumps({"workload": name, "N": c.N, "K": c.K, "draws": reps,
                          "eager_us_per_draw": eager_us, "graph_us_per_draw": graph_us,
                          "graph_draws_per_s": c.N / (graph_us * 1e-6)}), flush=True)
        del g, dev
        torch.cuda.empty_cache()
    return 0


# ---------------------------------------------------------------------------
# Profiling: the rocprofv3 runs behind profiles/, and the reductions of their
# csv files into the committed summaries.

# label -> (substring of the device kernel's name, bench.py arguments)
PROFILE_TARGETS = {
    "copy": ("copyBuffer", ["--copy"]),
    "hbm_read": ("read_kernel", ["--ceiling", "hbm", "--steps", "3"]),
    "mall_read": ("read_kernel", ["--ceiling", "mall", "--steps", "3"]),
    "draw_K1024": ("leaf_eighths_kernel", ["--only", "butterfly", "--workload", HEADLINE,
                                           "--steps", "3", "--warmup", "1"]),
    "floor_K1024": ("floor_kernel", ["--only", "floor", "--floor-config", "8,4,8",
                                     "--workload", HEADLINE, "--steps", "3", "--warmup", "1"]),
    "naive_K1024": ("naive_kernel", ["--only", "naive", "--workload", HEADLINE,
                                     "--steps", "2", "--warmup", "0"]),
    "count_K1024": ("count_kernel", ["--only", "count", "--workload", HEADLINE,
                                     "--steps", "3", "--warmup", "1"]),
    "cdocs_K1024": ("count_docs_kernel", ["--only", "count-docs", "--workload", HEADLINE,
                                          "--steps", "3", "--warmup", "1"]),
    "cwords_K1024": ("count_words_kernel", ["--only", "count-docs", "--workload", HEADLINE,
                                            "--steps", "3", "--warmup", "1"]),
    "cindexed_K1024": ("count_words_indexed", ["--only", "count-indexed", "--workload", HEADLINE,
                                               "--steps", "3", "--warmup", "1"]),
    "draw_K256": ("leaf_group_kernel", ["--only", "butterfly", "--workload", SECOND,
                                        "--steps", "3", "--warmup", "1"]),
    "floor_K256": ("floor_kernel", ["--only", "floor", "--floor-config", "16,2,0",
                                    "--workload", SECOND, "--steps", "3", "--warmup", "1"]),
    "naive_K256": ("naive_kernel", ["--only", "naive", "--workload", SECOND,
                                    "--steps", "3", "--warmup", "1"]),
    "draw_K64": ("leaf_group_kernel", ["--only", "butterfly", "--workload", "corpus1M-K64",
                                       "--steps", "3", "--warmup", "1"]),
    "floor_K64": ("floor_kernel", ["--only", "floor", "--floor-config", "8,2,0",
                                   "--workload", "corpus1M-K64", "--steps", "3", "--warmup", "1"]),
    # groups of 8 lanes, which keep their leaves' partial sums in LDS (no reload)
    "draw_W16": ("leaf_group_kernel", ["--only", "butterfly", "--workload", "wiki-shaped-K16",
                                       "--steps", "3", "--warmup", "1"]),
    "floor_W16": ("floor_kernel", ["--only", "floor", "--floor-config", "8,2,0",
                                   "--workload", "wiki-shaped-K16", "--steps", "3",
                                   "--warmup", "1"]),
    "draw_K2048": ("leaf_eighths_kernel", ["--only", "butterfly", "--workload",
                                           "poisson300-K2048", "--steps", "3", "--warmup", "1"]),
    "routed_K1024": ("routed_eighths_kernel", ["--only", "routed", "--workload", HEADLINE,
                                               "--steps", "3", "--warmup", "1"]),
}
PROFILE_PASSES = {"reads": PASS_READS, "dram": PASS_DRAM, "hit": PASS_HIT}


def profile_commands(d: str) -> list[str]:
    """The shell commands (repository root, on the MI355X machine) that take every counter
    pass of every target into ``d``, and the kernel trace of the default
    bench run; each rocprofv3 run under its own time limit."""
    cmds = ["cd /tmp && export TMPDIR=/tmp && cd \"$GRAFT_REPO_ROOT\" && "
            "export LDA_INPUT_CACHE=/tmp/lda_inputs"]
    for label, (_, bargs) in PROFILE_TARGETS.items():
        for pn, ctr in PROFILE_PASSES.items():
            out = f"{d}/{label}_{pn}"
            cmds.append(f"timeout -s KILL 300 rocprofv3 --pmc {' '.join(ctr)} -f csv -d {out} "
                        f"-o c -- python -u bench.py {' '.join(bargs)} > {out}.log 2>&1")
    cmds.append(f"timeout -k 10 600 rocprofv3 --kernel-trace --stats -f csv -d {d}/trace -o t "
                f"-- python -u bench.py > {d}/trace.log 2>&1")
    return cmds


def _bench_lines(path: str) -> list[dict]:
    with open(path) as f:
        return [json.loads(ln) for ln in f if ln.startswith("{")]


def _fmt_bytes(b):
    return "-" if b is None else f"{b / 1e9:10.3f}"


def report_counters(d: str, out_txt: str) -> int:
    """profiles/counters_all_kernels.txt, and the counter records of the draw
    on the two timed workloads, from the counter passes in ``d``."""
    rows = []
    for label, (kname, bargs) in PROFILE_TARGETS.items():
        if not os.path.isdir(f"{d}/{label}_reads"):
            continue
        rec = egress_record(f"{d}/{label}_reads", f"{d}/{label}_dram", kname,
                            f"{d}/{label}_hit" if os.path.isdir(f"{d}/{label}_hit") else None)
        lines = _bench_lines(f"{d}/{label}_reads.log")
        ms = None
        if lines:
            ms = lines[-1].get("ms_per_launch") or lines[-1].get("ms_per_launch_median")
        if label.startswith("draw_K") and kname in DEVICE_KERNEL.values():
            wl = bargs[bargs.index("--workload") + 1]
            if DEVICE_KERNEL.get(wl) == kname:
                full = {"kernel": "butterfly", "device_kernel": kname, "workload": wl,
                        "kernel_source_sha1": kernel_source_hash(kname)}
                full.update(rec)
                with open(counters_path(wl), "w") as f:
                    json.dump(full, f, indent=1)
                    f.write("\n")
        rows.append((label, kname, ms, rec))
    L = ["rocprofv3 counters per dispatch: bytes moved past L2, by request size (no calibration factor)",
         "",
         "commands (repository root, on the MI355X machine), one run per target and pass:",
         *("  " + c for c in profile_commands(d)[:1]),
         "  timeout -s KILL 300 rocprofv3 --pmc <pass counters> -f csv -d <dir>/<target>_<pass> -o c "
         "-- python -u bench.py <target args>",
         "passes:",
         *(f"  {pn:5s} {' '.join(c)}" for pn, c in PROFILE_PASSES.items()),
         "targets:",
         *(f"  {lb:12s} {k:22s} bench.py {' '.join(a)}" for lb, (k, a) in PROFILE_TARGETS.items()),
         f"reduced by: python bench.py --report-counters {d} --out {os.path.relpath(out_txt, ROOT)}",
         "",
         "read bytes  = 32 n(32 B) + 64 n(64 B) + 128 n(128 B) requests (TCC_EA0_RDREQ_{32B,64B,128B});",
         "  'sizes/all' = their count over all read requests (TCC_EA0_RDREQ): 1 means no request is",
         "  left out; 'DRAM-side' = 32 x TCC_EA0_RDREQ_DRAM_32B, the same reads counted by the",
         "  memory side in 32-byte units (the MALL is on that side: its hits are included);",
         "written bytes = 32 (all - n64) + 64 n64 (TCC_EA0_WRREQ, TCC_EA0_WRREQ_64B; atomics travel",
         "  over the same interface and count here);",
         "GB/s = (read + written) / the launch time of the same run (HIP events; under the profiler)",
         "",
         f"{'target':12s} {'kernel':22s} {'read GB':>10s} {'sizes/all':>9s} {'DRAM-side':>10s} "
         f"{'written GB':>10s} {'ms':>8s} {'GB/s':>7s} {'L2 hit':>6s} {'L2 req/load':>11s}"]
    for label, kname, ms, r in rows:
        gbps = (r["egress_bytes_per_launch"] / (ms * 1e-3) / 1e9) if ms else None
        L.append(f"{label:12s} {kname:22s} {_fmt_bytes(r['bytes_read'])} "
                 f"{r['read_sizes_cover_all_requests']:9.4f} {_fmt_bytes(r['bytes_read_dram_side'])} "
                 f"{_fmt_bytes(r['bytes_written'])} {ms if ms else float('nan'):8.3f} "
                 f"{gbps if gbps else float('nan'):7.0f} "
                 f"{r.get('tcc_hit_rate', float('nan')):6.3f} "
                 f"{r.get('l2_requests_per_load', float('nan')):11.2f}")
    with open(out_txt, "w") as f:
        f.write("\n".join(L) + "\n")
    print("\n".join(L))
    return 0


def report_trace(d: str, bench_log: str, out_txt: str) -> int:
    """profiles/kernel_trace_bench.txt: rocprofv3's kernel statistics of the
    default bench run, beside the HIP-event averages bench.py measured for
    the same launches."""
    stats = glob.glob(os.path.join(d, "*kernel_stats.csv"))
    if not stats:
        raise SystemExit(f"no kernel_stats.csv in {d}")
    with open(stats[0]) as f:
        rows = list(csv.DictReader(f))
    head = _bench_lines(bench_log)[-1]
    L = ["rocprofv3 kernel trace of the default benchmark run (every workload, every kernel)",
         "",
         "command (repository root, on the MI355X machine):",
         f"  {profile_commands(d)[-1]}",
         f"reduced by: python bench.py --report-trace {d} --bench-log {bench_log} "
         f"--out {os.path.relpath(out_txt, ROOT)}",
         "",
         f"{'kernel':70s} {'calls':>6s} {'avg ms':>9s} {'min ms':>9s} {'max ms':>9s}"]
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
        name = r["Name"].replace("(anonymous namespace)::", "")
        short = (name[5:] if name.startswith("void ") else name).split("(")[0]
        L.append(f"{short[:70]:70s} {int(r['Calls']):6d} {float(r['AverageNs']) / 1e6:9.4f} "
                 f"{float(r['MinNs']) / 1e6:9.4f} {float(r['MaxNs']) / 1e6:9.4f}")
    L += ["", "bench.py's HIP-event averages in the same run (ms per launch):"]
    for r in head["results"]:
        L.append(f"  {r['workload']:20s} {r['kernel']:16s} {r['ms_per_launch']:9.4f}")
    for w, f_ in head["floor"].items():
        L.append(f"  {w:20s} {'floor (best)':16s} {f_['ms']:9.4f}  ({f_['shape']})")
    with open(out_txt, "w") as f:
        f.write("\n".join(L) + "\n")
    print("\n".join(L))
    return 0


def report_bench(log: str, out_txt: str) -> int:
    """profiles/bench_roofline_parity.txt: the default run's JSON line --
    roofline, floors, ceilings, parity on every workload, CPU baseline."""
    r = _bench_lines(log)[-1]
    ro = r["roofline"]
    L = ["The default benchmark run: roofline against the draw's memory floor, ceilings, parity",
         "",
         "command (repository root, on the MI355X machine):",
         f"  python -u bench.py > {log}",
         f"reduced by: python bench.py --report-bench {log} --out {os.path.relpath(out_txt, ROOT)}",
         "",
         f"headline {r['config']['workload']} (N={r['config']['N']:,}, K={r['config']['K']}): "
         f"{r['value'] / 1e9:.3f} G draws/s, {r['ms_per_step']:.3f} ms per step",
         f"  roofline: achieved {ro['achieved']:,.0f} GB/s (algorithmic bytes / draw time), "
         f"peak {ro['peak']:,.0f} GB/s (the same bytes / floor time), frac {ro['frac']:.3f}",
         f"  bytes past L2 per launch (counters): "
         + (f"{ro['traffic'] / 1e9:.2f} GB = {ro['traffic_GBps']:,.0f} GB/s"
            if ro.get("traffic") else "null (no counter record for the current source)"),
         f"  effective {r['effective_GBps']:,.0f} GB/s = {r['effective_frac_of_hbm_peak']:.2f} x "
         f"the {r['hbm_peak_GBps']:,.0f} GB/s HBM peak (L2 and the MALL serve re-read rows)",
         "",
         "floors (memory-only probe of the same access pattern, fastest launch shape; 'routed': "
         "the probe over the routed arrays, in the routed draw's workgroup order):"]
    for w, f in r["floor"].items():
        L.append(f"  {w:25s} floor {f['ms']:8.4f} ms ({f['shape']})  draw {f['draw_ms']:8.4f} ms  "
                 f"floor/draw {f['frac_of_floor']:.3f}")
    shapes = r.get("floors", {})
    for w, f in shapes.items():
        L.append(f"  {w:25s} shapes: " + ", ".join(f"{k} {v:.4f}" for k, v in f["shapes_ms"].items()))
    c = r["ceilings"]
    L += ["", "ceilings measured in the same run:",
          f"  streaming read from HBM   {c['hbm_read_GBps']:8,.0f} GB/s  ({c['hbm_read']})",
          f"  streaming read, MALL      {c['mall_read_GBps']:8,.0f} GB/s  ({c['mall_read']})",
          f"  device copy (read+write)  {c['device_copy_GBps']:8,.0f} GB/s",
          "", f"topic counts (lda_count_topics, _docs, _indexed; word-index: the index build; "
          f"sweep: lda_draw_butterfly then lda_count_topics_indexed on one stream) ms per call: " +
          ", ".join(f"{k} {v:.4f}" for k, v in r["count_topics_ms"].items()),
          "", "parity on every token against the oracle (band |u S - S_k| <= 1e-5 S; 'not "
          "admitted': in-band mismatches at a topic whose prefix range does not come within "
          "the band of u S):",
          f"  {'workload':28s} {'tokens':>10s} {'mismatches':>10s} {'rate':>9s} "
          f"{'outside band':>12s} {'not admitted':>12s} {'in-band rate':>12s}"]
    for w, p in r["parity"].items():
        na = p.get("mismatches_not_admitted")
        L.append(f"  {w:28s} {p['tokens']:10d} {p['mismatches']:10d} {p['mismatch_rate']:9.2e} "
                 f"{p['mismatches_outside_band']:12d} {'-' if na is None else na:>12} "
                 f"{p['in_band_rate']:12.2e}")
    b = r["cpu_baseline"]
    L += ["", f"CPU baseline (the oracle, {b['cores']} threads, {b.get('cpu', '')}): "
              f"{b['value'] / 1e6:.1f} M draws/s on {b['sample']}; one thread "
              f"{b['single_thread']['value'] / 1e6:.2f} M draws/s ({b['single_thread']['sample']})"]
    with open(out_txt, "w") as f:
        f.write("\n".join(L) + "\n")
    print("\n".join(L))
    return 0


def report_jsonl(log: str, out_txt: str, title: str, command: str) -> int:
    """A table of the JSON lines a bench.py mode printed (one row per line,
    one column per numeric field)."""
    lines = _bench_lines(log)
    if not lines:
        raise SystemExit(f"no JSON lines in {log}")
    keys = []
    for r in lines:
        for k, v in r.items():
            if k not in keys and (isinstance(v, (int, float)) or k == "workload"):
                keys.append(k)
    L = [title, "", "command (repository root, on the MI355X machine):", f"  {command} > {log}",
         f"reduced by: python bench.py --report-jsonl {log} --out {os.path.relpath(out_txt, ROOT)} "
         "--title ... --command ...", ""]
    for r in lines:
        L.append(r.get("workload", "") + ":")
        for k in keys:
            if k == "workload" or k not in r:
                continue
            v = r[k]
            L.append(f"  {k:40s} {v:.6g}" if isinstance(v, float) else f"  {k:40s} {v}")
    with open(out_txt, "w") as f:
        f.write("\n".join(L) + "\n")
    print("\n".join(L))
    return 0


_PARITY_LINE = re.compile(r"^\[parity\] (?P<case>.+?): n=(?P<n>\d+) mismatches=(?P<mis>\d+) "
                          r"\((?P<rate>[^)]+)\) hard=(?P<hard>\d+) in_band=(?P<band>\d+) "
                          r"\((?P<brate>[^)]+)\)")


def report_parity(log: str, out_txt: str, command: str) -> int:
    """A table of the parity lines the GPU tests print ("[parity] <workload>
    <kernel>: n=... mismatches=... hard=... in_band=..."), for the named
    workloads (the five, the corpus shaped like the paper's, and the
    16.8M-token corpus at other K), every kernel, in the order the tests
    ran."""
    from paper_1505_03851_amd.inputs import CONFIGS
    rows = []
    with open(log, errors="replace") as f:
        for ln in f:
            m = _PARITY_LINE.match(ln.strip())
            name = m["case"].split()[0] if m else ""
            if m and (name in CONFIGS or name.startswith("corpus16M-sweep-K")):
                rows.append(m)
    if not rows:
        raise SystemExit(f"no parity lines for the named workloads in {log}")
    L = ["Parity of every kernel on every token of the named workloads, against the oracle: "
         "mismatches, their rate, 'hard' (outside the band |u S - S_k| <= 1e-5 S, or in it at a "
         "topic the band does not admit: must be 0) and the tokens in the band",
         "", "command (repository root, on the MI355X machine):", f"  {command} > {log}",
         f"reduced by: python bench.py --report-parity {log} --out "
         f"{os.path.relpath(out_txt, ROOT)} --command ...", "",
         f"  {'workload and kernel':44s} {'tokens':>10s} {'mismatches':>10s} {'rate':>9s} "
         f"{'hard':>5s} {'in band':>8s} {'band rate':>9s}"]
    for m in rows:
        L.append(f"  {m['case']:44s} {int(m['n']):10d} {int(m['mis']):10d} {m['rate']:>9s} "
                 f"{int(m['hard']):5d} {int(m['band']):8d} {m['brate']:>9s}")
    with open(out_txt, "w") as f:
        f.write("\n".join(L) + "\n")
    print("\n".join(L))
    return 0


def floor_configs(K: int):
    """Launch shapes of the floor probe tried for K: window 8 or 16, 2 or 4
    wavefronts per workgroup, no occupancy cap or the draw's."""
    wpg, wpc = draw_occupancy(K)
    return [(w, g, c) for w in (8, 16) for g in (2, 4) for c in (0, wpc)]


def measure_floor(name: str, c, dev, steps: int, warmup: int) -> dict:
    """The memory-only floor of the draw on this workload: every launch shape
    of ``floor_configs`` timed, the fastest kept."""
    shapes = {}
    for cfg in floor_configs(c.K):
        dev["floor_cfg"] = cfg
        r = measure(name, c, dev, "floor", steps, warmup)
        r.pop("z")
        shapes["w{}-g{}-c{}".format(*cfg)] = r["ms_per_launch"]
    best = min(shapes, key=shapes.get)
    dev.pop("floor_cfg")
    return {"ms_per_launch": shapes[best], "shape": best, "shapes_ms": shapes,
            "alg_GBps": algorithmic_bytes(c) / (shapes[best] * 1e-3) / 1e9}


def measure_routed_floor(name: str, c, dev, steps: int, warmup: int) -> dict:
    """The memory-only floor of the routed draw: the floor probe over the
    routing's own arrays (each routed position's document, word and uniform),
    laid out so that probe workgroup b takes tile b div 8 of list b mod 8, as
    routed workgroup b does, so every list stays on its XCD; 2 or 4
    wavefronts per workgroup (the routed draw uses one of them) and windows of
    8 or 16 tokens, the fastest kept.  Workgroups past a list's end read its
    last position again, where the draw's simply exit."""
    import torch
    import paper_1505_03851_amd as lda
    th, ph, d, w, u = (dev["theta"], dev["phi"], dev["doc_id"], dev["word_id"], dev["u"])
    if "route" not in dev:
        dev["route"] = lda.route_build(d, w, th.shape[0], ph.shape[0])
    route = dev["route"]
    a = route.arrays()
    if min(route.length) == 0:
        raise ValueError("an empty routed list: no routed floor")
    start = torch.tensor(route.start, dtype=torch.int64, device=d.device)
    length = torch.tensor(route.length, dtype=torch.int64, device=d.device)
    shapes = {}
    for wpb in (2, 4):
        tile = wpb * 64
        tiles = -(-max(route.length) // tile)
        b = torch.arange(8 * tiles, device=d.device)
        x, t = b % 8, b // 8
        off = t[:, None] * tile + torch.arange(tile, device=d.device)[None, :]
        pos = (start[x][:, None] + torch.minimum(off, (length[x] - 1)[:, None])).reshape(-1)
        probe_dev = {"theta": th, "phi": ph, "doc_id": a["rdoc"][pos], "word_id": a["rword"][pos],
                     "u": u[a["perm"][pos].long().clamp(min=0)]}
        for window in (8, 16):
            probe_dev["floor_cfg"] = (window, wpb, 0)
            _, per_ms, _ = time_kernel("floor", probe_dev, steps, warmup)
            ms = sum(per_ms) / len(per_ms)
            shapes[f"w{window}-g{wpb}-c0"] = ms
            print(f"[bench] {name} routed floor w{window}-g{wpb}: {ms:.3f} ms/launch",
                  file=sys.stderr, flush=True)
        del probe_dev, pos, off
    best = min(shapes, key=shapes.get)
    return {"ms_per_launch": shapes[best], "shape": best, "shapes_ms": shapes,
            "alg_GBps": algorithmic_bytes(c) / (shapes[best] * 1e-3) / 1e9}


def not_admitted(c, d, w, u, zg, z_ref, band) -> int:
    """In-band mismatches drawn at a topic the band does not admit.  In the
    band several topics are correct, but only those whose fp64 prefix range
    [S_{z-1}, S_z] comes within 1e-5 S of stop = u S (z = K - 1 also when stop
    lies past S_{K-1}; with S = 0 only K - 1)."""
    import numpy as np
    import oracle
    K = c.K
    bad = 0
    for i in np.nonzero((zg != z_ref) & band)[0]:
        S = oracle.prefix_np(c.theta[d[i]], c.phi[w[i]])
        total, k = S[-1], int(zg[i])
        if total == 0.0:
            bad += k != K - 1
            continue
        stop, tol = float(u[i]) * total, 1e-5 * total
        below = S[k - 1] if k > 0 else 0.0
        bad += not (below <= stop + tol and (S[k] >= stop - tol or k == K - 1))
    return int(bad)


def parity_report(c, z_gpu, ref=None) -> dict:
    """Every token of the GPU's z against the oracle: mismatches, and those
    outside the rounding band |u S - S_k| <= 1e-5 S (which must be 0)."""
    import oracle
    zg = z_gpu.cpu().numpy() if hasattr(z_gpu, "cpu") else z_gpu
    if ref is None:
        ref = oracle.draw(c.theta, c.phi, c.doc_id, c.word_id, c.u, with_band=True)
    z_ref, band = ref
    mism = zg != z_ref
    return {"tokens": int(c.N), "mismatches": int(mism.sum()),
            "mismatch_rate": float(mism.mean()) if c.N else 0.0,
            "mismatches_outside_band": int((mism & ~band).sum()),
            "mismatches_not_admitted": not_admitted(c, c.doc_id, c.word_id, c.u, zg,
                                                    z_ref, band),
            "in_band_rate": float(band.mean()) if c.N else 0.0}


def _brief(r: dict) -> dict:
    r = dict(r)
    r.pop("z", None)
    return r


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--cpu-sample", type=int, default=1 << 24,
                    help="tokens of the headline workload the oracle draws")
    ap.add_argument("--only", choices=KERNELS, default=None,
                    help="time one kernel on one workload (for profiling)")
    ap.add_argument("--workload", default=HEADLINE)
    ap.add_argument("--ceiling", choices=("mall", "hbm"), default=None,
                    help="time the streaming-read probe over 192 MiB x 8 passes "
                         "(the passes after the first served by the MALL) or 4 GiB "
                         "(HBM); one JSON line")
    ap.add_argument("--floor-config", default=None,
                    help="window,waves_per_group,waves_per_cu of the floor probe "
                         "(--only floor); default 16 and the draw's occupancy")
    ap.add_argument("--copy", action="store_true",
                    help="three plain 1 GiB device-to-device copies (a check of "
                         "the request-size counters: 2^30 bytes read, 2^30 written)")
    ap.add_argument("--k-sweep", action="store_true",
                    help="naive vs butterfly over K = 16, 48, ..., 240 on the "
                         "corpus shaped like the paper's evaluation corpus; one "
                         "JSON line per K")
    ap.add_argument("--graph", action="store_true",
                    help="launch overhead: draws launched one by one against the "
                         "same draws replayed from one captured HIP graph")
    ap.add_argument("--all-configs", action="store_true",
                    help="naive, transposed and butterfly (warm, and cold for the "
                         "butterfly) on every workload; one JSON line each")
    ap.add_argument("--route-sweep", action="store_true",
                    help="plain against routed draw on the 16.8M-token corpus at "
                         "K = 256 ... 2048; one JSON line per K")
    ap.add_argument("--floor-sweep", action="store_true",
                    help="each draw against its own floor on the 16.8M-token "
                         "corpus at K = 256 ... 2048; one JSON line per K")
    ap.add_argument("--floor-k", default=None,
                    help="with --floor-sweep: the topic counts to sweep (comma-separated)")
    ap.add_argument("--wiki", action="store_true",
                    help="with --floor-sweep: the corpus shaped like the paper's at "
                         "its eight K instead")
    ap.add_argument("--ablation", action="store_true",
                    help="time the block-table variants and the offsets form "
                         "of the documents; one JSON line per workload")
    ap.add_argument("--permuted-ids", action="store_true",
                    help="each workload with its word ids as generated and renamed by a "
                         "random permutation (phi's rows moved with them); one JSON line each")
    ap.add_argument("--wide-builds", action="store_true",
                    help="the default build of the draw kernels against the build "
                         "for tables past 4 GiB, on every workload; one JSON line each")
    ap.add_argument("--counters-summary", action="store_true",
                    help="write the counter record of the draw on --workload from "
                         "the csv directories of rocprofv3 counter passes (--reads, "
                         "--dram, optional --hitmiss) to --out")
    for opt in ("--reads", "--dram", "--hitmiss", "--out"):
        ap.add_argument(opt, default=None)
    ap.add_argument("--profile-commands", default=None, metavar="DIR",
                    help="print the rocprofv3 commands behind profiles/ (output to DIR)")
    ap.add_argument("--report-counters", default=None, metavar="DIR",
                    help="reduce the counter passes in DIR to --out (and the draw's "
                         "counter records under profiles/)")
    ap.add_argument("--report-trace", default=None, metavar="DIR",
                    help="reduce the kernel trace in DIR (with --bench-log) to --out")
    ap.add_argument("--bench-log", default=None)
    ap.add_argument("--report-bench", default=None, metavar="LOG",
                    help="summarise the default run's JSON line in LOG to --out")
    ap.add_argument("--report-jsonl", default=None, metavar="LOG",
                    help="tabulate the JSON lines in LOG to --out (--title, --command)")
    ap.add_argument("--report-parity", default=None, metavar="LOG",
                    help="tabulate the parity lines of a GPU test log (pytest -s) to --out")
    ap.add_argument("--title", default="")
    ap.add_argument("--command", default="")
    args = ap.parse_args()
    if args.counters_summary:
        return counters_summary(args)
    if args.profile_commands:
        print("\n".join(profile_commands(args.profile_commands)))
        return 0
    if args.report_counters:
        return report_counters(args.report_counters, args.out)
    if args.report_trace:
        return report_trace(args.report_trace, args.bench_log, args.out)
    if args.report_bench:
        return report_bench(args.report_bench, args.out)
    if args.report_jsonl:
        return report_jsonl(args.report_jsonl, args.out, args.title, args.command)
    if args.report_parity:
        return report_parity(args.report_parity, args.out, args.command)
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); "
              "the draw has no multi-GPU path (each GPU would draw its own "
              "document-aligned share of the tokens with no exchange).", file=sys.stderr)
        return 2

    import torch
    import paper_1505_03851_amd as lda
    from paper_1505_03851_amd.inputs import make_corpus

    lda.load()
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1

    if args.ceiling:
        nbytes, passes = {"mall": (MALL_PROBE_BYTES, MALL_PROBE_PASSES),
                          "hbm": (HBM_PROBE_BYTES, 1)}[args.ceiling]
        ms, gbps = read_ceiling(nbytes, passes, steps=args.steps)
        print(json.dumps({"ceiling": args.ceiling, "bytes": nbytes, "passes": passes,
                          "ms_per_launch_median": ms, "GBps": gbps}), flush=True)
        return 0

    if args.copy:
        n = 1 << 28                      # 1 GiB of float32
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": 4 * n, "copy_bytes_written": 4 * n,
                          "dispatches": 3}), flush=True)
        return 0

    if args.k_sweep:
        return k_sweep(args)
    if args.ablation:
        return ablation(args)
    if args.wide_builds:
        return wide_builds(args)
    if args.permuted_ids:
        return permuted_ids(args)
    if args.route_sweep:
        return route_sweep(args)
    if args.floor_sweep:
        return floor_sweep(args)
    if args.all_configs:
        return all_configs(args)
    if args.graph:
        return graph_timing(args)

    if args.only:
        c = make_corpus(args.workload)
        dev = upload(c)
        if args.floor_config:
            dev["floor_cfg"] = tuple(int(x) for x in args.floor_config.split(","))
        r = measure(args.workload, c, dev, args.only, args.steps, args.warmup)
        r.pop("z")
        print(json.dumps(r), flush=True)
        return 0

    steps, warmup = args.steps, args.warmup
    # ceilings of the memory system on this GPU
    hbm_ms, hbm_GBps = read_ceiling(HBM_PROBE_BYTES, 1)
    mall_ms, mall_GBps = read_ceiling(MALL_PROBE_BYTES, MALL_PROBE_PASSES)
    copy_GBps = device_copy_GBps()
    results, parity, floors, counts = [], {}, {}, {}

    # the small workloads: the draw, and its parity on every token
    for name in ("tiny-K32", "corpus1M-K64"):
        c = make_corpus(name)
        dev = upload(c)
        r = measure(name, c, dev, "butterfly", steps, warmup)
        parity[name] = parity_report(c, r["z"])
        results.append(_brief(r))
        del dev
    torch.cuda.empty_cache()

    # K = 64: the draw's floor
    c1 = make_corpus("corpus1M-K64")
    dev1 = upload(c1)
    d64 = measure(c1.name, c1, dev1, "butterfly", max(steps, 20), warmup)
    d64.pop("z")
    floors[c1.name] = measure_floor(c1.name, c1, dev1, max(steps, 20), warmup)
    floors[c1.name]["draw_ms"] = d64["ms_per_launch"]
    del dev1, c1
    torch.cuda.empty_cache()

    # K = 256: the draw against the naive and transposed kernels, its floor
    # and the topic counts of its draws
    c2 = make_corpus(SECOND)
    dev2 = upload(c2)
    second = measure(SECOND, c2, dev2, "butterfly", max(steps, 20), warmup)
    parity[SECOND] = parity_report(c2, second["z"])
    results.append(_brief(second))
    for k in ("transposed", "naive"):
        results.append(_brief(measure(SECOND, c2, dev2, k, max(steps, 20), warmup)))
    floors[SECOND] = measure_floor(SECOND, c2, dev2, max(steps, 20), warmup)
    floors[SECOND]["draw_ms"] = second["ms_per_launch"]
    for k in ("count", "count-docs", "count-indexed", "word-index", "sweep"):
        counts[f"{SECOND} {k}"] = measure(SECOND, c2, dev2, k, max(steps, 20),
                                          warmup)["ms_per_launch"]
    del dev2, c2
    torch.cuda.empty_cache()

    # K = 2048, Poisson document lengths: the draw (token order and routed)
    c5 = make_corpus("poisson300-K2048")
    dev5 = upload(c5)
    r = measure(c5.name, c5, dev5, "butterfly", steps, warmup)
    import oracle
    ref5 = oracle.draw(c5.theta, c5.phi, c5.doc_id, c5.word_id, c5.u, with_band=True)
    parity[c5.name] = parity_report(c5, r["z"], ref5)
    results.append(_brief(r))
    floors[c5.name] = measure_floor(c5.name, c5, dev5, steps, warmup)
    floors[c5.name]["draw_ms"] = r["ms_per_launch"]
    r = measure(c5.name, c5, dev5, "routed", steps, warmup)
    parity[c5.name + " routed"] = parity_report(c5, r["z"], ref5)
    results.append(_brief(r))
    floors[c5.name + " routed"] = measure_routed_floor(c5.name, c5, dev5, steps, warmup)
    floors[c5.name + " routed"]["draw_ms"] = r["ms_per_launch"]
    del dev5, c5, ref5
    torch.cuda.empty_cache()

    # the headline workload, K = 1024
    c = make_corpus(HEADLINE)
    dev = upload(c)
    results.append(_brief(measure(HEADLINE, c, dev, "naive", max(3, steps // 4), 1)))
    results.append(_brief(measure(HEADLINE, c, dev, "transposed", steps, warmup)))
    head = measure(HEADLINE, c, dev, "butterfly", steps, warmup)
    z_head = head.pop("z")
    results.append(head)
    # the same draw over tokens routed to the XCDs by word: routing built once
    # (as per corpus in a sampler), and built again in every step
    routed = {}
    for k in ("routed", "routed+build"):
        r = measure(HEADLINE, c, dev, k, steps, warmup)
        routed[k] = r.pop("z")
        r["differs_from_butterfly"] = int((routed[k] != z_head).sum())
        results.append(r)
        if k == "routed":
            floors[HEADLINE + " routed"] = measure_routed_floor(HEADLINE, c, dev, steps, warmup)
            floors[HEADLINE + " routed"]["draw_ms"] = r["ms_per_launch"]
    # the same launches with L2 and the MALL flushed before each (1 GiB fill)
    flush = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
    results.append(_brief(measure(HEADLINE, c, dev, "butterfly", steps, 1, flush=flush)))
    del flush
    floors[HEADLINE] = measure_floor(HEADLINE, c, dev, steps, warmup)
    floors[HEADLINE]["draw_ms"] = head["ms_per_launch"]
    for k in ("count", "count-docs", "count-indexed", "word-index", "sweep"):
        counts[f"{HEADLINE} {k}"] = measure(HEADLINE, c, dev, k, steps, warmup)["ms_per_launch"]

    base = cpu_baseline(c, z_head, args.cpu_sample)
    if base["parity"]["tokens"] == c.N:       # the baseline drew every token
        parity[HEADLINE] = base["parity"]
        ref4 = base.pop("_ref")
    else:
        base.pop("_ref")
        ref4 = oracle.draw(c.theta, c.phi, c.doc_id, c.word_id, c.u, with_band=True)
        parity[HEADLINE] = parity_report(c, z_head, ref4)
    parity[HEADLINE + " routed"] = parity_report(c, routed["routed"], ref4)
    del ref4

    wall = head["wall_s"]
    value = c.N * steps / wall
    fl = floors[HEADLINE]
    traffic = traffic_from_counters(HEADLINE)
    egress_GBps = traffic / (head["ms_per_launch"] * 1e-3) / 1e9 if traffic else None
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "draws/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": 1e3 * wall / steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": HEADLINE, "N": c.N, "M": c.M, "V": c.V,
                   "K": c.K, "kernel": "butterfly"},
        "roofline": {
            # memory-bound (HBM, with L2 and the MALL serving re-read rows);
            # the peak that binds is the memory system's rate for this access
            # pattern, measured by the floor probe, not the 8 TB/s datasheet
            # figure (reported beside it as hbm_peak_GBps)
            "bound": "hbm",
            "achieved": head["alg_GBps"],
            "peak": fl["alg_GBps"],
            "unit": "GB/s",
            "frac": fl["ms_per_launch"] / head["ms_per_launch"],
            "traffic": traffic,
            "peak_kind": "measured in this run: the launch's algorithmic bytes over the "
                         "time of the memory-only probe that moves them in the same token "
                         "order (lda_probe_draw_floor, fastest of its launch shapes)",
            "traffic_GBps": egress_GBps,
        },
        # algorithmic bytes over time: above the HBM peak, because L2 and the
        # MALL serve the re-read rows of Zipf-frequent words
        "effective_GBps": head["alg_GBps"],
        "effective_frac_of_hbm_peak": head["alg_GBps"] / PEAK_HBM_GBPS,
        "hbm_peak_GBps": PEAK_HBM_GBPS,
        "l2_egress_GBps": egress_GBps,
        "ceilings": {"hbm_read_GBps": hbm_GBps, "mall_read_GBps": mall_GBps,
                     "device_copy_GBps": copy_GBps,
                     "hbm_read": f"{HBM_PROBE_BYTES >> 20} MiB read once (lda_probe_read)",
                     "mall_read": f"{MALL_PROBE_BYTES >> 20} MiB read {MALL_PROBE_PASSES} "
                                  "times per launch (lda_probe_read)"},
        "floor": {w: {"ms": f["ms_per_launch"], "shape": f["shape"],
                      "draw_ms": f["draw_ms"],
                      "frac_of_floor": f["ms_per_launch"] / f["draw_ms"]}
                  for w, f in floors.items()},
        "second": {"workload": SECOND, "draws_per_s": second["draws_per_s"],
                   "ms_per_launch": second["ms_per_launch"],
                   "effective_GBps": second["alg_GBps"],
                   "frac_of_floor": floors[SECOND]["ms_per_launch"] / second["ms_per_launch"]},
        "count_topics_ms": counts,
        "parity": parity,
        "cpu_baseline": base,
        "results": results,
        "floors": floors,
        "kernel_source_sha1": {k: kernel_source_hash(k) for k in KERNEL_SOURCES},
    }
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
