#!/usr/bin/env python3
"""Benchmark of the per-token LDA topic draw on one MI355X.

One step = one launch of the draw over every token of the workload (all inputs
resident in HBM).  The headline workload is the K=1024 corpus (N=16,777,216
tokens, M=65,536 documents x 256, V=100,000 Zipf(1.05) words); the K=256
corpus and the naive kernel are reported beside it.

Prints ONE JSON line.  ``roofline.achieved`` is the algorithmic bytes of one
launch divided by the launch's average duration (HIP events on the launch
stream); ``roofline.traffic`` is the HBM traffic per launch taken from the
committed rocprofv3 counter summary, or null when the kernel source changed
since the counters were collected.
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("z draws/sec and achieved HBM GB/s (% of peak) at K=256 and K=1024, "
          "1 MI355X")
PEAK_HBM_GBPS = 8000.0            # MI355X HBM3E, published
HEADLINE = "corpus16M-K1024"
# the device kernel lda_draw_butterfly launches on the headline workload
HEADLINE_KERNEL = "leaf_eighths_kernel"
SECOND = "corpus1M-K256"
COUNTERS = os.path.join(ROOT, "profiles", "butterfly_corpus16M-K1024_counters.json")
KERNEL_SOURCES = sorted(glob.glob(os.path.join(ROOT, "paper_1505_03851_amd", "csrc", "*.[hc]*")))


def kernel_source_hash() -> str:
    h = hashlib.sha1()
    for p in KERNEL_SOURCES:
        with open(p, "rb") as f:
            h.update(f.read())
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
           "variant-register", "variant-lds", "variant-lds_alt", "variant-leaf8", "philox",
           "routed",
           "routed+build", "routed-philox")
PHILOX_SEED = 0x5EED20150513


def launcher(kernel: str, dev):
    """A function (out, stream) that launches ``kernel`` once over ``dev``.
    "routed" draws the tokens routed to the XCDs with the routing built once
    beforehand (as a sampler does once per corpus); "routed+build" builds the
    routing again in every launch (one stream synchronisation inside)."""
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


def measure(name: str, c, dev, kernel: str, steps: int, warmup: int, flush=None) -> dict:
    wall, per_ms, z = time_kernel(kernel, dev, steps, warmup, flush)
    avg_ms = sum(per_ms) / len(per_ms)
    srt = sorted(per_ms)
    med_ms = srt[len(srt) // 2]
    b_alg = algorithmic_bytes(c)
    gbps = b_alg / (avg_ms * 1e-3) / 1e9
    tag = " cold" if flush is not None else ""
    print(f"[bench] {name} {kernel}{tag}: {avg_ms:.3f} ms/launch "
          f"(median {med_ms:.3f}, min {srt[0]:.3f}, max {srt[-1]:.3f}), "
          f"{c.N / (avg_ms * 1e-3) / 1e9:.3f} G draws/s, "
          f"{gbps:.0f} GB/s algorithmic ({100 * gbps / PEAK_HBM_GBPS:.1f}% of "
          f"8 TB/s)", file=sys.stderr, flush=True)
    return {
        "workload": name, "kernel": kernel + ("-cold" if flush is not None else ""),
        "N": c.N, "K": c.K, "steps": steps, "wall_s": wall,
        "ms_per_launch": avg_ms, "ms_per_launch_median": med_ms,
        "ms_per_launch_min": srt[0], "ms_per_launch_max": srt[-1],
        "draws_per_s": c.N / (avg_ms * 1e-3),
        "alg_bytes_per_launch": b_alg,
        "alg_GBps": gbps, "frac_of_hbm_peak": gbps / PEAK_HBM_GBPS,
        "z": z,
    }


def device_copy_GBps(steps: int = 10) -> float:
    """Bytes read plus bytes written per second by a plain 1 GiB device copy
    (torch's copy kernel, HIP events): the practical HBM ceiling on the box."""
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


def traffic_from_counters():
    """HBM bytes per launch from the committed counter summary, if it was
    taken on the current kernel source."""
    try:
        with open(COUNTERS) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_sha1") != kernel_source_hash():
        return None
    return rec.get("hbm_bytes_per_launch")


def _counter_means(d: str, kernel_substr: str) -> dict:
    """Mean per-dispatch value of each counter in a rocprofv3 --pmc csv
    directory, over the dispatches whose kernel name contains
    ``kernel_substr`` (per-dispatch values are summed over instances)."""
    import csv
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
    return {k: sum(v) / len(v) for k, v in out.items()}


def counters_summary(args) -> int:
    """Turn rocprofv3 counter runs of the draw's kernel (dispatches whose name
    contains ``--kernel-name``) and of the 1 GiB copy into the record
    ``traffic_from_counters`` reads."""
    kname = args.kernel_name
    copy = "copyBuffer"
    fetch = _counter_means(args.fetch, kname)["FETCH_SIZE"]
    write = _counter_means(args.write, kname)["WRITE_SIZE"]
    copy_fetch = _counter_means(args.copy_fetch, copy)["FETCH_SIZE"]
    copy_write = _counter_means(args.copy_write, copy)["WRITE_SIZE"]
    copy_kib = (1 << 30) / 1024
    f_scale, w_scale = copy_kib / copy_fetch, copy_kib / copy_write
    rec = {
        "kernel": "butterfly", "device_kernel": kname, "workload": args.workload,
        "kernel_source_sha1": kernel_source_hash(),
        "fetch_kib_per_dispatch": fetch, "write_kib_per_dispatch": write,
        "copy_1GiB_fetch_kib": copy_fetch, "copy_1GiB_write_kib": copy_write,
        "fetch_scale": f_scale, "write_scale": w_scale,
        "hbm_bytes_per_launch": 1024 * (fetch * f_scale + write * w_scale),
    }
    if args.hitmiss:
        hm = _counter_means(args.hitmiss, kname)
        rec["tcc_hit_per_dispatch"] = hm["TCC_HIT_sum"]
        rec["tcc_miss_per_dispatch"] = hm["TCC_MISS_sum"]
        rec["tcc_hit_rate"] = hm["TCC_HIT_sum"] / (hm["TCC_HIT_sum"] + hm["TCC_MISS_sum"])
    with open(args.out, "w") as f:
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
            r = measure(c.name, c, dev, kernel, args.steps, args.warmup)
            z = r.pop("z")
            if z_bf is None:
                z_bf = z
            else:
                rec[kernel + "_differs_from_butterfly"] = int((z != z_bf).sum())
            rec[kernel + "_ms"] = r["ms_per_launch"]
        rec["routed_speedup"] = rec["butterfly_ms"] / rec["routed_ms"]
        rec["routed_build_speedup"] = rec["butterfly_ms"] / rec["routed+build_ms"]
        print(json.dumps(rec), flush=True)
        del dev, c
        torch.cuda.empty_cache()
    return 0


def ablation(args) -> int:
    """The table variants of Section 4 (the paper's rule with the table in
    registers or LDS, the alternative rule in LDS), 8-topic leaves, the offsets form of the
    documents, the document-per-lane driver, the draw with in-kernel
    uniforms and the default dispatch, on the two corpora and the corpus
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
                   "variant-leaf8", "docs", "doc_lanes"] + \
                  (["doc_lanes_cache"] if c.K <= 256 else []) + ["philox"]
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
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run plain 1 GiB device-to-device copies (the "
                         "reference for scaling HBM counters)")
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
    ap.add_argument("--ablation", action="store_true",
                    help="time the block-table variants and the offsets form "
                         "of the documents; one JSON line per workload")
    ap.add_argument("--counters-summary", action="store_true",
                    help="write the HBM-traffic record from rocprofv3 csv "
                         "directories (--fetch, --write, --copy-fetch, "
                         "--copy-write, optional --hitmiss) to --out")
    for opt in ("--fetch", "--write", "--copy-fetch", "--copy-write",
                "--hitmiss"):
        ap.add_argument(opt, default=None)
    ap.add_argument("--out", default=COUNTERS)
    ap.add_argument("--kernel-name", default=HEADLINE_KERNEL,
                    help="substring of the device kernel's name in the counter "
                         "csv files (--counters-summary)")
    args = ap.parse_args()
    if args.counters_summary:
        return counters_summary(args)
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); "
              "the draw has no multi-GPU path in this build.", file=sys.stderr)
        return 2

    import torch
    import paper_1505_03851_amd as lda
    from paper_1505_03851_amd.inputs import make_corpus

    lda.load()
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1

    if args.copy_calibration:
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
    if args.route_sweep:
        return route_sweep(args)
    if args.all_configs:
        return all_configs(args)
    if args.graph:
        return graph_timing(args)

    if args.only:
        c = make_corpus(args.workload)
        dev = upload(c)
        r = measure(args.workload, c, dev, args.only, args.steps, args.warmup)
        r.pop("z")
        print(json.dumps(r), flush=True)
        return 0

    results = []
    c2 = make_corpus(SECOND)
    dev2 = upload(c2)
    for k in ("butterfly", "transposed", "naive"):
        r = measure(SECOND, c2, dev2, k, max(args.steps, 20), args.warmup)
        r.pop("z")
        results.append(r)
    del dev2, c2
    torch.cuda.empty_cache()

    c = make_corpus(HEADLINE)
    dev = upload(c)
    naive = measure(HEADLINE, c, dev, "naive", max(3, args.steps // 4), 1)
    naive.pop("z")
    results.append(naive)
    tr = measure(HEADLINE, c, dev, "transposed", args.steps, args.warmup)
    tr.pop("z")
    results.append(tr)
    head = measure(HEADLINE, c, dev, "butterfly", args.steps, args.warmup)
    z_head = head.pop("z")
    results.append(head)
    # the same draw over tokens routed to the XCDs by word: routing built once
    # (as per corpus in a sampler), and built again in every step
    for k in ("routed", "routed+build"):
        r = measure(HEADLINE, c, dev, k, args.steps, args.warmup)
        r["differs_from_butterfly"] = int((r.pop("z") != z_head).sum())
        results.append(r)
    # the same launches with L2 and the MALL flushed before each (1 GiB fill)
    flush = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
    cold = measure(HEADLINE, c, dev, "butterfly", args.steps, 1, flush=flush)
    cold.pop("z")
    results.append(cold)
    del flush

    wall = head["wall_s"]
    value = c.N * args.steps / wall
    traffic = traffic_from_counters()
    copy_GBps = device_copy_GBps()
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "draws/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": 1e3 * wall / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": HEADLINE, "N": c.N, "M": c.M, "V": c.V,
                   "K": c.K, "kernel": "butterfly"},
        "roofline": {
            "bound": "hbm",
            "achieved": head["alg_GBps"],
            "peak": PEAK_HBM_GBPS,
            "unit": "GB/s",
            "frac": head["alg_GBps"] / PEAK_HBM_GBPS,
            "traffic": traffic,
        },
        # the counted bytes that leave L2 (FETCH_SIZE + WRITE_SIZE, scaled by
        # a plain copy) per launch, over the measured launch time
        "hbm_traffic_GBps": (traffic / (head["ms_per_launch"] * 1e-3) / 1e9
                             if traffic else None),
        "hbm_traffic_frac": (traffic / (head["ms_per_launch"] * 1e-3) / 1e9 /
                             PEAK_HBM_GBPS if traffic else None),
        # a plain 1 GiB device copy on the same GPU (bytes read + written per
        # second), and the counted L2 traffic of the draw against it
        "device_copy_GBps": copy_GBps,
        "hbm_traffic_frac_of_copy": (traffic / (head["ms_per_launch"] * 1e-3) / 1e9 /
                                     copy_GBps if traffic else None),
        "cpu_baseline": cpu_baseline(c, z_head, args.cpu_sample),
        "results": results,
        "kernel_source_sha1": kernel_source_hash(),
    }
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
