"""The measurement logic of bench.py, on the CPU: the algorithmic bytes the
roofline divides by, the source hash that decides whether a counter record
still applies, and the reducer of the GPU tests' parity lines."""
import os
import shutil
import sys
from types import SimpleNamespace

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_algorithmic_bytes_by_hand():
    # 5 tokens, K = 8: documents 0 0 1 1 0 are three runs of one document
    c = SimpleNamespace(N=5, K=8, doc_id=np.array([0, 0, 1, 1, 0], np.int32))
    assert bench.algorithmic_bytes(c) == 5 * (4 * 8 + 16) + 3 * 4 * 8
    c0 = SimpleNamespace(N=0, K=8, doc_id=np.zeros(0, np.int32))
    assert bench.algorithmic_bytes(c0) == 0


def test_algorithmic_bytes_of_the_headline_workload():
    # 65,536 documents of 256 tokens at K = 1024: 4,112 B per token and
    # 4,096 B per document, 69,256,347,648 B per launch
    doc = np.repeat(np.arange(65536, dtype=np.int32), 256)
    c = SimpleNamespace(N=doc.size, K=1024, doc_id=doc)
    assert bench.algorithmic_bytes(c) == 69_256_347_648


def test_source_hash_ignores_comments_and_spacing_only(tmp_path, monkeypatch):
    src = tmp_path / "csrc"
    shutil.copytree(bench.CSRC, src)
    monkeypatch.setattr(bench, "CSRC", str(src))
    h0 = bench.kernel_source_hash("leaf_eighths_kernel")
    f = src / "tuning.hpp"
    text = f.read_text()
    f.write_text("// a new line of comment\n" + text.replace("\n", "\n\n", 3) +
                 "\n/* a block\n   comment */\n")
    assert bench.kernel_source_hash("leaf_eighths_kernel") == h0
    f.write_text(text.replace("#define LDA_EIGHTHS_WINDOW 16", "#define LDA_EIGHTHS_WINDOW 8"))
    assert bench.kernel_source_hash("leaf_eighths_kernel") != h0


def test_committed_counter_records_match_the_source():
    # the bench's roofline.traffic is null once the headline kernel's code
    # changed after its counters were taken: retake them with the kernel
    for workload in (bench.HEADLINE, bench.SECOND):
        assert bench.traffic_from_counters(workload) is not None, workload


def test_report_parity_keeps_the_named_workloads(tmp_path):
    log = tmp_path / "parity.log"
    log.write_text(
        "tests/test_x.py ..\n"
        "[parity] corpus16M-K1024 routed philox: n=16777216 mismatches=46 (2.74e-06) "
        "hard=0 in_band=14818 (8.83e-04)\n"
        "[parity] random-N5 butterfly: n=5 mismatches=0 (0.00e+00) hard=0 in_band=0 "
        "(0.00e+00)\n")
    out = tmp_path / "parity.txt"
    assert bench.report_parity(str(log), str(out), "cmd") == 0
    text = out.read_text()
    assert "corpus16M-K1024 routed philox" in text and "16777216" in text
    assert "random-N5" not in text
