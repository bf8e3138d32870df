"""Host logic of bench.py: the counter summaries it reads count only while
their source hash is the current kernel source's, and a request for more than
one GPU ends with a message."""
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def write(path, lines):
    path.write_text("\n".join(lines) + "\n")
    return str(path)


def test_traffic_needs_the_current_source(tmp_path, monkeypatch):
    body = ["# summary", "fetch_kib_per_dispatch: 1.0", "hbm_bytes_per_launch: 12345"]
    monkeypatch.setattr(bench, "PMC_FILE", write(tmp_path / "a.txt", ["source_hash: " + bench.source_hash()] + body))
    assert bench.measured_traffic() == 12345
    monkeypatch.setattr(bench, "PMC_FILE", write(tmp_path / "b.txt", ["source_hash: 0000000000000000"] + body))
    assert bench.measured_traffic() is None
    monkeypatch.setattr(bench, "PMC_FILE", str(tmp_path / "missing.txt"))
    assert bench.measured_traffic() is None


def test_valu_count_needs_the_current_source(tmp_path, monkeypatch):
    row = bench.HEADLINE_KERNEL + " | C3 | 4 | 58.5 | 94.3 | 0.032 | 0.0055 | 5.73 | 2048 | 181700798 | 0.590 | 4486061"
    other = "kendall_sort_kernel | C5 | 8 | 77.2 | 95.2 | 11.9 | 0.37 | 43.8 | 80000 | 1756487446 | 0.780 | 297487296"
    monkeypatch.setattr(bench, "UTIL_FILE", write(tmp_path / "a.txt", ["# x", "source_hash: " + bench.source_hash(), other, row]))
    assert bench.measured_valu() == 181700798
    monkeypatch.setattr(bench, "UTIL_FILE", write(tmp_path / "b.txt", ["source_hash: ffffffffffffffff", row]))
    assert bench.measured_valu() is None
    monkeypatch.setattr(bench, "UTIL_FILE", write(tmp_path / "c.txt", ["source_hash: " + bench.source_hash(), other]))
    assert bench.measured_valu() is None


def test_committed_summaries_parse():
    # whatever their hashes, the committed summaries have the fields bench.py reads
    for name, key in (("sim_c3_pmc.txt", "hbm_bytes_per_launch:"), ("kernel_util_counters.txt", bench.HEADLINE_KERNEL + " |")):
        text = open(os.path.join(ROOT, "profiles", name)).read()
        assert "source_hash:" in text and key in text


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""
