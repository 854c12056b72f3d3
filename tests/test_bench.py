"""Host logic of bench.py (CPU): the comment-insensitive kernel hash that keys
the committed HBM-traffic summary, the summary lookup, and the refusal of
more than one GPU."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_kernel_hash_ignores_comments_trailing_blanks_and_blank_lines():
    code = "int a = 1;\nint b = a + 2;\n"
    commented = "// header\nint a = 1;   // one\n\n   \nint b = a + 2;  \n// trailer\n"
    assert bench.kernel_sha256(code) == bench.kernel_sha256(commented)
    assert bench.kernel_sha256(code) != bench.kernel_sha256("int a = 1;\nint b = a + 3;\n")
    # indentation is code
    assert bench.kernel_sha256(code) != bench.kernel_sha256("int a = 1;\n  int b = a + 2;\n")


def test_kernel_hash_covers_the_kernel_source_and_its_header():
    texts = []
    for path in (bench.KERNEL_SRC, bench.KERNEL_HDR):
        with open(path, encoding="utf-8") as f:
            texts.append(f.read())
    assert bench.kernel_sha256() == bench.kernel_sha256("\n".join(texts))
    assert bench.kernel_sha256() != bench.kernel_sha256(texts[0])  # the header's constants count


def _traffic_file(path, sha, hbm="123456789"):
    path.write_text("# a comment line: with a colon\n"
                    "workload: gpt_1p3b world 1 rank 0 d=0.01\n"
                    f"kernel_source_sha256: {sha}\n"
                    f"hbm_bytes_per_launch: {hbm}\n")


def test_traffic_is_reported_only_for_the_kernel_it_was_measured_on(tmp_path, monkeypatch):
    src = tmp_path / "kernel.hip"
    src.write_text("__global__ void k() {}\n")
    hdr = tmp_path / "kernel.h"
    hdr.write_text("constexpr int kTile = 1024;\n")
    traffic = tmp_path / "traffic.txt"
    monkeypatch.setattr(bench, "KERNEL_SRC", str(src))
    monkeypatch.setattr(bench, "KERNEL_HDR", str(hdr))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(traffic))
    assert bench.read_traffic() is None  # no summary
    _traffic_file(traffic, bench.kernel_sha256())
    assert bench.read_traffic() == 123456789.0
    src.write_text("// the same code, commented\n__global__ void k() {}  // empty\n")
    assert bench.read_traffic() == 123456789.0
    src.write_text("__global__ void k() { int x = 0; }\n")
    assert bench.read_traffic() is None  # the code changed: the counters are stale
    src.write_text("__global__ void k() {}\n")
    assert bench.read_traffic() == 123456789.0
    hdr.write_text("constexpr int kTile = 2048;\n")
    assert bench.read_traffic() is None  # a constant of the header changed
    _traffic_file(traffic, bench.kernel_sha256(), hbm="not a number")
    assert bench.read_traffic() is None


@pytest.mark.parametrize("path,values", [("TRAFFIC_FILE", 1_315_723_264), ("TRAFFIC_FILE_BERT", 41_892_736)])
def test_committed_traffic_summaries_name_a_hash_and_a_byte_count(path, values):
    fields = {}
    for line in open(getattr(bench, path)):
        if ":" in line and not line.startswith("#"):
            key, val = line.split(":", 1)
            fields[key.strip()] = val.strip()
    assert len(fields["kernel_source_sha256"]) == 64
    assert float(fields["hbm_bytes_per_launch"]) > 12 * values  # at least the algorithmic bytes


@pytest.mark.parametrize("n", ["2", "8"])
def test_more_than_one_gpu_is_refused(n):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", n],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "not supported" in r.stderr and "one GPU" in r.stderr
    assert r.stdout == ""
