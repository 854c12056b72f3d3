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


@pytest.mark.parametrize("path,min_bytes", [
    ("TRAFFIC_FILE", 12 * 1_315_723_264),        # the step's 12 B per partition value
    ("TRAFFIC_FILE_BERT", 12 * 41_892_736),
    ("TRAFFIC_FILE_EF", 12 * 335_141_888),       # the full pass: 12 B per value of the vector
    ("TRAFFIC_FILE_SWEEP", 12 * 11_689_512),
    ("TRAFFIC_FILE_UNION", 16 * 3_351_416),      # gather and update of the BERT-large union
    ("TRAFFIC_FILE_TOPK", 12 * 41_892_736),      # top-k: at least the step's 12 B per value
])
def test_committed_traffic_summaries_name_a_workload_a_hash_and_a_byte_count(path, min_bytes):
    fields = {}
    for line in open(getattr(bench, path)):
        if ":" in line and not line.startswith("#"):
            key, val = line.split(":", 1)
            fields[key.strip()] = val.strip()
    assert fields["workload"]
    assert len(fields["kernel_source_sha256"]) == 64
    assert float(fields["hbm_bytes_per_launch"]) > min_bytes  # at least the algorithmic bytes


def test_traffic_is_reported_only_for_the_workload_it_was_measured_on(tmp_path, monkeypatch):
    src = tmp_path / "kernel.hip"
    src.write_text("__global__ void k() {}\n")
    hdr = tmp_path / "kernel.h"
    hdr.write_text("constexpr int kTile = 1024;\n")
    traffic = tmp_path / "traffic.txt"
    monkeypatch.setattr(bench, "KERNEL_SRC", str(src))
    monkeypatch.setattr(bench, "KERNEL_HDR", str(hdr))
    _traffic_file(traffic, bench.kernel_sha256())
    with open(traffic, "a") as f:
        f.write("workload: toy world 4 rank 0 d=0.01\n")
    assert bench.read_traffic(str(traffic), "toy world 4 rank 0 d=0.01") == 123456789.0
    assert bench.read_traffic(str(traffic), "toy world 4 rank 1 d=0.01") is None
    assert bench.read_traffic(str(traffic)) == 123456789.0  # no workload asked for


def test_one_core_pins_and_restores_the_affinity():
    before = os.sched_getaffinity(0)
    with bench.OneCore() as pin:
        assert os.sched_getaffinity(0) == {pin.core}
        assert pin.core in before
        assert f"core {pin.core}" in pin.describe()
    assert os.sched_getaffinity(0) == before


@pytest.mark.parametrize("n", ["2", "8"])
def test_more_than_one_gpu_is_refused(n):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", n],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "not supported" in r.stderr and "one GPU" in r.stderr
    assert r.stdout == ""


def test_paths_default_to_their_workloads_and_the_topk_hint_to_the_last_theta(monkeypatch):
    """--path topk / ef / union / sweep fall back to the workloads they are
    measured on (world 1 makes them degenerate), and top-k calls get the last
    k-th magnitude as their hint unless --topk-hint says otherwise."""
    cases = [(["--path", "topk"], "bert_large", "last"),
             (["--path", "topk", "--topk-hint", "high"], "bert_large", "high"),
             (["--path", "topk", "--workload", "gpt_1p3b", "--topk-hint", "none"], "gpt_1p3b", "none"),
             (["--path", "sweep"], "resnet18", "last"),
             (["--path", "ef"], "bert_large", "last"),
             ([], "gpt_1p3b", "last")]
    for argv, workload, hint in cases:
        monkeypatch.setattr(sys, "argv", ["bench.py"] + argv)
        args = bench.parse_args()
        assert (args.workload, args.topk_hint) == (workload, hint), argv
    monkeypatch.setattr(sys, "argv", ["bench.py", "--path", "topk", "--topk-hint", "sometimes"])
    with pytest.raises(SystemExit):
        bench.parse_args()
