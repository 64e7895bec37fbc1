"""Host-side pieces of bench.py (no GPU): the one-GPU guard, the kernel-code hash that
keys the committed HBM counter summary, and the machine record of the JSON line."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_exits_with_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_kernel_code_hash_ignores_comments_and_blank_lines(tmp_path):
    a = tmp_path / "a.hip"
    b = tmp_path / "b.hip"
    c = tmp_path / "c.hip"
    a.write_text("int f() {\n  return 1;\n}\n")
    b.write_text("// header\nint f() {   \n\n  return 1;  // one\n}\n")
    c.write_text("int f() {\n  return 2;\n}\n")
    assert bench.kernel_code_sha(str(a)) == bench.kernel_code_sha(str(b))
    assert bench.kernel_code_sha(str(a)) != bench.kernel_code_sha(str(c))


def test_committed_counter_summary_matches_kernel_code():
    # the bench line reports HBM traffic only while the counters were taken on the current
    # kernel code; a kernel change must come with fresh counter passes
    t = bench.counter_traffic("opt-6.7b", 0, 1)
    assert t is not None
    algo = sum(n * k * 2 + k * 2 + 2 * n * 2 for n, k in bench.shapes(4096, 16384)) / 4
    assert 0.99 < t / algo < 1.05


def test_host_record_fields():
    torch = pytest.importorskip("torch")
    h = bench.host_info(torch)
    for k in ("cpu", "physical_cores", "logical_cpus", "numa_nodes", "rocm", "hip", "torch"):
        assert k in h
    assert h["logical_cpus"] >= 1 and h["torch"] == torch.__version__
