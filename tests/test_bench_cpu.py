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


def test_kernel_labels_follow_the_measured_rules():
    # bench.py names the kernels a step runs from the library's dispatch rules; on a 256-CU
    # device the split counts of the OPT linears are the ones the library's sweep picked
    # (unsplit where one workgroup per 16-row tile loads the CUs evenly), and the LayerNorm
    # partials are used up to a hidden size of 6144
    splits = {(12288, 4096): 1, (4096, 4096): 1, (16384, 4096): 1, (4096, 16384): 1,      # OPT-6.7B
              (15360, 5120): 1, (5120, 5120): 4, (20480, 5120): 1, (5120, 20480): 4,      # OPT-13B
              (21504, 7168): 1, (7168, 7168): 1, (28672, 7168): 1, (7168, 28672): 1,      # OPT-30B
              (27648, 9216): 1, (9216, 9216): 2, (36864, 9216): 1, (9216, 36864): 2,      # OPT-66B
              (16400, 36864): 2, (4112, 36864): 8, (256, 1024): 1, (37, 72): 1}
    for (n, k), g in splits.items():
        assert bench.mfma_splits(n, k, 256) == g, (n, k)
    env = os.environ.pop("HETEGEN_LN_PARTIALS", None)
    try:
        assert bench.ln_partials_on(4096) and bench.ln_partials_on(5120)
        assert not bench.ln_partials_on(7168) and not bench.ln_partials_on(9216)
    finally:
        if env is not None:
            os.environ["HETEGEN_LN_PARTIALS"] = env
    label = bench.gemv_label(8, 4096, 16384, 0, True, True, 256)
    assert "k-major" in label and "K split" not in label
    # unsplit linears without the LayerNorm take 8 tiles per request at B >= 2, whatever K
    assert "gemv_mfma_kernel<F16,8,8> k-major: layer 0's qkv, out, fc2" in label
    label = bench.gemv_label(8, 9216, 36864, 1, True, False, 256)
    assert "K split 2" in label and "k-major" not in label and "LayerNorm from partials" not in label
