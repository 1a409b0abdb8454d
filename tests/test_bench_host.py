"""Host-side pieces of bench.py, on the CPU: the one-GPU guard, the algorithmic
byte counts the roofline uses, the counter lookup and the CPU-baseline leg on the
small workload."""
import os
import subprocess
import sys

import bench
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "exactly one GPU" in r.stderr and r.stdout == ""


def test_algorithmic_bytes():
    # per parameter: grad 2 (bf16), weight 4 + 4, codes 1 + 1 read and 1 + 1 written;
    # per block: two fp32 scales read and written
    assert bench.step_kernel_bytes([4096], 2048, 2) == 4096 * 14 + 2 * 16
    assert bench.step_kernel_bytes([4097], 2048, 4) == 4097 * 16 + 3 * 16
    assert bench.norm_bytes([10, 20], 2) == 60
    w = synth.full_3b()
    assert bench.step_kernel_bytes(w.numels, w.block_size, 2) == 43225930880
    assert bench.norm_bytes(w.numels, 2) == 6171688960


def test_counter_lookup():
    assert bench.counter_traffic("no-such-workload") is None


def test_cpu_baseline_on_the_small_workload():
    w = synth.tiny()
    cb = bench.cpu_baseline(w, 2, 0.5)
    assert cb["kind"] == "oracle" and cb["unit"] == "params/s" and cb["cores"] == 2
    assert cb["value"] > 0 and cb["single_thread"]["value"] > 0
    assert "of 4 tensors" in cb["sample"]


def test_source_digest_ignores_comments_only(tmp_path):
    a = tmp_path / "a.hip"
    b = tmp_path / "b.hip"
    c = tmp_path / "c.hip"
    a.write_text("int f(int x) {\n  return x + 1;  // one\n}\n")
    b.write_text("/* header */\nint f(int x)   {\n\n  return x + 1;\n}  // end\n")
    c.write_text("int f(int x) {\n  return x + 2;\n}\n")
    assert bench.source_digest(str(a)) == bench.source_digest(str(b))
    assert bench.source_digest(str(a)) != bench.source_digest(str(c))
