"""The benchmark's command-line contract and its link to the committed
counter profiles (host only, no GPU)."""
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr


def test_traffic_profiles_match_the_kernel_code():
    """Every committed traffic summary was taken from the kernels as they
    are (same code digest), so the benchmark reports its traffic."""
    for name in ("tiny", "mixtral", "qwen3", "dsv3"):
        assert bench.measured_traffic(name, "plan") is not None, name
    for kernel in ("hist", "solve", "reroute"):
        assert bench.measured_traffic("stress", kernel) is not None, kernel


def test_digest_ignores_comments(tmp_path, monkeypatch):
    src = tmp_path / "k.hip"
    src.write_text("int a = 1;  // one\n\n// note\nint b = 2;\n")
    monkeypatch.setattr(bench, "KERNEL_SRCS", [str(src)])
    d0 = bench.source_digest()
    src.write_text("// header\nint a = 1;\nint b = 2;  // two\n")
    assert bench.source_digest() == d0
    src.write_text("int a = 1;\nint b = 3;\n")
    assert bench.source_digest() != d0
