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


def test_traffic_is_reported_only_for_the_profiled_code(tmp_path, monkeypatch):
    """The bench line carries a kernel's measured traffic only while the
    committed counter summary was taken from the same kernel code (same
    digest); after a code change it reports null until the counters are
    taken again."""
    prof = tmp_path / "profiles"
    prof.mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    digest = bench.source_digest()
    (prof / "traffic_x.txt").write_text("kernel_source_sha1: %s\nplan_kernel_bytes_per_launch: 1234.0\n" % digest)
    assert bench.measured_traffic("x", "plan") == 1234.0
    assert bench.measured_traffic("x", "solve") is None
    (prof / "traffic_x.txt").write_text("kernel_source_sha1: 0123456789ab\nplan_kernel_bytes_per_launch: 1234.0\n")
    assert bench.measured_traffic("x", "plan") is None
    assert bench.measured_traffic("missing", "plan") is None


def test_committed_traffic_profiles_parse():
    """Each committed traffic summary names its code digest and a per-launch
    byte count for every kernel of its workload."""
    for name, kernels in (("tiny", ["plan"]), ("mixtral", ["plan"]), ("qwen3", ["plan"]), ("dsv3", ["plan"]),
                          ("stress", ["hist", "solve", "reroute"])):
        path = os.path.join(ROOT, "profiles", "traffic_%s.txt" % name)
        text = open(path).read()
        assert "kernel_source_sha1:" in text, name
        for k in kernels:
            assert "%s_kernel_bytes_per_launch:" % k in text, (name, k)


def test_digest_ignores_comments(tmp_path, monkeypatch):
    src = tmp_path / "k.hip"
    src.write_text("int a = 1;  // one\n\n// note\nint b = 2;\n")
    monkeypatch.setattr(bench, "KERNEL_SRCS", [str(src)])
    d0 = bench.source_digest()
    src.write_text("// header\nint a = 1;\nint b = 2;  // two\n")
    assert bench.source_digest() == d0
    src.write_text("int a = 1;\nint b = 3;\n")
    assert bench.source_digest() != d0
