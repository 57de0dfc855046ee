"""bench.py's contract checks that need no GPU: one GPU only, and the measured-traffic
lookup that ties a bench line to a committed counter summary of the same kernel sources."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       timeout=300)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_measured_traffic_reads_the_summary_only_for_matching_sources(tmp_path, monkeypatch):
    sys.argv = ["bench.py"]
    import bench
    prof = tmp_path / "profiles"
    prof.mkdir()
    h = bench.kernel_source_hash()
    (prof / "hbm_traffic_demo.md").write_text(f"# demo\n\n- kernel_source_hash: `{h}`\n"
                                              "- traffic_bytes_per_launch: `12345`\n")
    (prof / "hbm_traffic_stale.md").write_text("- kernel_source_hash: `0000000000000000`\n"
                                               "- traffic_bytes_per_launch: `999`\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_source_hash", lambda sources=None: h)
    assert bench.measured_traffic("demo") == 12345
    assert bench.measured_traffic("stale") is None
    assert bench.measured_traffic("absent") is None


def test_kernel_source_hash_covers_the_kernel_sources():
    sys.argv = ["bench.py"]
    import bench
    assert bench.kernel_source_hash() == bench.kernel_source_hash(bench.KERNEL_SOURCES)
    assert bench.kernel_source_hash(bench.MULTI_SOURCES) != bench.kernel_source_hash(bench.KERNEL_SOURCES)
    assert all(os.path.exists(p) for p in bench.KERNEL_SOURCES + bench.MULTI_SOURCES)
