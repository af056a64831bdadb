"""bench.py's command line on the CPU: more than one GPU is refused with a
message before any GPU work, and the traffic figure is read only from a
counter summary taken on the current kernel sources."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_traffic_only_for_the_current_sources(tmp_path, monkeypatch):
    sys.path.insert(0, ROOT)
    import bench
    sha = bench.kernel_sha()
    good = tmp_path / "good.md"
    good.write_text(f"kernel_source_sha: {sha}\nhbm_bytes_per_launch: 123456\n")
    stale = tmp_path / "stale.md"
    stale.write_text("kernel_source_sha: 0000000000000000\nhbm_bytes_per_launch: 123456\n")
    monkeypatch.setattr(bench, "PROFILE_PMC", str(good))
    assert bench.read_traffic() == 123456.0
    monkeypatch.setattr(bench, "PROFILE_PMC", str(stale))
    assert bench.read_traffic() is None
    monkeypatch.setattr(bench, "PROFILE_PMC", str(tmp_path / "missing.md"))
    assert bench.read_traffic() is None
