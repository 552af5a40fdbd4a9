"""bench.py's command line on the CPU: more than one GPU is refused with a
message (the path does not shard), and the source hash that gates the
committed traffic figures covers exactly the decode path's sources."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def test_more_than_one_gpu_is_refused():
    out = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                         text=True, timeout=120)
    assert out.returncode == 2
    assert "one GPU" in out.stderr


def test_traffic_hash_ignores_host_only_sources(tmp_path, monkeypatch):
    import bench

    h0 = bench.kernel_source_hash()
    csrc = os.path.join(ROOT, "paper_2606_24506_amd", "csrc")
    names = sorted(os.listdir(csrc))
    assert "planner.cpp" in names and "kernels.hip" in names
    # the hash reads the device code, the launcher and the allocator only
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    dst = tmp_path / "paper_2606_24506_amd" / "csrc"
    dst.mkdir(parents=True)
    for n in names:
        (dst / n).write_bytes(open(os.path.join(csrc, n), "rb").read())
    assert bench.kernel_source_hash() == h0
    (dst / "planner.cpp").write_text("// changed\n")
    assert bench.kernel_source_hash() == h0
    (dst / "kernels.hip").write_text("// changed\n")
    assert bench.kernel_source_hash() != h0
