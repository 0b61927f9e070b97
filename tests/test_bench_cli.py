"""bench.py's command line on the host: more than one GPU is refused with a
message and exit status 2, before any device is touched."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert res.returncode == 2
    assert "one GPU" in res.stderr and res.stdout == ""


def test_source_digest_covers_every_kernel_source():
    sys.path.insert(0, ROOT)
    import bench
    names = sorted(os.listdir(bench.CSRC))
    assert any(n.endswith(".hip") for n in names) and "api.cpp" in names
    assert len(bench.source_digest()) == 16
