"""Host-side parts of bench.py that run without a GPU: the one-GPU guard and
the oracle's CPU baseline (a pool of single-threaded worker processes)."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], cwd=ROOT,
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
    assert r.stdout == ""


def test_world_size_above_one_is_refused():
    env = dict(os.environ, WORLD_SIZE="2")
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py")], cwd=ROOT, env=env,
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr


def test_cpu_baseline_record():
    sys.path.insert(0, ROOT)
    import bench
    pool = bench.CpuPool()
    try:
        rec = pool.rate("pr1_tiny", 1.0)
    finally:
        pool.close()
    assert rec["kind"] == "oracle" and rec["unit"] == "events/s"
    assert 1 <= rec["cores"] <= 16
    assert rec["value"] > 0
    # the sample names how many events were done and by how many workers
    assert f"in {rec['cores']} single-threaded worker processes" in rec["sample"]
