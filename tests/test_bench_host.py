"""Host-side checks of bench.py that need no GPU."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    # the library has no multi-GPU path: --gpus N > 1 exits (status 2) before any GPU work
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 2
    assert "measures one GPU" in r.stderr
    assert r.stdout == ""


def test_a_world_size_above_one_is_refused():
    env = dict(os.environ, WORLD_SIZE="2")
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py")], capture_output=True,
                       text=True, timeout=300, env=env)
    assert r.returncode == 2
    assert "measures one GPU" in r.stderr


def test_source_hash_is_per_family_and_deterministic():
    sys.path.insert(0, ROOT)
    import bench
    hashes = {fam: bench.kernel_source_hash(fam) for fam in ("tri", "lnl", "trn")}
    assert len(set(hashes.values())) == 3
    assert all(len(h) == 16 for h in hashes.values())
    assert bench.kernel_source_hash("tri") == hashes["tri"]  # deterministic
