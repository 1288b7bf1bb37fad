"""bench.py measures one GPU: a request for more GPUs, by flag or by a
multi-rank launcher's environment, ends with a message and exit status 2
before anything touches a device (CPU)."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench(args, env_extra=None):
    env = dict(os.environ)
    env.update(env_extra or {})
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True,
                          text=True, env=env, cwd=ROOT, timeout=120)


def test_more_than_one_gpu_is_refused():
    r = _bench(["--gpus", "2", "--steps", "1", "--warmup", "0"])
    assert r.returncode == 2, r.stderr
    assert "one GPU" in r.stderr and "--gpus 2" in r.stderr
    assert r.stdout == ""   # no JSON line


def test_multi_rank_launch_is_refused():
    r = _bench(["--steps", "1"], {"WORLD_SIZE": "4", "RANK": "0", "LOCAL_RANK": "0"})
    assert r.returncode == 2, r.stderr
    assert "one GPU" in r.stderr
