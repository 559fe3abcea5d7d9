"""The bench's command line on the host: it measures one GPU and refuses more,
before touching any device."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(*args, env=None):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args],
                          capture_output=True, text=True, timeout=120, env=env, cwd=ROOT)


def test_more_than_one_gpu_is_refused():
    r = _run("--gpus", "2")
    assert r.returncode != 0
    assert "measures one GPU" in (r.stdout + r.stderr)
    assert not r.stdout.lstrip().startswith("{")     # no bench line


def test_distributed_launch_is_refused():
    env = dict(os.environ, WORLD_SIZE="2", RANK="0", LOCAL_RANK="0")
    r = _run(env=env)
    assert r.returncode != 0
    assert "measures one GPU" in (r.stdout + r.stderr)
