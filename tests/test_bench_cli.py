"""bench.py's command line (no GPU): more than one GPU is refused with a
message before anything touches the device."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def run(*args, env=None):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                          timeout=120, env=env)


def test_more_than_one_gpu_is_refused():
    r = run("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_a_distributed_launch_is_refused():
    env = dict(os.environ, WORLD_SIZE="4")
    r = run(env=env)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_unknown_workload_is_rejected():
    r = run("--workload", "no_such_workload")
    assert r.returncode != 0 and "invalid choice" in r.stderr
