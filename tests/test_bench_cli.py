"""bench.py's command-line contract that runs without a GPU: more than one
GPU is refused with a JSON message (the step is measured on one GPU), and
the flags the measurement scripts pass are accepted by the parser."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def run(*args, env=None):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                          timeout=120, env=env, cwd=ROOT)


def test_more_than_one_gpu_is_refused():
    r = run("--gpus", "2")
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert msg["n_gpus"] == 2 and "one GPU" in msg["error"]


def test_world_size_above_one_is_refused():
    env = dict(os.environ, WORLD_SIZE="4")
    r = run(env=env)
    assert r.returncode == 2 and "error" in json.loads(r.stdout.strip().splitlines()[-1])


def test_help_lists_the_variant_switches():
    r = run("--help")
    assert r.returncode == 0
    for flag in ("--no-cpu-baseline", "--no-full-tier", "--no-sampling", "--no-drafter", "--no-prefill-gemm",
                 "--breakdown", "--copy-probe", "--steps", "--warmup", "--config"):
        assert flag in r.stdout, flag
