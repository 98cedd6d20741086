"""bench.py's command-line contract on a host without a GPU: a request for
more than one GPU is refused with a message before anything is imported or
measured, and a single-GPU run on a host without one stops with an error
instead of measuring anything else."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def run_bench(args, env_extra=None):
    env = dict(os.environ)
    env.pop("WORLD_SIZE", None)
    env.update(env_extra or {})
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py")] + args,
                          stdout=subprocess.PIPE, stderr=subprocess.PIPE,
                          universal_newlines=True, env=env, timeout=300)


@pytest.mark.parametrize("gpus", [2, 8])
def test_more_than_one_gpu_is_refused(gpus):
    r = run_bench(["--gpus", str(gpus), "--steps", "1", "--warmup", "0"])
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""  # no JSON line


def test_a_distributed_launch_is_refused():
    r = run_bench(["--steps", "1", "--warmup", "0"], {"WORLD_SIZE": "4"})
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_no_gpu_no_measurement():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present: this checks the host-only exit")
    r = run_bench(["--steps", "1", "--warmup", "0"])
    assert r.returncode == 1
    assert "needs a GPU" in r.stderr
    assert r.stdout == ""
