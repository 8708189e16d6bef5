"""bench.py's guards, on the CPU: it runs on exactly one GPU, and says so
(exit status 2) when asked for more, by flag or by a launcher's WORLD_SIZE."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def run_bench(args, env_extra=None):
    env = dict(os.environ)
    env.update(env_extra or {})
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py")] + args, cwd=ROOT,
                          env=env, capture_output=True, text=True, timeout=300)


@pytest.mark.parametrize("args,env", [
    (["--gpus", "2"], None),
    (["--gpus", "8", "--steps", "3"], None),
    ([], {"WORLD_SIZE": "2"}),
])
def test_bench_refuses_more_than_one_gpu(args, env):
    r = run_bench(args, env)
    assert r.returncode == 2
    assert "exactly one GPU" in r.stderr
    assert r.stdout == ""  # no JSON line


def test_bench_without_a_gpu_fails_loudly():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present: the bench itself would run")
    r = run_bench(["--steps", "1", "--warmup", "0"])
    assert r.returncode != 0
    assert r.stdout == ""
