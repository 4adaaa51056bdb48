"""bench.py host logic that needs no GPU: the one-GPU contract and the option set."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                          timeout=120, cwd=ROOT)


def test_more_than_one_gpu_is_refused_with_a_message():
    r = _run("--gpus", "2")
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)


def test_options_listed():
    r = _run("--help")
    assert r.returncode == 0
    for opt in ("--steps", "--warmup", "--workload", "--budget", "--context", "--select-path", "--score-kind",
                "--compensation", "--n-var-groups", "--page-tokens", "--host-kv", "--host-summaries"):
        assert opt in r.stdout, opt
