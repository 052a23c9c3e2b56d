"""bench.py's command-line contract, checked without a GPU."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                          timeout=120, cwd=ROOT)


def test_more_than_one_gpu_exits_with_a_message():
    r = _run("--gpus", "2", "--steps", "1", "--warmup", "0")
    assert r.returncode != 0
    assert "one GPU" in r.stderr and r.stdout.strip() == ""


def test_help_lists_the_contract_flags():
    r = _run("--help")
    assert r.returncode == 0
    for flag in ("--gpus", "--steps", "--warmup", "--workload", "--mode"):
        assert flag in r.stdout


def test_block_delivery_modes_need_a_shard():
    for mode in ("ring", "gather"):
        r = _run("--workload", "c3", "--mode", mode, "--steps", "1", "--warmup", "0", "--no-cpu-baseline")
        assert r.returncode == 2
        assert "no shard segments" in r.stderr and r.stdout.strip() == ""
