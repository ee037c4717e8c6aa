"""bench.py's command-line contract on the CPU: one GPU only, the --objects
limits, and the oracle baseline leg (its child process runs the fp64 oracle
on a small workload and reports seconds and frames)."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCH = os.path.join(ROOT, "bench.py")


def _run(*args, timeout=600):
    env = dict(os.environ, HIP_VISIBLE_DEVICES="")
    return subprocess.run([sys.executable, BENCH, *args], stdout=subprocess.PIPE, stderr=subprocess.PIPE,
                          text=True, env=env, timeout=timeout, cwd=ROOT)


def test_more_than_one_gpu_is_refused():
    p = _run("--gpus", "2", "--no-cpu-baseline")
    assert p.returncode == 2
    assert "single GPU" in p.stderr


def test_objects_limits():
    for extra in (["--objects", "65", "--no-cpu-baseline"], ["--objects", "8"],
                  ["--objects", "8", "--stack", "2", "--no-cpu-baseline"]):
        p = _run(*extra)
        assert p.returncode == 2, extra
        assert "--objects" in p.stderr


def test_oracle_baseline_child():
    # the leg bench.py times on the host: select + readout + commit of a few
    # frames after the prefill, fp64 oracle, one thread
    p = _run("--cpu-child", "--workload", "tiny_f32", "--cpu-frames", "3")
    assert p.returncode == 0, p.stderr[-2000:]
    r = json.loads(p.stdout.strip().splitlines()[-1])
    assert r["frames"] == 3 and r["prefill"] == 2 and r["seconds"] > 0


def test_oracle_baseline_child_stack():
    # the stack's baseline leg: select + the L-layer stack + commit per frame
    p = _run("--cpu-child", "--stack", "1", "--workload", "tiny_f32", "--cpu-frames", "1")
    assert p.returncode == 0, p.stderr[-2000:]
    r = json.loads(p.stdout.strip().splitlines()[-1])
    assert r["frames"] == 1 and r["seconds"] > 0
