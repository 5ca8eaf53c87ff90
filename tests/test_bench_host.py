"""Host behaviour of bench.py that needs no GPU (CPU only): the one-GPU refusal, the exit without a
visible GPU, and the oracle's thread count."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench(*args, env=None):
    e = dict(os.environ)
    e.update(env or {})
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                          timeout=300, env=e, cwd=ROOT)


@pytest.mark.parametrize("gpus", ["2", "8"])
def test_more_than_one_gpu_is_refused(gpus):
    r = _bench("--gpus", gpus)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_world_size_above_one_is_refused():
    r = _bench(env={"WORLD_SIZE": "2"})
    assert r.returncode == 2 and r.stdout == ""


def test_no_visible_gpu_exits_without_a_line():
    r = _bench("--workload", "tiny", env={"HIP_VISIBLE_DEVICES": "", "CUDA_VISIBLE_DEVICES": ""})
    if "needs a GPU" not in r.stderr:
        pytest.skip("a GPU is visible here")
    assert r.returncode == 1 and r.stdout == ""


def test_host_threads_follow_affinity_and_share():
    """The oracle's threads: the CPUs the process may run on, capped by a set OMP_NUM_THREADS (bench.py
    is imported in a child process, since importing it sets the BLAS thread variables)."""
    code = "import bench, os; print(bench.HOST_THREADS, len(os.sched_getaffinity(0)), os.environ['OPENBLAS_NUM_THREADS'])"
    for share in ("3", ""):
        e = dict(os.environ, OMP_NUM_THREADS=share)
        out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300, env=e, cwd=ROOT)
        n, cpus, blas = (int(v) for v in out.stdout.split())
        assert n == (min(3, cpus) if share else cpus) and blas == n
