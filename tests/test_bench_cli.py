"""The benchmark's command-line contract on a host without a GPU: more than
one GPU is refused with a message, and the help lists the modes."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_help_lists_the_modes():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--help"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 0
    for flag in ("--steps", "--warmup", "--workload", "--no-merge", "--reuse-store",
                 "--signatures", "--sig-nodes", "--priorities", "--prio-only", "--batch-curve",
                 "--seed", "--oracle-threads", "--raw-ids", "--cpu-sample", "--corpus-rows",
                 "--batch-sizes", "--graph", "--corpus-layout"):
        assert flag in r.stdout, flag
    # the no-flag run is the largest single-GPU workload
    assert "mfma4m (default)" in r.stdout


def test_host_side_helpers():
    # dedup path rule and oracle thread choice, without a GPU
    sys.path.insert(0, ROOT)
    import numpy as np
    import bench
    assert bench.dedup_path(np.arange(100, dtype=np.int64)).startswith("lds-hash")
    assert bench.dedup_path(np.arange(3000, dtype=np.int64)).startswith("bitonic")
    assert bench.dedup_path(np.arange(10000, dtype=np.int64) % 5000).startswith("direct")
    big = np.array([0, 1 << 40] * 5000, dtype=np.int64)
    assert bench.dedup_path(big) == "radix (6 passes of 8 bits)"
    assert bench.oracle_threads(7) == 7
    assert bench.oracle_threads(0) >= 1
    info = bench.host_cpu()
    assert info["logical_cpus"] == os.cpu_count()
