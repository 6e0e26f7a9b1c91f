"""bench.py's command-line contract and its traffic bookkeeping (CPU only)."""
import os
import re
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_traffic_is_reported_only_for_the_profiled_sources():
    text = open(bench.TRAFFIC_FILE).read()
    recorded = re.search(r"gemm_source_sha256_16:\s*([0-9a-f]+)", text).group(1)
    hbm = float(re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", text).group(1))
    assert hbm > 0
    if recorded == bench.gemm_source_hash():
        assert bench.committed_traffic() == hbm
    else:
        assert bench.committed_traffic() is None
    for path in bench.GEMM_SOURCES:
        assert os.path.exists(os.path.join(ROOT, path)), path
