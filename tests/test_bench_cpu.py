"""Parts of bench.py's contract that need no GPU: more than one GPU is refused
with a message, and the measured-counter tables are keyed by workload, layer
count and a hash of the score-phase sources."""
import os
import re
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)


def test_source_hash_is_stable_and_hex():
    h = bench.kernel_source_hash()
    assert re.fullmatch(r"[0-9a-f]{16}", h)
    assert bench.kernel_source_hash() == h


def test_measured_tables_are_well_formed():
    for table in (bench.MEASURED_TRAFFIC, bench.MEASURED_MFMA):
        for (name, layers, h), val in table.items():
            assert isinstance(name, str) and layers >= 1
            assert re.fullmatch(r"[0-9a-f]{16}", h)
            assert val
    for v in bench.MEASURED_TRAFFIC.values():
        assert v > 0
    for v in bench.MEASURED_MFMA.values():
        assert v["executed_flops_per_launch"] > 0
        assert all(0 < f < 1 for f in v["busy_frac"].values())
