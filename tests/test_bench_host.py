"""Host-side parts of bench.py (no GPU): the oracle baseline's fields on the tiny
workload, its thread cap, and the refusal of more than one GPU."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2607_12121_amd import workloads as wl  # noqa: E402


@pytest.mark.parametrize("threads", [None, 1])
def test_cpu_baseline_fields_on_tiny(threads):
    w = wl.WORKLOADS["tiny"]
    params = wl.make_params(w, device="cpu")
    r = bench.cpu_baseline(w, params, M_expected=128, budget_s=1.0, threads=threads)
    assert r["kind"] == "oracle" and r["unit"] == "active tokens/s"
    assert r["value"] > 0 and r["seconds_per_step"] > 0
    assert r["cores"] >= 1 and (threads is None or r["cores"] <= threads)
    assert r["host"]["nproc"] == os.cpu_count()
    assert isinstance(r["host"]["cpu"], str)
    assert "tiny step (M=128 active rows)" in r["sample"]


def test_more_than_one_gpu_is_refused():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300, cwd=ROOT)
    assert p.returncode != 0
    assert "single GPU" in p.stdout
