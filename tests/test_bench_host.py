"""Host-side logic of bench.py: the oracle baseline leg and the one-GPU guard
(no GPU needed)."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import oracle  # noqa: E402
import parity  # noqa: E402
from paper_2405_19261_amd import workloads as W  # noqa: E402


def test_cpu_baseline_fields_and_thread_restore():
    wl = W.WORKLOADS[3].with_(B=2, V=3000)
    inp = W.generate(wl, 0, "cpu")
    # the oracle's own outputs stand in for the GPU's: the parity check must
    # then report every sequence exact
    o = parity.run_oracle(parity.host_inputs(inp))
    threads = oracle.num_threads()
    cb, rep = bench.cpu_baseline(wl, inp, o, min_seconds=0.05)
    assert oracle.num_threads() == threads
    assert cb["kind"] == "oracle" and cb["unit"] == "positions/s"
    assert cb["cores"] == threads
    assert cb["value"] > 0 and cb["one_thread_value"] > 0
    assert "one_thread" in cb["sample"]
    assert rep["exact"] == wl.B


def test_thread_count_does_not_change_results():
    wl = W.WORKLOADS[5].with_(B=6, V=2000)
    h = parity.host_inputs(W.generate(wl, 1, "cpu"))
    threads = oracle.num_threads()
    try:
        oracle.set_num_threads(1)
        a = parity.run_oracle(h)
    finally:
        oracle.set_num_threads(threads)
    b = parity.run_oracle(h)
    for k in a:
        assert (a[k] == b[k]).all() or k.endswith("margin"), k


@pytest.mark.parametrize("n", [2, 8])
def test_more_than_one_gpu_is_refused(n):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", str(n)],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in r.stderr or "1 GPU" in r.stderr or "single" in r.stderr, r.stderr
