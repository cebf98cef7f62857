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


class _OracleBackend:
    """The decoding loop's two backend calls answered by the oracle, checking
    the parameters as the library does (a rule id, a finite alpha and a
    temperature >= 0 per sequence)."""

    def __init__(self):
        self.verifies = 0

    def draft_sample(self, logits, temperature, uniforms):
        import torch
        t = temperature.numpy()
        tok, _ = oracle.draft_sample(parity.host_logits(logits), t, uniforms.numpy())
        return torch.from_numpy(tok.astype("int32"))

    def verify(self, q, p, drafts, uniforms, rule, alpha, temperature):
        import numpy as np
        import torch
        r, a, t = rule.numpy(), alpha.numpy(), temperature.numpy()
        assert ((r >= 0) & (r <= W.OPTLOG)).all(), r
        assert np.isfinite(a).all() and (t >= 0).all()
        o = oracle.verify(parity.host_logits(q), parity.host_logits(p), drafts.numpy(),
                          uniforms.numpy(), r, a, t)
        self.verifies += 1
        return torch.from_numpy(o["accept_len"]), torch.from_numpy(o["next_token"])


@pytest.mark.parametrize("cfg", [3, 5])
def test_decode_bench_runs_every_workload(cfg):
    """bench.py --decode: the stress mix passes per-sequence arrays (its
    scalar rule is a placeholder), and the loop completes on the oracle."""
    import argparse
    wl = W.WORKLOADS[cfg].with_(B=6, V=700, gamma=3)
    rule, alpha, temp = bench.decode_params(wl)
    if cfg == 5:
        assert rule.shape == (wl.B,) and {int(x) for x in rule} <= {r for r, _ in W.CFG5_RULES}
        assert {round(float(x), 6) for x in temp} <= set(W.CFG5_TEMPS)
    be = _OracleBackend()
    line = bench.bench_decode(argparse.Namespace(decode=3, graph=False), wl, "cpu", backend=be)
    assert be.verifies == 2 + 3
    assert line["value"] > 0 and 1.0 <= line["tokens_per_round"] <= wl.gamma + 1


def test_traffic_record_scales_each_kernel_by_the_copy(tmp_path):
    """--traffic-from: each counter is scaled by what it reads for the copy
    of known size; the record names the roofline kernel and the step's
    other kernels, matched by their own names (not by substrings of others)."""
    import csv
    rows = [("void at::native::vectorized_elementwise_kernel<4, "
             "at::native::neg_kernel_cuda(at::TensorIteratorBase&)>", 131072.0, 262144.0),
            ("void spc::(anonymous namespace)::k_tiles<1, true, 0, 0>(spc::Params)",
             128000.0, 512.0),
            ("void spc::(anonymous namespace)::k_res<1, true>(spc::Params)", 16000.0, 8.0)]
    paths = {}
    for counter, col in (("FETCH_SIZE", 1), ("WRITE_SIZE", 2)):
        p = tmp_path / f"{counter}.csv"
        with open(p, "w", newline="") as fh:
            w = csv.writer(fh)
            w.writerow(["Kernel_Name", "Counter_Name", "Counter_Value"])
            for r in rows:
                w.writerow([r[0], counter, r[col]])
        paths[counter] = str(p)
    rec = bench.traffic_record(paths["FETCH_SIZE"], paths["WRITE_SIZE"], 256)
    assert rec["kernel"] == "k_tiles"
    assert rec["fetch_scale"] == pytest.approx(2.0) and rec["write_scale"] == pytest.approx(1.0)
    assert rec["fetch_bytes"] == pytest.approx(128000.0 * 1024 * 2)
    assert rec["write_bytes"] == pytest.approx(512.0 * 1024)
    assert set(rec["other_kernels"]) == {"k_res"}
    assert rec["other_kernels"]["k_res"]["fetch_bytes"] == pytest.approx(16000.0 * 1024 * 2)
