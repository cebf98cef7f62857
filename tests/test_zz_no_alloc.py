"""spc_verify_noalloc (static scratch, no device allocation) against
spc_verify_ex on the same inputs: two calls in a row, the second smaller.
Both run the same kernels, so every output must be bitwise equal."""
import numpy as np
import pytest
import torch

from paper_2405_19261_amd import spc
from paper_2405_19261_amd import workloads as W

import parity

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _call(entry, inp):
    q, p = inp["q"], inp["p"]
    B, g1, _ = q.shape
    stats = torch.full((B, g1, 8), float("nan"), device=DEV)
    argmax = torch.full((B, g1, 2), -7, dtype=torch.int32, device=DEV)
    norm = torch.full((B,), float("nan"), device=DEV)
    acc, tok, dm = entry(q, p, inp["draft"], inp["uniforms"], 0, 0.0, 1.0,
                         rule_per_seq=inp["rule"], alpha_per_seq=inp["alpha"],
                         temp_per_seq=inp["temperature"], out_row_stats=stats,
                         out_argmax=argmax, out_sample_norm=norm,
                         rules_present=parity.rules_mask(inp["rule"]))
    torch.cuda.synchronize()
    return [x.cpu().numpy() for x in (acc, tok, dm, stats, argmax, norm)]


def test_noalloc_matches_verify_ex():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    first = W.generate(W.WORKLOADS[5].with_(B=64), 71, DEV)  # mixed rules and temperatures
    second = W.generate(W.WORKLOADS[2].with_(B=3), 72, DEV)  # smaller, float32, OPT
    for inp in (first, second):
        want = _call(spc.spc_verify_ex, inp)
        got = _call(spc.spc_verify_noalloc, inp)
        for a, b in zip(want, got):
            np.testing.assert_array_equal(a, b)
        assert (want[0] >= 0).all()


def test_noalloc_rejects_caller_workspace():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    inp = W.generate(W.WORKLOADS[1], 3, DEV)
    ws = torch.zeros(1 << 20, dtype=torch.uint8, device=DEV)
    with pytest.raises(spc.SpcError):
        spc.spc_verify_noalloc(inp["q"], inp["p"], inp["draft"], inp["uniforms"], W.CHOW, 0.5,
                               1.0, workspace=ws)
