"""Decomposition invariance and the draw's edge uniforms (needs an MI355X).

The launch layout depends on the batch: how many sequences a launch holds,
how many workgroups the job pass gets, whether the statistics tiles take
their rows' TV passes or a kernel of its own does, one or two tiles per
workgroup.  None of it may change a result: the same sequences verified inside
batches of B = 1, 8, 32 and 256 at the Gemma vocabulary must give bitwise
identical outputs, row statistics and sampled masses.  The draws at
u = 0 and u = 1 - 2^-24 reach the ends of the inverse-CDF search (the first
entry with mass, and the rounding fallback to the last one) and are checked
against the oracle for both the residual and the extra-token draw."""
import numpy as np
import pytest
import torch

from paper_2405_19261_amd import workloads as W

import parity

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.init()
    yield
    torch.cuda.synchronize()


def _flush(msg):
    print(msg, flush=True)


def _sub(inp, idx):
    return {k: v[idx].contiguous() for k, v in inp.items()}


def _bits(a):
    a = np.ascontiguousarray(a)
    return a.view(np.uint32) if a.dtype == np.float32 else a


# the same sequences at several batch sizes: (B, first sequence)
_SPLITS = [(1, 77), (8, 248), (32, 100), (32, 0)]
_MODES = {
    # Diff at T = 1 (the Gemma-vocabulary step), through the scalar entry point
    "diff-plain": (3, dict(), False, False),
    "diff": (3, dict(), True, False),
    # OPT: TV passes from the rows' own tiles (B = 1) or the TV pass kernel
    "opt": (3, dict(rule=W.OPT, alpha=0.1), True, False),
    # OPT without row statistics: rows D_TV cannot change skip their TV pass
    "opt-plain": (3, dict(rule=W.OPT, alpha=0.1), False, False),
    # the stress mix: per-sequence rules and temperatures, identical and
    # independent drafters
    "mix": (5, dict(), True, False),
    # temperature 0 (argmax drafts, deterministic deferral)
    "greedy": (4, dict(), True, True),
}


@pytest.mark.parametrize("mode", list(_MODES))
def test_same_sequences_in_any_batch(mode):
    cfg, kw, stats, greedy = _MODES[mode]
    wl = W.WORKLOADS[cfg].with_(B=256, gamma=7, V=256000, **kw)
    _flush(f"[invariance] {mode}: B=256 gamma=7 V=256000 {wl.dtype}")
    inp = W.generate(wl, 61, DEV)
    full = parity.run_gpu(inp, greedy=greedy, stats=stats)
    for B, b0 in _SPLITS:
        _flush(f"[invariance] {mode}: sequences {b0}..{b0 + B - 1} as a batch of {B}")
        part = parity.run_gpu(_sub(inp, slice(b0, b0 + B)), greedy=greedy, stats=stats)
        for k, v in part.items():
            ref = full[k][b0:b0 + B]
            assert np.array_equal(_bits(v), _bits(ref)), \
                f"{mode}: {k} of sequences {b0}..{b0 + B - 1} differs at B={B}"
    del inp
    torch.cuda.empty_cache()


_U_LAST = [0.0, 1.0 - 2.0 ** -24]
_EDGE_SHAPES = {
    # the single-launch small path, the T5 vocabulary in float32, the Gemma
    # vocabulary in bfloat16 (OPT and Diff)
    "tiny": (1, dict(B=8)),
    "t5": (2, dict(B=8)),
    "gemma-diff": (3, dict(B=8)),
    "gemma-opt": (3, dict(B=8, rule=W.OPT, alpha=0.1)),
}


@pytest.mark.parametrize("u_last", _U_LAST, ids=["u0", "u1m"])
@pytest.mark.parametrize("shape", list(_EDGE_SHAPES))
def test_draw_at_edge_uniforms(shape, u_last):
    """Sequences 0-3 reject (every acceptance uniform 1 - 2^-24, drafters
    noisy): a residual draw.  Sequences 4-7 have p = q: every draft is kept
    and the extra token is drawn.  Every draw takes u = u_last."""
    cfg, kw = _EDGE_SHAPES[shape]
    wl = W.WORKLOADS[cfg].with_(**kw)
    rep = None
    kinds = {"residual": 0, "extra": 0}
    for step in range(3):
        inp = W.generate(wl, 70 + step, DEV)
        inp["p"][4:] = inp["q"][4:]
        inp["uniforms"][:4, :wl.gamma] = 1.0 - 2.0 ** -24
        inp["uniforms"][:, wl.gamma] = u_last
        g = parity.run_gpu(inp)
        h = parity.host_inputs(inp)
        o = parity.run_oracle(h)
        rep = parity.compare(g, o, h, wl.dtype, rep=rep)
        kinds["residual"] += int((o["accept_len"][:4] < wl.gamma).sum())
        kinds["extra"] += int((o["accept_len"][4:] == wl.gamma).sum())
        assert ((g["next_token"] >= 0) & (g["next_token"] < wl.V)).all()
    _flush(f"[u-edge] {shape} u={u_last!r}: {kinds} {dict(rep)}")
    assert kinds["residual"] >= 6 and kinds["extra"] == 12
    # the ends of the search are exact draws, not near-ties
    assert rep["exact"] >= rep["sequences"] - 2


def test_tv_slice_jobs_match_the_tv_pass_kernel():
    """Where the rules come per sequence, a large batch's TV rows go to the job
    pass as single slices; where one rule holds for the batch, to the TV pass
    kernel.  With every sequence OPT and the row statistics requested (so no
    row is settled without its TV pass) B = 256, gamma = 8 at the Gemma
    vocabulary publishes 2304 rows x 32 tiles x 4 slices = 294 912 slice
    jobs: more than 64 per wavefront of the job pass's 4096, so each
    wavefront requests its job entries in more than one round.  Both routes
    must give bitwise identical outputs, row statistics (D_TV in column 6)
    and sampled masses; eight sequences are also checked against the
    oracle."""
    wl = W.WORKLOADS[3].with_(B=256, gamma=8, V=256000, rule=W.OPT, alpha=0.1)
    _flush(f"[tv-jobs] B=256 gamma=8 V=256000 {wl.dtype} OPT: TV pass kernel")
    inp = W.generate(wl, 64, DEV)
    batch_wide = parity.run_gpu(inp, stats=True)
    _flush("[tv-jobs] the same batch with per-sequence rules: TV slices as jobs")
    per_seq = parity.run_gpu(inp, stats=True, per_seq=True)
    for k, v in per_seq.items():
        assert np.array_equal(_bits(v), _bits(batch_wide[k])), f"{k} differs between the routes"
    sub = _sub(inp, slice(0, 8))
    h = parity.host_inputs(sub)
    del inp
    torch.cuda.empty_cache()
    o = parity.run_oracle(h)
    g = {k: v[:8] for k, v in per_seq.items()}
    rep = parity.compare(g, o, h, wl.dtype)
    _flush(f"[tv-jobs] first 8 sequences against the oracle: {dict(rep)}")
    assert rep["exact"] >= rep["sequences"] - 1
