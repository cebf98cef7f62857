"""GPU path vs the fp64 oracle, through the C interface (needs an MI355X).

Full-size workloads run in the launch configuration the benchmark times;
edge cases cover ragged and unaligned vocabularies, masked logits,
out-of-range drafts, identical drafter/verifier rows, block-size extremes,
per-sequence parameters, caller workspaces, streams and run-to-run
determinism."""
import os

import numpy as np
import pytest
import torch

from paper_2405_19261_amd import spc
from paper_2405_19261_amd import workloads as W

import parity

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _steps(cfg, default):
    return int(os.environ.get(f"SPC_PARITY_STEPS_{cfg}", default))


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.init()
    yield
    torch.cuda.synchronize()


def _flush(msg):
    print(msg, flush=True)


# ------------------------------------------------------------ full workloads

@pytest.mark.parametrize("cfg,steps", [(1, 1000), (3, 100), (4, 50)])
def test_workload_parity(cfg, steps):
    wl = W.WORKLOADS[cfg]
    _flush(f"[parity] cfg{cfg} {wl.name} steps={_steps(cfg, steps)}")
    rep = parity.parity_workload(wl, _steps(cfg, steps))
    _flush(f"[parity] cfg{cfg} {dict(rep)}")
    parity.check_accounting(rep)


@pytest.mark.parametrize("part", range(4))
def test_workload2_parity(part):
    """T5-vocabulary workload (OPT): the seeded steps split into four parts."""
    wl = W.WORKLOADS[2]
    n = _steps(2, 10000) // 4
    _flush(f"[parity] cfg2 part {part} steps={n}")
    rep = parity.parity_workload(wl, n, step0=part * n, stats=(part == 0),
                                 report_name=f"cfg2.{part}")
    _flush(f"[parity] cfg2.{part} {dict(rep)}")
    parity.check_accounting(rep)


@pytest.mark.parametrize("part", range(2))
def test_workload5_parity(part):
    """Stress mix: per-sequence temperature and rule, identical and independent drafters."""
    wl = W.WORKLOADS[5]
    n = _steps(5, 20) // 2
    _flush(f"[parity] cfg5 part {part} steps={n}")
    rep = parity.parity_workload(wl, n, step0=part * n, report_name=f"cfg5.{part}")
    _flush(f"[parity] cfg5.{part} {dict(rep)}")
    parity.check_accounting(rep)


@pytest.mark.parametrize("rule,alpha", [(W.OPT, 0.1), (W.OPT, -0.05), (W.OPTLOG, 0.5)])
@pytest.mark.parametrize("cfg,B", [(2, 8), (3, 16)])
def test_tv_rules_without_row_statistics(rule, alpha, cfg, B):
    """Without row statistics to report, an OPT / OPTLog row whose decision
    D_TV in [0, 1] cannot change is decided at its merge and takes no TV pass
    (at the T5 shape its own waiting tiles skip theirs; at the Gemma shape
    the TV pass kernel skips it).  Decisions, accept lengths and tokens must
    still match the oracle, for alpha of either sign."""
    wl = W.WORKLOADS[cfg].with_(B=B, rule=rule, alpha=alpha, temperature=1.0)
    name = f"tvfree.cfg{cfg}.{W.RULE_NAMES[rule]}.{alpha:g}"
    _flush(f"[parity] {name}")
    rep = parity.parity_workload(wl, 3, stats=False, step0=840, report_name=name)
    parity.check_accounting(rep)
    assert rep["sequences"] == 3 * B


@pytest.mark.parametrize("cfg", [2, 3])
def test_tv_wait_timeout_takes_the_job_pass(cfg, monkeypatch):
    """A statistics workgroup's wait for a TV row's merge is bounded; with the
    bound at 0 ticks every wait that does not find the row merged gives up at
    once and the job pass takes the tile.  The T5 shape (a resident grid)
    takes its TV passes from the rows' own tiles and so waits; the Gemma
    shape takes them in the TV pass kernel and never waits.  Both must match
    the oracle."""
    monkeypatch.setenv("SPC_TV_WAIT_TICKS", "0")
    wl = W.WORKLOADS[cfg].with_(B=8, rule=W.OPT, alpha=0.1, temperature=1.0)
    _flush(f"[parity] tv wait 0: cfg{cfg} OPT B=8")
    rep = parity.parity_workload(wl, 3, step0=810, report_name=f"tvwait0.cfg{cfg}")
    parity.check_accounting(rep)
    assert rep["sequences"] == 3 * 8


def test_workload3_bench_entry_point():
    """The batch-wide entry point the benchmark times (no optional outputs)."""
    wl = W.WORKLOADS[3]
    rep = parity.parity_workload(wl, 8, stats=False, step0=500, report_name="cfg3.plain")
    assert rep["sequences"] == 8 * 32


def test_workload4_greedy_entry_point_deterministic():
    wl = W.WORKLOADS[4]
    inp = W.generate(wl, 7, DEV)
    a = parity.run_gpu(inp, greedy=True, stats=False)
    b = parity.run_gpu(inp, greedy=True, stats=False)
    for k in a:
        np.testing.assert_array_equal(a[k], b[k])
    h = parity.host_inputs(inp)
    o = parity.run_oracle(h, greedy=True)
    parity.compare(a, o, h, wl.dtype, greedy=True)


# ----------------------------------------------------------------- edge cases

@pytest.mark.parametrize("dtype,V", [("bf16", 2), ("bf16", 3), ("bf16", 1000), ("bf16", 1001),
                                     ("bf16", 16383), ("bf16", 16385), ("bf16", 40000),
                                     ("f32", 2), ("f32", 999), ("f32", 8193), ("f32", 32128)])
def test_ragged_vocabularies(dtype, V):
    for cfg in (3, 2):
        wl = W.WORKLOADS[cfg].with_(B=6, V=V, dtype=dtype, rule=W.OPT, alpha=0.1)
        _flush(f"[edge] ragged cfg{cfg} {dtype} V={V}")
        parity.parity_workload(wl, 3, report_name=f"ragged.{dtype}.{V}")


@pytest.mark.parametrize("gamma,B", [(1, 5), (63, 2), (7, 1)])
def test_block_size_extremes(gamma, B):
    wl = W.WORKLOADS[3].with_(B=B, gamma=gamma, V=5000)
    parity.parity_workload(wl, 3, report_name=f"gamma{gamma}")
    parity.parity_workload(wl.with_(temperature=0.0, cfg=4), 2, report_name=f"gamma{gamma}.g")


@pytest.mark.parametrize("dtype,rule,alpha", [("bf16", W.DIFF, 0.05), ("f32", W.OPT, 0.1)])
def test_maximum_rows(dtype, rule, alpha):
    """B*(gamma+1) = 100000 rows: more than one launch holds (16384 rows), so
    the call runs consecutive launches of whole sequences."""
    wl = W.WORKLOADS[3].with_(B=20000, gamma=4, V=37, dtype=dtype, rule=rule, alpha=alpha)
    _flush(f"[edge] maximum rows {dtype} rule={rule}")
    parity.parity_workload(wl, 1, report_name=f"maxrows.{dtype}")
    parity.parity_workload(wl.with_(temperature=0.0, cfg=4), 1, report_name=f"maxrows.{dtype}.g")


def test_identical_models_accept_all():
    wl = W.WORKLOADS[3].with_(B=16, V=20000)
    for rule, alpha in ((W.DIFF, 0.0), (W.OPT, 0.1), (W.ALWAYS, 0.0), (W.CHOW, 0.3)):
        inp = W.generate(wl, 3, DEV)
        inp["p"] = inp["q"].clone()
        inp["rule"][:] = rule
        inp["alpha"][:] = alpha
        g = parity.run_gpu(inp)
        assert (g["accept_len"] == wl.gamma).all()
        if rule == W.OPT:
            assert (g["row_stats"][..., 6] == 0).all()
        if rule in (W.DIFF, W.OPT):
            assert (g["defer"] == 0).all()
        h = parity.host_inputs(inp)
        parity.compare(g, parity.run_oracle(h), h, wl.dtype)


def test_out_of_range_drafts():
    wl = W.WORKLOADS[3].with_(B=8, V=3000)
    inp = W.generate(wl, 1, DEV)
    inp["draft"][:, 2] = torch.tensor([-1, 3000, 1 << 30, -(1 << 30), 2999, 0, -5, 3001],
                                      dtype=torch.int32, device=DEV)
    inp["uniforms"][:, :2] = 0.0
    for rule in (W.DIFF, W.NEVER, W.ALWAYS, W.TOKEN_V1, W.TOKEN_V2, W.TOKEN_V3):
        inp["rule"][:] = rule
        inp["alpha"][:] = 0.3 if rule == W.TOKEN_V3 else 0.05
        g = parity.run_gpu(inp)
        h = parity.host_inputs(inp)
        o = parity.run_oracle(h)
        parity.compare(g, o, h, wl.dtype)


@pytest.mark.parametrize("rule,alpha", [(W.OPT, 0.1), (W.TOKEN_V2, 0.05), (W.TOKEN_V3, 0.3)])
def test_masked_logits(rule, alpha):
    """-inf entries (masked tokens) in both tensors."""
    for cfg, dtype in ((3, "bf16"), (2, "f32")):
        wl = W.WORKLOADS[cfg].with_(B=8, V=12345, dtype=dtype, rule=rule, alpha=alpha)
        inp = W.generate(wl, 2, DEV)
        g0 = torch.Generator(device=DEV).manual_seed(99)
        for k in ("q", "p"):
            m = torch.rand(inp[k].shape, generator=g0, device=DEV) < 0.3
            m[..., 0] = False  # at least one finite entry per row
            inp[k][m] = float("-inf")
        inp["draft"] = W.draw_drafts(inp["q"], inp["temperature"], g0)
        g = parity.run_gpu(inp)
        h = parity.host_inputs(inp)
        parity.compare(g, parity.run_oracle(h), h, wl.dtype)


def test_greedy_opt_equals_diff_on_gpu():
    """Lemma 6 on the GPU path: OPT and Diff emit the same tokens at T = 0."""
    wl = W.WORKLOADS[4].with_(B=64, V=50000)
    inp = W.generate(wl, 5, DEV)
    outs = []
    for rule in (W.OPT, W.DIFF):
        for alpha in (0.0, 0.1, 0.3):
            inp["rule"][:] = rule
            inp["alpha"][:] = alpha
            outs.append(parity.run_gpu(inp, greedy=True, stats=False))
    for a, b in zip(outs[:3], outs[3:]):
        np.testing.assert_array_equal(a["accept_len"], b["accept_len"])
        np.testing.assert_array_equal(a["next_token"], b["next_token"])


def test_mixed_greedy_and_sampled_sequences():
    """Per-sequence temperature 0 selects the greedy step for that sequence only."""
    wl = W.WORKLOADS[5].with_(B=24, V=30000)
    inp = W.generate(wl, 4, DEV)
    inp["temperature"][::3] = 0.0
    g = parity.run_gpu(inp)
    h = parity.host_inputs(inp)
    greedy = h["temperature"] == 0
    for sel, gr in ((greedy, True), (~greedy, False)):
        hs = {k: v[sel] for k, v in h.items()}
        o = parity.run_oracle(hs, greedy=gr)
        gs = {k: v[sel] for k, v in g.items()}
        parity.compare(gs, o, hs, wl.dtype, greedy=gr)


@pytest.mark.parametrize("V", [4000, 40000])
def test_invalid_per_sequence_values(V):
    """Invalid per-sequence values (an unknown rule, a NaN alpha, a negative
    temperature) report -1 for that sequence only, on the single-launch path
    (V = 4000) and on the statistics-tile path (V = 40000)."""
    wl = W.WORKLOADS[3].with_(B=6, V=V)
    inp = W.generate(wl, 0, DEV)
    inp["rule"][1] = 13
    inp["alpha"][2] = float("nan")
    inp["temperature"][3] = -1.0
    g = parity.run_gpu(inp)
    assert list(g["accept_len"][1:4]) == [-1, -1, -1]
    assert list(g["next_token"][1:4]) == [-1, -1, -1]
    keep = np.array([0, 4, 5])
    h = {k: v[keep] for k, v in parity.host_inputs(inp).items()}
    parity.compare({k: v[keep] for k, v in g.items()}, parity.run_oracle(h), h, wl.dtype)


def test_per_sequence_arrays_match_scalar_api():
    wl = W.WORKLOADS[3].with_(B=16, V=70000, rule=W.OPT, alpha=0.1, temperature=0.7)
    inp = W.generate(wl, 9, DEV)
    a = parity.run_gpu(inp, stats=True)
    b = parity.run_gpu(inp, stats=False)
    for k in ("accept_len", "next_token", "defer"):
        np.testing.assert_array_equal(a[k], b[k])


def test_caller_workspace_and_stream():
    wl = W.WORKLOADS[3].with_(B=8, V=50000)
    inp = W.generate(wl, 11, DEV)
    n = spc.spc_workspace_bytes(8, wl.gamma, wl.V, spc.SPC_BF16)
    z = spc.spc_workspace_zero_bytes(8, wl.gamma, wl.V, spc.SPC_BF16)
    ws = torch.zeros(n, dtype=torch.uint8, device=DEV)
    s = torch.cuda.Stream()
    ref = parity.run_gpu(inp, stats=False)
    for _ in range(3):  # the counters must come back to zero after each call
        with torch.cuda.stream(s):
            acc, tok, dm = spc.spc_verify_ex(inp["q"], inp["p"], inp["draft"], inp["uniforms"],
                                             W.DIFF, 0.05, 1.0, workspace=ws, stream=s)
        s.synchronize()
        assert (ws[:z] == 0).all()
        np.testing.assert_array_equal(acc.cpu().numpy(), ref["accept_len"])
        np.testing.assert_array_equal(tok.cpu().numpy(), ref["next_token"])
        np.testing.assert_array_equal(dm.cpu().numpy(), ref["defer"])


def test_run_to_run_determinism_full_size():
    """Config-3 and config-5 shapes: two runs are bitwise identical, statistics included."""
    for cfg in (3, 5):
        wl = W.WORKLOADS[cfg]
        inp = W.generate(wl, 123, DEV)
        a = parity.run_gpu(inp)
        b = parity.run_gpu(inp)
        for k in a:
            np.testing.assert_array_equal(a[k], b[k])
        del inp


# ------------------------------------------------- token-specific rules (4.4)

TOKEN_ALPHAS = {W.TOKEN_V1: (0.0, 0.05, 0.3), W.TOKEN_V2: (0.0, 0.05, 0.3),
                W.TOKEN_V3: (0.1, 0.5, 0.9)}


@pytest.mark.parametrize("rule", [W.TOKEN_V1, W.TOKEN_V2, W.TOKEN_V3])
@pytest.mark.parametrize("cfg,steps", [(2, 40), (3, 6)])
def test_token_rule_parity(rule, cfg, steps):
    """Alg. 6 target on the T5-vocabulary float32 shape and the Gemma-vocabulary
    bfloat16 shape, several alpha per rule."""
    for alpha in TOKEN_ALPHAS[rule]:
        wl = W.WORKLOADS[cfg].with_(rule=rule, alpha=alpha, temperature=1.0)
        name = f"cfg{cfg}.{W.RULE_NAMES[rule]}.{alpha}"
        _flush(f"[token] {name} steps={steps}")
        rep = parity.parity_workload(wl, steps, step0=900, report_name=name)
        _flush(f"[token] {name} {dict(rep)}")


@pytest.mark.parametrize("rule", [W.TOKEN_V1, W.TOKEN_V2, W.TOKEN_V3])
def test_token_rule_plain_entry_point(rule):
    """The batch-wide entry point without statistics, at the benchmark's shape."""
    wl = W.WORKLOADS[3].with_(rule=rule, alpha=0.3 if rule == W.TOKEN_V3 else 0.05)
    rep = parity.parity_workload(wl, 3, stats=False, step0=700,
                                 report_name=f"cfg3.plain.{W.RULE_NAMES[rule]}")
    assert rep["sequences"] == 3 * 32


@pytest.mark.parametrize("rule", [W.TOKEN_V1, W.TOKEN_V2, W.TOKEN_V3])
def test_token_rule_greedy_parity(rule):
    """Temperature 0: r read at the drafter's argmax, one-hot target."""
    for alpha in (0.0, 0.05, 0.3):
        wl = W.WORKLOADS[4].with_(B=64, V=50000, rule=rule, alpha=alpha)
        _flush(f"[token] greedy {W.RULE_NAMES[rule]} alpha={alpha}")
        parity.parity_workload(wl, 4, step0=300, report_name=f"greedy.{W.RULE_NAMES[rule]}")


def test_token_greedy_v1_equals_diff_on_gpu():
    """At T = 0 the drafter's argmax carries max q, so TokenV1 is the Diff rule."""
    wl = W.WORKLOADS[4].with_(B=64, V=50000)
    inp = W.generate(wl, 6, DEV)
    for alpha in (0.0, 0.05, 0.3):
        outs = []
        for rule in (W.TOKEN_V1, W.DIFF):
            inp["rule"][:] = rule
            inp["alpha"][:] = alpha
            outs.append(parity.run_gpu(inp, greedy=True, stats=False))
        for k in ("accept_len", "next_token", "defer"):
            np.testing.assert_array_equal(outs[0][k], outs[1][k])


@pytest.mark.parametrize("rule,alpha", [(W.TOKEN_V2, -0.5), (W.TOKEN_V3, -0.5),
                                        (W.TOKEN_V1, 1.0), (W.TOKEN_V2, 1.5),
                                        (W.TOKEN_V3, 1.0), (W.TOKEN_V3, 2.0)])
def test_token_rule_extremes(rule, alpha):
    """alpha < 0 defers every token under V2/V3 (eta = 1, the target is p);
    alpha >= 1 under V1/V2 and V3 at alpha >= 1 (threshold <= 0) defers none
    (eta = 0, the target is q)."""
    for cfg in (3, 2):
        wl = W.WORKLOADS[cfg].with_(B=8, V=30000, rule=rule, alpha=alpha)
        inp = W.generate(wl, 12, DEV)
        g = parity.run_gpu(inp)
        h = parity.host_inputs(inp)
        parity.compare(g, parity.run_oracle(h), h, wl.dtype)
        eta = g["row_stats"][..., 6]
        if alpha < 0:
            np.testing.assert_allclose(eta, 1.0, rtol=0, atol=1e-5)
            assert (g["defer"][:, :-1] == 1).all()
        else:
            assert (eta == 0).all()
            assert (g["defer"] == 0).all()
            assert (g["accept_len"] == wl.gamma).all()


def test_token_rules_mixed_per_sequence():
    """Token rules next to sequence-level rules and per-sequence temperatures."""
    wl = W.WORKLOADS[5].with_(B=24, V=30000)
    inp = W.generate(wl, 8, DEV)
    rules = [W.TOKEN_V1, W.TOKEN_V2, W.TOKEN_V3, W.OPT, W.DIFF, W.CHOW]
    inp["rule"][:] = torch.tensor([rules[i % 6] for i in range(24)], dtype=torch.int32,
                                  device=DEV)
    inp["alpha"][:] = torch.tensor([0.05, 0.05, 0.3, 0.1, 0.05, 0.3] * 4, device=DEV)
    g = parity.run_gpu(inp)
    h = parity.host_inputs(inp)
    rep = parity.compare(g, parity.run_oracle(h), h, wl.dtype)
    _flush(f"[token] mixed {dict(rep)}")


def test_token_rule_identical_models():
    """p = q: V1 and V2 coincide (both compare q(v) with max q - alpha), and a
    draft the rule accepts is always kept, since pi(v) = q(v) (1 + eta) there."""
    wl = W.WORKLOADS[3].with_(B=16, V=20000)
    inp = W.generate(wl, 3, DEV)
    inp["p"] = inp["q"].clone()
    outs = {}
    for rule in (W.TOKEN_V1, W.TOKEN_V2, W.TOKEN_V3):
        inp["rule"][:] = rule
        inp["alpha"][:] = 0.05
        g = outs[rule] = parity.run_gpu(inp)
        for b in range(wl.B):
            j = int(g["accept_len"][b])
            if j < wl.gamma:  # a rejected draft must carry r = 1
                assert g["defer"][b, j] == 1
        h = parity.host_inputs(inp)
        parity.compare(g, parity.run_oracle(h), h, wl.dtype)
    for k in ("accept_len", "next_token", "defer", "row_stats"):
        np.testing.assert_array_equal(outs[W.TOKEN_V1][k], outs[W.TOKEN_V2][k])


# --------------------------- other targets of Tables 1 and 3 (lossy, BiLD*, log)

NEXT2_RULES = (W.LOSSY, W.BILD, W.CHOWLOG, W.DIFFLOG, W.OPTLOG)
LOSSY_ALPHAS = (0.0, 0.3, 0.7)


def _log_alphas(inp, rule, greedy):
    """Three alphas for a log-loss rule (or BiLD*) at the quartiles of its
    statistic on these inputs, taken from the oracle, so that both deferral
    outcomes occur; for OPTLOG the statistic is divided by D_TV."""
    h = parity.host_inputs(inp)
    h["rule"][:] = rule
    h["alpha"][:] = 0.0
    o = parity.run_oracle(h, greedy=greedy)
    s, tv = o["row_stats"][..., 7].ravel(), o["row_stats"][..., 6].ravel()
    keep = np.isfinite(s) & ((tv > 1e-3) if rule == W.OPTLOG else True)
    s = s[keep] / tv[keep] if rule == W.OPTLOG else s[keep]
    return [float(np.float32(x)) for x in np.quantile(s, (0.25, 0.5, 0.75))]


def _alphas(rule, inp, greedy=False):
    return LOSSY_ALPHAS if rule == W.LOSSY else _log_alphas(inp, rule, greedy)


@pytest.mark.parametrize("rule", NEXT2_RULES)
@pytest.mark.parametrize("cfg,steps", [(2, 12), (3, 3)])
def test_next2_rule_parity(rule, cfg, steps):
    """Lossy speculative decoding (Lemma 2), BiLD* and the log-loss rules on the
    T5-vocabulary float32 shape and the Gemma-vocabulary bfloat16 shape."""
    wl = W.WORKLOADS[cfg].with_(rule=rule, temperature=1.0)
    for alpha in _alphas(rule, W.generate(wl, 950, DEV)):
        wa = wl.with_(alpha=alpha)
        name = f"cfg{cfg}.{W.RULE_NAMES[rule]}.{alpha:.4g}"
        _flush(f"[next2] {name} steps={steps}")
        rep = parity.parity_workload(wa, steps, step0=950, report_name=name)
        _flush(f"[next2] {name} {dict(rep)}")
        assert rep["exact"] + rep["excused_defer"] + rep["excused_accept"] + \
            rep["excused_token"] == rep["sequences"]


@pytest.mark.parametrize("rule", NEXT2_RULES)
def test_next2_plain_entry_point(rule):
    """Batch-wide spc_verify at the benchmark's shape (moments without the
    per-sequence path)."""
    wl = W.WORKLOADS[3].with_(rule=rule)
    alpha = _alphas(rule, W.generate(wl, 720, DEV))[1]
    rep = parity.parity_workload(wl.with_(alpha=alpha), 2, stats=False, step0=720,
                                 report_name=f"cfg3.plain.{W.RULE_NAMES[rule]}")
    assert rep["sequences"] == 2 * 32


@pytest.mark.parametrize("rule", NEXT2_RULES)
def test_next2_greedy_parity(rule):
    """Temperature 0: log-loss rules on temperature-1 entropies, BiLD* with
    D = -log p(argmax q), lossy's one-hot target at argmax p."""
    wl = W.WORKLOADS[4].with_(B=64, V=50000, rule=rule)
    for alpha in _alphas(rule, W.generate(wl, 310, DEV), greedy=True):
        _flush(f"[next2] greedy {W.RULE_NAMES[rule]} alpha={alpha:.4g}")
        parity.parity_workload(wl.with_(alpha=alpha), 3, step0=310,
                               report_name=f"greedy.{W.RULE_NAMES[rule]}")


def test_lossy_alpha0_is_speculative_sampling():
    """Lemma 2 at alpha = 0 (beta = 1): the target is p, so every draw matches
    the always-defer rule (standard speculative sampling) exactly."""
    for cfg in (3, 2):
        wl = W.WORKLOADS[cfg].with_(B=16, V=40000)
        inp = W.generate(wl, 21, DEV)
        out = {}
        for rule in (W.LOSSY, W.ALWAYS):
            inp["rule"][:] = rule
            inp["alpha"][:] = 0.0
            out[rule] = parity.run_gpu(inp)
        for k in ("accept_len", "next_token", "sample_norm"):
            np.testing.assert_array_equal(out[W.LOSSY][k], out[W.ALWAYS][k])
        assert (out[W.LOSSY]["defer"] == 0).all() and (out[W.ALWAYS]["defer"] == 1).all()


def test_next2_mixed_per_sequence():
    """The new rules next to Table 1 and token rules, with per-sequence
    temperatures including 0 (the argmax-and-moments statistics kernel)."""
    wl = W.WORKLOADS[5].with_(B=30, V=30000)
    inp = W.generate(wl, 17, DEV)
    rules = [W.LOSSY, W.BILD, W.CHOWLOG, W.DIFFLOG, W.OPTLOG, W.DIFF, W.TOKEN_V2, W.OPT]
    alphas = {W.LOSSY: 0.3, W.BILD: 7.5, W.CHOWLOG: 6.5, W.DIFFLOG: 0.5, W.OPTLOG: 1.5,
              W.DIFF: 0.05, W.TOKEN_V2: 0.05, W.OPT: 0.1}
    sel = [rules[i % len(rules)] for i in range(wl.B)]
    inp["rule"][:] = torch.tensor(sel, dtype=torch.int32, device=DEV)
    inp["alpha"][:] = torch.tensor([alphas[r] for r in sel], device=DEV)
    inp["temperature"][::4] = 0.0
    g = parity.run_gpu(inp)
    h = parity.host_inputs(inp)
    greedy = h["temperature"] == 0
    for s, gr in ((greedy, True), (~greedy, False)):
        hs = {k: v[s] for k, v in h.items()}
        gs = {k: v[s] for k, v in g.items()}
        rep = parity.compare(gs, parity.run_oracle(hs, greedy=gr), hs, wl.dtype, greedy=gr)
        _flush(f"[next2] mixed greedy={gr} {dict(rep)}")


@pytest.mark.parametrize("rule,alpha", [(W.BILD, 6.0), (W.OPTLOG, 1.0), (W.LOSSY, 0.3),
                                        (W.CHOWLOG, 5.0)])
def test_next2_masked_logits(rule, alpha):
    """-inf entries in both tensors: BiLD*'s cross-entropy is infinite where q
    keeps mass on a token p masks."""
    for cfg, dtype in ((3, "bf16"), (2, "f32")):
        wl = W.WORKLOADS[cfg].with_(B=8, V=12345, dtype=dtype, rule=rule, alpha=alpha)
        inp = W.generate(wl, 2, DEV)
        g0 = torch.Generator(device=DEV).manual_seed(98)
        for k in ("q", "p"):
            m = torch.rand(inp[k].shape, generator=g0, device=DEV) < 0.3
            m[..., 0] = False
            if k == "p" and rule == W.BILD:
                m[::2] = False  # half the sequences keep a finite cross-entropy
            inp[k][m] = float("-inf")
        inp["draft"] = W.draw_drafts(inp["q"], inp["temperature"], g0)
        g = parity.run_gpu(inp)
        h = parity.host_inputs(inp)
        rep = parity.compare(g, parity.run_oracle(h), h, wl.dtype)
        if rule == W.BILD:
            assert rep["inf_stat7"] > 0


def test_next2_out_of_range_and_identical():
    """Out-of-range drafts are rejected under every new rule; with p = q the
    log-loss difference is 0 and lossy decoding keeps every draft."""
    wl = W.WORKLOADS[3].with_(B=8, V=3000)
    inp = W.generate(wl, 1, DEV)
    inp["draft"][:, 2] = torch.tensor([-1, 3000, 1 << 30, -(1 << 30), 2999, 0, -5, 3001],
                                      dtype=torch.int32, device=DEV)
    inp["uniforms"][:, :2] = 0.0
    for rule, alpha in ((W.LOSSY, 0.3), (W.BILD, 5.0), (W.CHOWLOG, 4.0), (W.DIFFLOG, 0.2),
                        (W.OPTLOG, 0.5)):
        inp["rule"][:] = rule
        inp["alpha"][:] = alpha
        g = parity.run_gpu(inp)
        h = parity.host_inputs(inp)
        parity.compare(g, parity.run_oracle(h), h, wl.dtype)
    same = W.generate(wl.with_(B=16, V=20000), 3, DEV)
    same["p"] = same["q"].clone()
    for rule, alpha in ((W.LOSSY, 0.3), (W.DIFFLOG, 0.0), (W.OPTLOG, 0.5)):
        same["rule"][:] = rule
        same["alpha"][:] = alpha
        g = parity.run_gpu(same)
        assert (g["accept_len"] == wl.gamma).all()
        assert (g["defer"] == 0).all()
        h = parity.host_inputs(same)
        parity.compare(g, parity.run_oracle(h), h, wl.dtype)


def test_rules_present_hint():
    """A rules_present mask that covers the per-sequence rules changes nothing;
    a sequence whose rule lies outside it is invalid."""
    wl = W.WORKLOADS[5].with_(B=24, V=30000)
    inp = W.generate(wl, 5, DEV)
    inp["temperature"][::5] = 0.0
    mask = sum(1 << r for r, _ in W.CFG5_RULES)
    out = {}
    for m in (0, mask):
        acc, tok, dm = spc.spc_verify_ex(inp["q"], inp["p"], inp["draft"], inp["uniforms"], 0,
                                         0.0, 1.0, rule_per_seq=inp["rule"],
                                         alpha_per_seq=inp["alpha"],
                                         temp_per_seq=inp["temperature"], rules_present=m)
        torch.cuda.synchronize()
        out[m] = (acc.cpu().numpy(), tok.cpu().numpy(), dm.cpu().numpy())
    for a, b in zip(out[0], out[mask]):
        np.testing.assert_array_equal(a, b)
    inp["rule"][3] = W.BILD  # outside the mask
    acc, tok, _ = spc.spc_verify_ex(inp["q"], inp["p"], inp["draft"], inp["uniforms"], 0, 0.0,
                                    1.0, rule_per_seq=inp["rule"], alpha_per_seq=inp["alpha"],
                                    temp_per_seq=inp["temperature"], rules_present=mask)
    torch.cuda.synchronize()
    assert acc[3].item() == -1 and tok[3].item() == -1
    keep = [b for b in range(wl.B) if b != 3]
    np.testing.assert_array_equal(acc.cpu().numpy()[keep], out[0][0][keep])


# ------------------------------------------- one read vs two for the second pass

def _ex_outputs(inp, mask):
    B, g1, _ = inp["q"].shape
    stats = torch.full((B, g1, 8), float("nan"), device=DEV)
    am = torch.full((B, g1, 2), -7, dtype=torch.int32, device=DEV)
    norm = torch.full((B,), float("nan"), device=DEV)
    acc, tok, dm = spc.spc_verify_ex(inp["q"], inp["p"], inp["draft"], inp["uniforms"], 0, 0.0,
                                     1.0, rule_per_seq=inp["rule"], alpha_per_seq=inp["alpha"],
                                     temp_per_seq=inp["temperature"], out_row_stats=stats,
                                     out_argmax=am, out_sample_norm=norm, rules_present=mask)
    torch.cuda.synchronize()
    return [x.cpu().numpy() for x in (acc, tok, dm, stats, am, norm)]


# ------------------------------------------------------------- argmax ties

def _plant_ties(t, seed):
    """Give every row of t [B, g1, V] a new maximum repeated at positions that
    tie within one lane load, across the lane loads of one thread, across
    threads, workgroups and tiles, and at the row ends; returns the lowest
    index of each row's maximum."""
    B, g1, V = t.shape
    g = np.random.default_rng(seed)
    x = t.float().cpu().numpy().reshape(B * g1, V)
    low = np.empty(B * g1, np.int64)
    for r in range(B * g1):
        kind = r % 4
        if kind == 0:    # a tie at both row ends
            pos = [V - 1, 0, V - 2]
        elif kind == 1:  # ties inside one 8-entry lane load and one thread
            b0 = int(g.integers(0, V - 20000)) & ~7
            pos = [b0 + 5, b0 + 3, b0 + 3 + 2048, b0 + 3 + 6144, b0 + 7]
        elif kind == 2:  # ties in other threads, workgroups and tiles
            b0 = int(g.integers(0, V - 20000))
            pos = [b0 + 8192 + 1, b0 + 9, b0 + 8 * 64 + 9, b0 + 8192 * 2]
        else:            # many random ties
            pos = list(g.choice(V, size=40, replace=False))
        m = float(np.ceil(x[r].max())) + 1.0
        x[r, pos] = m
        low[r] = min(pos)
    t.copy_(torch.from_numpy(x.reshape(B, g1, V)).to(t.dtype))
    return low.reshape(B, g1)


@pytest.mark.parametrize("dtype,V", [("bf16", 50000), ("f32", 50000), ("bf16", 50003)])
def test_argmax_ties_lowest_index(dtype, V):
    """Greedy rows (per-sequence temperatures 0 and >0 mixed, and the
    batch-wide greedy entry point) take the lowest index attaining the
    maximum on both tensors, as the oracle does."""
    wl = W.WORKLOADS[4].with_(B=16, V=V, dtype=dtype)
    inp = W.generate(wl, 9, DEV)
    lq = _plant_ties(inp["q"], 1)
    lp = _plant_ties(inp["p"], 2)
    _flush(f"[ties] {dtype} V={V}")
    g = parity.run_gpu(inp, greedy=True)
    np.testing.assert_array_equal(g["argmax"][..., 0], lq)
    np.testing.assert_array_equal(g["argmax"][..., 1], lp)
    h = parity.host_inputs(inp)
    parity.compare(g, parity.run_oracle(h, greedy=True), h, dtype, greedy=True)
    # the same rows inside a batch that also samples
    inp["temperature"][1::2] = 0.7
    g2 = parity.run_gpu(inp)
    sel = np.arange(wl.B) % 2 == 0
    np.testing.assert_array_equal(g2["argmax"][sel][..., 0], lq[sel])
    np.testing.assert_array_equal(g2["argmax"][sel][..., 1], lp[sel])


# ------------------------------------------------- more than 64 tiles per row

@pytest.mark.parametrize("dtype,V,rule,alpha", [
    ("bf16", 600000, W.DIFF, 0.05),      # 74 tiles per row
    ("bf16", 600001, W.OPT, 0.1),        # unaligned rows: 293 tiles, 3 groups of part loads
    ("f32", 1100000, W.TOKEN_V3, 0.3),   # 269 tiles
    ("bf16", 600000, W.DIFFLOG, 0.5),    # moments merged over 74 tiles
])
def test_large_vocabulary(dtype, V, rule, alpha):
    """Rows of more than 64 statistics tiles: the merge takes several partials
    per lane and the draw's part search loads several groups."""
    wl = W.WORKLOADS[3].with_(B=3, gamma=3, V=V, dtype=dtype, rule=rule, alpha=alpha)
    _flush(f"[large] {dtype} V={V} rule={rule}")
    rep = parity.parity_workload(wl, 2, report_name=f"large.{dtype}.{V}.{rule}")
    assert rep["sequences"] == 2 * wl.B
    greedy = parity.parity_workload(wl.with_(temperature=0.0, cfg=4), 1,
                                    report_name=f"large.{dtype}.{V}.{rule}.g")
    assert greedy["sequences"] == wl.B


def test_verify_ex_scalar_temperature_zero_is_greedy_step():
    """spc_verify_ex with a scalar temperature of 0 runs spc_greedy_verify's
    step (uniforms not needed) and fills the optional outputs."""
    wl = W.WORKLOADS[4].with_(B=16, V=30000)
    inp = W.generate(wl, 3, DEV)
    a = spc.spc_greedy_verify(inp["q"], inp["p"], inp["draft"], wl.rule, wl.alpha)
    stats = torch.full((wl.B, wl.gamma + 1, 8), float("nan"), device=DEV)
    am = torch.full((wl.B, wl.gamma + 1, 2), -7, dtype=torch.int32, device=DEV)
    b = spc.spc_verify_ex(inp["q"], inp["p"], inp["draft"], None, wl.rule, wl.alpha, 0.0,
                          out_row_stats=stats, out_argmax=am)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x.cpu().numpy(), y.cpu().numpy())
    g = parity.run_gpu(inp, greedy=True)  # per-sequence zero temperatures
    np.testing.assert_array_equal(am.cpu().numpy(), g["argmax"])
    np.testing.assert_allclose(stats.cpu().numpy(), g["row_stats"], rtol=0, atol=0)
