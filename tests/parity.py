"""GPU-vs-oracle parity harness shared by the GPU tests, the smoke check and
the benchmark's parity leg.

Rule (applied per sequence, in the order delta_j for all j, accept draws up to
j*, j*, token): outputs must be identical, except that the FIRST mismatch may
sit on an oracle decision whose margin is below NEAR (a near-tie); such a
sequence is counted as excused and its later outputs, which depend on that
decision, are not compared.  For a token rule every r(v) of a row feeds eta,
so the oracle's row margin is the smallest relative r-margin over the row,
and a near-tie there excuses the sequence's later outputs too.

Every call checks the accounting: each sequence is exact or excused once,
each kind of excusal is bounded by the number of near-ties of that kind the
oracle reports, and token-rule near-ties stay below ETA_FRAC of the
token-rule sequences.

Row statistics and the sampled mass W must agree to ARITH_TOL relative with
the floors in FLOOR below, for both input dtypes (inside the 1e-5 / 2e-3
contract for float32 / bfloat16 logits): both sides compute them from the
exactly widened logits, the kernels in float32 exponentials summed in
float64, so the input dtype does not enter their error.
"""
import json
import os
from collections import Counter

import numpy as np
import torch

import oracle
from paper_2405_19261_amd import spc
from paper_2405_19261_amd import workloads as W

NEAR = 1e-6
TOKEN_RULES = (W.TOKEN_V1, W.TOKEN_V2, W.TOKEN_V3)
# The contract on floating outputs, per input dtype ...
FLOAT_TOL = {"f32": 1e-5, "bf16": 2e-3}
# ... and the bound the arithmetic gives, which the checks apply to both:
# every probability carries a relative error of a few float32 ulps (float32
# exp2 of an exactly scaled logit, float64 sums, a log-normaliser good to
# ~1e-7), so the measured errors sit near 1e-7.
ARITH_TOL = 1e-5
# Floors of the relative criterion, per row-statistic column
# {m_q, lse_q, maxprob_q, m_p, lse_p, maxprob_p, tv, log statistic}: m and
# lse are log-scale (an absolute error e there is a relative error e in every
# probability), so their floor is 1.  TV (and eta) and the sampled mass W are
# sums of probability differences: each term carries the relative error of
# its probabilities, so the absolute error is ~1e-7 times the mass summed,
# whatever the difference; below 0.1 they are held to ARITH_TOL * 0.1 = 1e-6
# absolute.  Column 7 is a log-loss statistic in nats (D, H(q) or
# H(q) - H(p)), whose entropies (~log V) carry absolute errors of ~1e-7 each:
# floor 1, i.e. 1e-5 nats absolute.
FLOOR = {0: 1.0, 1: 1.0, 2: 1e-6, 3: 1.0, 4: 1.0, 5: 1e-6, 6: 0.1, 7: 1.0}
# Excusals and the near-ties that bound them.
EXCUSE_OF = {"excused_defer": "near_defer", "excused_accept": "near_accept",
             "excused_token": "near_token", "excused_eta": "near_eta_seqs"}
# Token-rule sequences with an r(v) near-tie on some row: at most this
# fraction of the token-rule sequences (plus one).  The seeded token-rule
# workloads show at most 2 in 320 (0.6%, T5 vocabulary), none at the Gemma
# vocabulary.
ETA_FRAC = 0.02
LOG_RULES = (W.BILD, W.CHOWLOG, W.DIFFLOG, W.OPTLOG)
TV_RULES = (W.OPT, W.OPTLOG)


def host_logits(t):
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def _uniform_params(inp):
    r, a, t = inp["rule"], inp["alpha"], inp["temperature"]
    if bool((r == r[0]).all()) and bool((a == a[0]).all()) and bool((t == t[0]).all()):
        return int(r[0]), float(a[0]), float(t[0])
    return None


def rules_mask(rule):
    """rules_present bitmask of the valid rule ids in a per-sequence array."""
    return sum(1 << r for r in set(int(x) for x in rule.tolist()) if 0 <= r <= W.OPTLOG)


def run_gpu(inp, greedy=False, stats=True, stream=None, per_seq=False):
    """One call through the C interface; returns numpy outputs.  Batch-wide
    parameters go through spc_verify / spc_greedy_verify (the entry points
    the benchmark times), or with statistics the scalar form of
    spc_verify_ex.  Per-sequence parameters go through spc_verify_ex with the
    arrays and the rules the batch holds (rules_present), as the benchmark's
    mixed workload does; per_seq sends batch-wide parameters that way too."""
    q, p = inp["q"], inp["p"]
    B, g1, V = q.shape
    dev = q.device
    row_stats = torch.full((B, g1, 8), float("nan"), device=dev) if stats else None
    argmax = torch.full((B, g1, 2), -7, dtype=torch.int32, device=dev) if stats else None
    norm = torch.full((B,), float("nan"), device=dev) if stats else None
    uni = None if per_seq else _uniform_params(inp)
    if greedy and not stats and uni is not None:
        acc, tok, dm = spc.spc_greedy_verify(q, p, inp["draft"], uni[0], uni[1], stream=stream)
    elif not greedy and not stats and uni is not None:
        acc, tok, dm = spc.spc_verify(q, p, inp["draft"], inp["uniforms"], *uni, stream=stream)
    elif uni is not None:
        # batch-wide parameters with the optional outputs: the scalar form of
        # spc_verify_ex (temperature 0: the batch-wide greedy step)
        acc, tok, dm = spc.spc_verify_ex(
            q, p, inp["draft"], None if greedy else inp["uniforms"], uni[0], uni[1],
            0.0 if greedy else uni[2], out_row_stats=row_stats, out_argmax=argmax,
            out_sample_norm=norm, stream=stream)
    else:
        temp = inp["temperature"]
        acc, tok, dm = spc.spc_verify_ex(
            q, p, inp["draft"], inp["uniforms"], 0, 0.0, 1.0, rule_per_seq=inp["rule"],
            alpha_per_seq=inp["alpha"], temp_per_seq=(torch.zeros_like(temp) if greedy else temp),
            out_row_stats=row_stats, out_argmax=argmax, out_sample_norm=norm, stream=stream,
            rules_present=rules_mask(inp["rule"]))
    torch.cuda.synchronize()
    out = dict(accept_len=acc.cpu().numpy(), next_token=tok.cpu().numpy(),
               defer=dm.cpu().numpy())
    if stats:
        out.update(row_stats=row_stats.cpu().numpy(), argmax=argmax.cpu().numpy(),
                   sample_norm=norm.cpu().numpy())
    return out


def host_inputs(inp):
    return dict(q=host_logits(inp["q"]), p=host_logits(inp["p"]),
                draft=inp["draft"].cpu().numpy(), uniforms=inp["uniforms"].cpu().numpy(),
                rule=inp["rule"].cpu().numpy(), alpha=inp["alpha"].cpu().numpy(),
                temperature=inp["temperature"].cpu().numpy())


def run_oracle(h, greedy=False):
    if greedy:
        return oracle.greedy_verify(h["q"], h["p"], h["draft"], h["rule"], h["alpha"])
    return oracle.verify(h["q"], h["p"], h["draft"], h["uniforms"], h["rule"], h["alpha"],
                         h["temperature"])


def check_accounting(rep):
    """Each sequence exact or excused once; excusals within their near-ties."""
    excused = sum(rep[k] for k in EXCUSE_OF)
    assert rep["exact"] + excused == rep["sequences"], dict(rep)
    for k, n in EXCUSE_OF.items():
        assert rep[k] <= rep[n], f"{k}={rep[k]} exceeds {n}={rep[n]}"
    assert rep["near_eta_seqs"] <= 1 + ETA_FRAC * rep["token_seqs"], \
        f"token-rule near-ties on {rep['near_eta_seqs']} of {rep['token_seqs']} sequences"


def compare(g, o, h, dtype, greedy=False, rep=None):
    """Margin-aware comparison of one call; returns (and accumulates) a Counter."""
    rep = Counter() if rep is None else rep
    B, g1 = o["defer"].shape
    gamma = g1 - 1
    tol = min(FLOAT_TOL[dtype], ARITH_TOL)
    for k in ("exact", "token_seqs", *EXCUSE_OF, *EXCUSE_OF.values()):
        rep[k] += 0
    for b in range(B):
        rep["sequences"] += 1
        if not greedy and int(h["rule"][b]) in TOKEN_RULES:
            rep["token_seqs"] += 1
            rep["near_eta_seqs"] += int(o["defer_margin"][b].min() < NEAR)
        # near-ties among the decisions the oracle actually took
        jo = int(o["accept_len"][b])
        rep["near_defer"] += int((o["defer_margin"][b] < NEAR).sum())
        if not greedy:
            rep["near_accept"] += int((o["accept_margin"][b, :jo + 1 if jo < gamma else gamma]
                                       < NEAR).sum())
            rep["near_token"] += int(o["sample_margin"][b] < NEAR)
        bad = np.flatnonzero(g["defer"][b] != o["defer"][b])
        if bad.size:
            j = int(bad[0])
            m = o["defer_margin"][b, j]
            assert m < NEAR, f"seq {b}: defer[{j}] gpu={g['defer'][b, j]} oracle=" \
                             f"{o['defer'][b, j]} margin={m:.3g}"
            rep["excused_defer"] += 1
            continue
        ja = int(g["accept_len"][b])
        # token rules: a near-tie in any r(v) of a row up to j* moves eta
        eta_near = not greedy and int(h["rule"][b]) in TOKEN_RULES and \
            o["defer_margin"][b, :max(ja, jo) + 1].min() < NEAR
        if (ja != jo or g["next_token"][b] != o["next_token"][b]) and eta_near:
            rep["excused_eta"] += 1
            continue
        if ja != jo:
            j = min(ja, jo)
            m = 0.0 if greedy else o["accept_margin"][b, j]
            assert m < NEAR, f"seq {b}: accept_len gpu={ja} oracle={jo} margin a_{j}={m:.3g}"
            rep["excused_accept"] += 1
            continue
        if g["next_token"][b] != o["next_token"][b]:
            m = 0.0 if greedy else o["sample_margin"][b]
            assert m < NEAR, f"seq {b}: token gpu={g['next_token'][b]} oracle=" \
                             f"{o['next_token'][b]} margin={m:.3g} (j*={jo})"
            rep["excused_token"] += 1
            continue
        rep["exact"] += 1
    if "row_stats" in g:
        gs, os_ = g["row_stats"].astype(np.float64), o["row_stats"]
        opt_rows = np.isin(h["rule"], TV_RULES + TOKEN_RULES)[:, None] & np.ones((1, g1), bool)
        # eta of a token row with a near-tie r(v) is the exact sum only up to
        # the q mass of the tied tokens (greedy: column 6 is r at argmax q,
        # whose near-tie the defer check excused): such rows, and the
        # normalisers drawn from them, are counted, not compared
        tok_near = np.isin(h["rule"], TOKEN_RULES)[:, None] & (o["defer_margin"] < NEAR)
        opt_rows &= ~tok_near
        rep["near_eta_rows"] += int(tok_near.sum())
        cols = [0, 1, 2, 3, 4, 5]
        for c in cols + [6, 7]:
            sel = np.ones(gs.shape[:2], bool) if c != 6 else (opt_rows if not greedy else
                                                             ~tok_near)
            if c == 7:
                # the same infinite cross-entropy (q mass where p is 0) agrees
                same_inf = np.isinf(gs[..., 7]) & (gs[..., 7] == os_[..., 7])
                sel = sel & ~same_inf
                rep["inf_stat7"] += int(same_inf.sum())
            if not sel.any():
                continue
            err = np.abs(gs[..., c] - os_[..., c])[sel] / np.maximum(np.abs(os_[..., c][sel]),
                                                                        FLOOR[c])
            rep[f"maxrel_stat{c}"] = max(rep.get(f"maxrel_stat{c}", 0.0), float(err.max()))
            rep[f"maxabs_stat{c}"] = max(rep.get(f"maxabs_stat{c}", 0.0),
                                         float(np.abs(gs[..., c] - os_[..., c])[sel].max()))
            assert err.max() <= tol, f"row stat {c}: max rel err {err.max():.3g} > {tol}"
        if greedy:
            np.testing.assert_array_equal(g["argmax"], o["argmax"])
        else:
            ok = g["accept_len"] == o["accept_len"]
            ok &= ~np.array([tok_near[b, :jo + 1].any() for b, jo in enumerate(o["accept_len"])])
            if ok.any():
                err = np.abs(g["sample_norm"][ok] - o["sample_norm"][ok]) / np.maximum(
                    np.abs(o["sample_norm"][ok]), FLOOR[6])
                rep["maxrel_norm"] = max(rep.get("maxrel_norm", 0.0), float(err.max()))
                assert err.max() <= tol, f"sample norm: max rel err {err.max():.3g}"
    check_accounting(rep)
    return rep


def parity_workload(wl, steps, device="cuda", stats=True, step0=0, report_name=None):
    """Run `steps` seeded steps of workload `wl` on the GPU and the oracle."""
    rep = Counter()
    for s in range(step0, step0 + steps):
        inp = W.generate(wl, s, device)
        g = run_gpu(inp, greedy=wl.greedy, stats=stats)
        h = host_inputs(inp)
        del inp
        o = run_oracle(h, greedy=wl.greedy)
        compare(g, o, h, wl.dtype, greedy=wl.greedy, rep=rep)
    rep["steps"] = steps
    write_report(report_name or f"cfg{wl.cfg}", wl, rep)
    return rep


def write_report(name, wl, rep):
    path = os.environ.get("SPC_PARITY_REPORT")
    if not path:
        return
    with open(path, "a") as f:
        f.write(json.dumps(dict(name=name, workload=wl.name, B=wl.B, gamma=wl.gamma, V=wl.V,
                                **{k: v for k, v in rep.items()})) + "\n")
