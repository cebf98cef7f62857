"""Pins of the oracle's other targets of Tables 1 and 3.

Lossy speculative decoding (Lemma 2, beta = 1), BiLD* with the cross-entropy
discrepancy, and the log-loss rules ChowLog, DiffLog and OPTLog.  Checks use
closed forms (entropy of a uniform row, D(q, q) = H(q), D = H + KL), scipy's
entropy and relative entropy as library pins, Lemma 2's acceptance and
residual formulas, reductions to standard speculative sampling and to the
drafter, exhaustive first-token laws, and hand cases at temperature 0.
"""
import math

import numpy as np
import pytest
from scipy.special import rel_entr
from scipy.stats import entropy as scipy_entropy

from test_oracle_pins import (_first_token_law, _random_step, _rng, _softmax64,
                              _textbook_specdecode)

LOSSY, BILD, CHOWLOG, DIFFLOG, OPTLOG = 8, 9, 10, 11, 12
ALWAYS = 3


# ----------------------------------------------------------------- entropies

@pytest.mark.parametrize("V", [1, 2, 7, 1000])
def test_entropy_uniform_row_is_log_v(orc, V):
    assert orc.entropy_row(np.full(V, 3.25)) == pytest.approx(math.log(V), abs=1e-12)


def test_entropy_single_live_entry_is_zero(orc):
    z = np.full(50, -np.inf)
    z[17] = 1.5
    assert orc.entropy_row(z) == 0.0


@pytest.mark.parametrize("T", [1.0, 0.5, 2.0])
def test_entropy_matches_scipy(orc, T):
    r = _rng(200)
    for _ in range(10):
        z = r.normal(0, 3, int(r.integers(2, 3000)))
        assert orc.entropy_row(z, T) == pytest.approx(scipy_entropy(_softmax64(z, T)), rel=1e-12)


def test_entropy_masked_entries_contribute_nothing(orc):
    r = _rng(201)
    z = r.normal(0, 2, 400)
    zm = z.copy()
    zm[::3] = -np.inf
    assert orc.entropy_row(zm) == pytest.approx(scipy_entropy(_softmax64(z[np.isfinite(zm)])),
                                                rel=1e-12)


def test_cross_entropy_closed_forms(orc):
    r = _rng(202)
    for T in (1.0, 0.6):
        for _ in range(10):
            V = int(r.integers(2, 2000))
            zq, zp = r.normal(0, 2, V), r.normal(0, 2, V)
            q, p = _softmax64(zq, T), _softmax64(zp, T)
            # D(q, q) = H(q)
            assert orc.cross_entropy_row(zq, zq, T) == pytest.approx(orc.entropy_row(zq, T),
                                                                     rel=1e-12)
            # D(q, p) = H(q) + KL(q || p), KL from scipy
            assert orc.cross_entropy_row(zq, zp, T) == pytest.approx(
                scipy_entropy(q) + rel_entr(q, p).sum(), rel=1e-11)


def test_cross_entropy_infinite_where_p_vanishes(orc):
    zq = np.array([0.0, 1.0, -np.inf, 2.0])
    zp = np.array([0.0, 0.5, 1.0, 1.0])
    zp_masked = zp.copy()
    zp_masked[1] = -np.inf
    assert orc.cross_entropy_row(zq, zp_masked) == np.inf
    # a verifier zero where the drafter is zero too costs nothing
    zp_both = zp.copy()
    zp_both[2] = -np.inf
    q = _softmax64(zq)
    keep = np.isfinite(zq)
    lp = zp_both - np.log(np.exp(zp_both[np.isfinite(zp_both)]).sum())
    assert orc.cross_entropy_row(zq, zp_both) == pytest.approx(-(q[keep] * lp[keep]).sum(),
                                                               rel=1e-12)


def test_log_defer_strict_and_margin(orc):
    assert orc.log_defer(2.5, 2.0) == (1, pytest.approx(0.2))     # |0.5| / 2.5
    assert orc.log_defer(2.0, 2.0) == (0, 0.0)                    # strict: no deferral
    assert orc.log_defer(0.1, 0.3) == (0, pytest.approx(0.2))     # scale floor 1
    assert orc.log_defer(np.inf, 5.0) == (1, np.inf)
    # a difference of entropies is rounded relative to the entropies
    assert orc.log_defer(0.5, 0.4, 8.0) == (1, pytest.approx(0.1 / 8.0))


# ------------------------------------------------------------- lossy (Lemma 2)

@pytest.mark.parametrize("alpha", [0.0, 0.1, 0.5, 0.9])
def test_lossy_acceptance_and_residual_are_lemma_2(orc, alpha):
    """With pi = max{min{q, p/(1-alpha)}, p}: min(1, pi/q) is the lossy
    acceptance min(1, p/((1-alpha) q)), and max(0, pi - q) is max(0, p - q)."""
    r = _rng(210)
    for _ in range(20):
        V = int(r.integers(2, 500))
        q = _softmax64(r.normal(0, 2, V))
        p = _softmax64(r.normal(0, 2, V))
        pi = orc.lossy_target(alpha, q, p)
        np.testing.assert_allclose(np.minimum(1.0, pi / q),
                                   np.minimum(1.0, p / ((1.0 - alpha) * q)), rtol=1e-14)
        np.testing.assert_allclose(np.maximum(0.0, pi - q), np.maximum(0.0, p - q),
                                   rtol=0, atol=1e-17)


@pytest.mark.parametrize("alpha", [0.0, -0.5])
def test_lossy_without_slack_is_speculative_decoding(orc, alpha):
    """alpha <= 0 makes pi = p: standard speculative sampling, extra token from p."""
    qz, pz, draft, u = _random_step(211, 200, 4, 50)
    ref_acc, ref_tok = _textbook_specdecode(qz, pz, draft, u, 1.0)
    out = orc.verify(qz, pz, draft, u, LOSSY, alpha, 1.0)
    assert (out["defer"] == 0).all()
    ok = (out["accept_len"] == ref_acc) & (out["next_token"] == ref_tok)
    for b in np.flatnonzero(~ok):
        assert min(out["accept_margin"][b].min(), out["sample_margin"][b]) < 1e-9, b
    assert ok.mean() > 0.99


def test_lossy_procedure_written_independently(orc):
    """Tran-Thien's lossy procedure with beta = 1, restated in the test: keep x
    with probability min(1, p/((1-alpha) q)); replace from norm(max(0, p - q));
    if every draft is kept, draw the extra token from p."""
    for alpha, T, seed in ((0.3, 1.0, 212), (0.8, 0.7, 213)):
        qz, pz, draft, u = _random_step(seed, 150, 3, 40, T=T)
        out = orc.verify(qz, pz, draft, u, LOSSY, alpha, T)
        for b in range(150):
            qs, ps = _softmax64(qz[b], T), _softmax64(pz[b], T)
            n = 3
            for j in range(3):
                x = draft[b, j]
                if not (u[b, j] < min(1.0, ps[j, x] / ((1 - alpha) * qs[j, x]))):
                    n = j
                    break
            dist = np.maximum(0.0, ps[n] - qs[n]) if n < 3 else ps[3]
            tok = np.searchsorted(np.cumsum(dist) / dist.sum(), np.float64(u[b, 3]),
                                  side="right")
            if (out["accept_len"][b], out["next_token"][b]) != (n, tok):
                m = min(out["accept_margin"][b].min(), out["sample_margin"][b])
                assert m < 1e-9, b


def test_lossy_first_token_law(orc):
    """Exhaustive law of the first emitted token: q(v) min(1, pi/q) plus the
    rejection mass sum max(0, q - pi) spread by norm(max(0, p - q))."""
    r = _rng(214)
    V, alpha = 6, 0.4
    pz = r.normal(0, 1.5, (1, 2, V))
    qz = r.normal(0, 1.5, (1, 2, V))
    law, bonus, _ = _first_token_law(orc, qz, pz, LOSSY, alpha, 1.0)
    q0, p0 = _softmax64(qz[0, 0]), _softmax64(pz[0, 0])
    acc = np.minimum(1.0, p0 / ((1 - alpha) * q0))
    res = np.maximum(0.0, p0 - q0)
    expect = q0 * acc + (q0 * (1 - acc)).sum() * res / res.sum()
    N = 1 << 14
    np.testing.assert_allclose(law, expect, atol=3.0 / N)
    np.testing.assert_allclose(bonus, _softmax64(pz[0, 1]), atol=2.0 / N)


def test_lossy_greedy_is_greedy_speculative_decoding(orc):
    r = _rng(215)
    B, gamma, V = 300, 4, 12
    pz = r.normal(0, 1, (B, gamma + 1, V))
    qz = pz + r.normal(0, 0.8, (B, gamma + 1, V))
    draft = np.argmax(qz[:, :gamma], -1).astype(np.int32)
    a = orc.greedy_verify(qz, pz, draft, LOSSY, 0.5)
    b = orc.greedy_verify(qz, pz, draft, ALWAYS, 0.0)
    np.testing.assert_array_equal(a["accept_len"], b["accept_len"])
    np.testing.assert_array_equal(a["next_token"], b["next_token"])
    assert (a["defer"] == 0).all()


# ------------------------------------------------------ BiLD* and log rules

def _stat_independent(rule, qz, pz, T):
    q, p = _softmax64(qz, T), _softmax64(pz, T)
    hq, hp = scipy_entropy(q), scipy_entropy(p)
    if rule == BILD:
        return scipy_entropy(q) + rel_entr(q, p).sum()
    if rule == CHOWLOG:
        return hq
    return hq - hp


@pytest.mark.parametrize("rule", [BILD, CHOWLOG, DIFFLOG, OPTLOG])
@pytest.mark.parametrize("T", [1.0, 0.6])
def test_log_rule_delta_and_statistic(orc, rule, T):
    """delta and row statistic column 7 against scipy restatements; column 6
    carries D_TV for OPTLog."""
    T = float(np.float32(T))  # the temperature the oracle receives
    qz, pz, draft, u = _random_step(220 + rule, 60, 3, 300, T=T, noise=1.5)
    for alpha in (0.0, 0.2, 1.0, 3.0):
        out = orc.verify(qz, pz, draft, u, rule, alpha, T)
        for b in range(60):
            for j in range(4):
                s = _stat_independent(rule, qz[b, j], pz[b, j], T)
                assert out["row_stats"][b, j, 7] == pytest.approx(s, rel=1e-10, abs=1e-12)
                th = alpha
                if rule == OPTLOG:
                    q, p = _softmax64(qz[b, j], T), _softmax64(pz[b, j], T)
                    th = alpha * np.maximum(0, p - q).sum()
                if abs(s - th) > 1e-9:
                    assert out["defer"][b, j] == int(s > th)


@pytest.mark.parametrize("rule", [BILD, CHOWLOG])
def test_negative_alpha_defers_everywhere(orc, rule):
    """D and H are non-negative, so alpha < 0 gives delta = 1: speculative sampling."""
    qz, pz, draft, u = _random_step(230 + rule, 150, 3, 40)
    ref_acc, ref_tok = _textbook_specdecode(qz, pz, draft, u, 1.0)
    out = orc.verify(qz, pz, draft, u, rule, -0.01, 1.0)
    assert (out["defer"] == 1).all()
    ok = (out["accept_len"] == ref_acc) & (out["next_token"] == ref_tok)
    for b in np.flatnonzero(~ok):
        assert min(out["accept_margin"][b].min(), out["sample_margin"][b]) < 1e-9, b


@pytest.mark.parametrize("rule", [BILD, CHOWLOG, DIFFLOG])
def test_large_alpha_samples_drafter(orc, rule):
    """alpha above log V bounds every statistic (D is finite here but can
    exceed log V, so BiLD's alpha is taken far above the rows' D)."""
    qz, pz, draft, u = _random_step(240 + rule, 80, 3, 30)
    alpha = 1e3
    out = orc.verify(qz, pz, draft, u, rule, alpha, 1.0)
    assert (out["defer"] == 0).all()
    assert (out["accept_len"] == 3).all()


def test_identical_models_never_defer_under_difference_rules(orc):
    """p = q: H(q) - H(p) = 0 and D_TV = 0, so DiffLog and OPTLog keep q for alpha >= 0."""
    qz, _, draft, u = _random_step(250, 50, 3, 40)
    for rule in (DIFFLOG, OPTLOG):
        out = orc.verify(qz, qz, draft, u, rule, 0.0, 1.0)
        assert (out["defer"] == 0).all()
        assert (out["accept_len"] == 3).all()


@pytest.mark.parametrize("rule,alpha,seed", [(BILD, 1.5, 260), (CHOWLOG, 1.2, 261),
                                             (DIFFLOG, 0.05, 262), (OPTLOG, 0.3, 263)])
def test_log_rule_emitted_token_law(orc, rule, alpha, seed):
    """The first emitted token is distributed as T_delta(q, p) with the rule's delta."""
    r = _rng(seed)
    V = 6
    pz = r.normal(0, 1.5, (1, 2, V))
    qz = r.normal(0, 1.5, (1, 2, V))
    law, bonus, defer = _first_token_law(orc, qz, pz, rule, alpha, 1.0)
    q0, p0 = _softmax64(qz[0, 0]), _softmax64(pz[0, 0])
    q1, p1 = _softmax64(qz[0, 1]), _softmax64(pz[0, 1])
    N = 1 << 14
    np.testing.assert_allclose(law, p0 if defer[0] else q0, atol=3.0 / N)
    np.testing.assert_allclose(bonus, p1 if defer[1] else q1, atol=2.0 / N)


def test_greedy_bild_reads_log_p_at_drafter_argmax(orc):
    """T = 0: D = -log p(argmax q) with the temperature-1 p."""
    qz = np.array([[[2.0, 0.0, 1.0], [0.0, 2.0, 0.0]]])
    pz = np.array([[[-2.0, 0.0, 3.0], [0.0, 3.0, 0.0]]])
    draft = np.array([[0]], np.int32)
    d0 = -math.log(_softmax64(pz[0, 0])[0])          # about 5.02
    out = orc.greedy_verify(qz, pz, draft, BILD, 5.0)
    assert out["row_stats"][0, 0, 7] == pytest.approx(d0, rel=1e-14)
    assert out["defer"][0, 0] == 1 and out["accept_len"][0] == 0 and out["next_token"][0] == 2
    out = orc.greedy_verify(qz, pz, draft, BILD, 5.1)
    assert out["defer"][0, 0] == 0 and out["accept_len"][0] == 1 and out["next_token"][0] == 1


def test_greedy_log_rules_use_temperature_one_entropies(orc):
    r = _rng(270)
    B, gamma, V = 40, 3, 25
    pz = r.normal(0, 1.5, (B, gamma + 1, V))
    qz = r.normal(0, 1.5, (B, gamma + 1, V))
    draft = np.argmax(qz[:, :gamma], -1).astype(np.int32)
    for rule, alpha in ((CHOWLOG, 2.5), (DIFFLOG, 0.0), (OPTLOG, 0.2)):
        out = orc.greedy_verify(qz, pz, draft, rule, alpha)
        for b in range(B):
            for j in range(gamma + 1):
                s = _stat_independent(rule, qz[b, j], pz[b, j], 1.0)
                th = alpha
                if rule == OPTLOG:
                    th = alpha * float(np.argmax(qz[b, j]) != np.argmax(pz[b, j]))
                assert out["row_stats"][b, j, 7] == pytest.approx(s, rel=1e-10, abs=1e-12)
                if abs(s - th) > 1e-9:
                    assert out["defer"][b, j] == int(s > th)
