"""Pins of the oracle's token-specific rules (Section 4.4, Alg. 6).

Each check uses an independent restatement or an invariant: the target's
normalisation, the paper's Top-alpha form of TokenV3, hand-derived rule
values, the reductions r = 1 everywhere (standard speculative sampling, Alg. 1)
and r = 0 everywhere (the drafter), the exact law of the first emitted token,
and the greedy identity TokenV1 = Diff.
"""
import numpy as np
import pytest

from test_oracle_pins import (_first_token_law, _random_step, _rng, _softmax64,
                              _textbook_specdecode)

V1, V2, V3 = 5, 6, 7
DIFF = 1


def _r_independent(rule, alpha, q, p):
    """r(v) of the TokenV1/V2/V3 plug-in rules, restated with numpy."""
    mp = p.max()
    if rule == V1:
        return (q < mp - alpha).astype(np.float64)
    if rule == V2:
        return (p < mp - alpha).astype(np.float64)
    return (p < mp * (1.0 - alpha)).astype(np.float64)


@pytest.mark.parametrize("rule", [V1, V2, V3])
@pytest.mark.parametrize("alpha", [-0.3, 0.0, 0.05, 0.2, 0.7, 1.0, 1.5])
def test_token_target_is_distribution(orc, rule, alpha):
    r = _rng(100 + rule)
    for _ in range(20):
        V = int(r.integers(2, 300))
        q = _softmax64(r.normal(0, 2, V))
        p = _softmax64(r.normal(0, 2, V))
        pi, eta, _ = orc.token_target(rule, alpha, q, p, p.max())
        assert (pi >= 0).all()
        assert pi.sum() == pytest.approx(1.0, abs=1e-12)
        rr = _r_independent(rule, alpha, q, p)
        assert eta == pytest.approx(float((rr * q).sum()), abs=1e-15)
        np.testing.assert_allclose(pi, q * (1 - rr) + p * eta, rtol=0, atol=1e-15)


def test_token_v3_top_alpha_form(orc):
    """TokenV3's target is q on Top_alpha = {v: p(v) >= max p (1 - alpha)} and a
    rescaled p elsewhere, the mass of q outside Top_alpha."""
    r = _rng(110)
    for alpha in (0.0, 0.1, 0.3, 0.9):
        for _ in range(20):
            V = 64
            q = _softmax64(r.normal(0, 1.5, V))
            p = _softmax64(r.normal(0, 1.5, V))
            top = p >= p.max() * (1.0 - alpha)
            expect = np.where(top, q, 0.0) + p * q[~top].sum()
            pi, _, _ = orc.token_target(V3, alpha, q, p, p.max())
            np.testing.assert_allclose(pi, expect, rtol=0, atol=1e-15)


def test_token_rule_hand_cases(orc):
    """r on hand-picked values, strict inequalities as printed."""
    # V1: q(v) < max p - alpha
    assert orc.token_r(V1, 0.1, 0.39, 0.0, 0.5)[0] == 1
    assert orc.token_r(V1, 0.25, 0.25, 0.9, 0.5)[0] == 0  # equality: acceptable
    # V2: p(v) < max p - alpha
    assert orc.token_r(V2, 0.1, 0.9, 0.39, 0.5)[0] == 1
    assert orc.token_r(V2, 0.25, 0.0, 0.25, 0.5)[0] == 0
    # V3: p(v) < max p (1 - alpha)
    assert orc.token_r(V3, 0.5, 0.0, 0.24, 0.5)[0] == 1
    assert orc.token_r(V3, 0.5, 0.0, 0.25, 0.5)[0] == 0
    # margins: |0.3 - 0.4| / max(0.3, 0.4, max p = 0.5) for V1 (the threshold
    # max p - alpha carries the rounding of max p), |0.2 - 0.3| / 0.3 for V3
    assert orc.token_r(V1, 0.1, 0.3, 0.0, 0.5)[1] == pytest.approx(0.2)
    assert orc.token_r(V3, 0.4, 0.0, 0.2, 0.5)[1] == pytest.approx(1.0 / 3.0)
    # a token attaining max p: max p < max p - alpha  <=>  alpha < 0, exactly
    for rule in (V2, V3):
        assert orc.token_r(rule, 0.0, 0.9, 0.5, 0.5) == (0, np.inf)
        assert orc.token_r(rule, -1e-30, 0.9, 0.5, 0.5) == (1, np.inf)
        assert orc.token_r(rule, 1e-30, 0.9, 0.5, 0.5) == (0, np.inf)
    # V1 has no such tie: q(v) = max p at alpha = 0 is a plain equality
    assert orc.token_r(V1, 0.0, 0.5, 0.1, 0.5) == (0, 0.0)


@pytest.mark.parametrize("rule", [V2, V3])
def test_token_all_deferred_is_speculative_decoding(orc, rule):
    """alpha < 0 makes r(v) = 1 for every v under V2 and V3: eta = 1 and pi = p,
    so Alg. 4 with the token target is standard speculative sampling."""
    qz, pz, draft, u = _random_step(120 + rule, 200, 4, 50)
    ref_acc, ref_tok = _textbook_specdecode(qz, pz, draft, u, 1.0)
    out = orc.verify(qz, pz, draft, u, rule, -0.5, 1.0)
    np.testing.assert_allclose(out["row_stats"][..., 6], 1.0, atol=1e-12)  # eta
    ok = (out["accept_len"] == ref_acc) & (out["next_token"] == ref_tok)
    for b in np.flatnonzero(~ok):
        m = min(out["accept_margin"][b].min(), out["sample_margin"][b])
        assert m < 1e-9, b
    assert ok.mean() > 0.99


@pytest.mark.parametrize("rule", [V1, V2])
def test_token_none_deferred_samples_drafter(orc, rule):
    """alpha >= 1 makes r(v) = 0 for every v under V1 and V2 (max p - alpha <= 0):
    pi = q, every draft is kept and the extra token comes from q_gamma."""
    qz, pz, draft, u = _random_step(130 + rule, 100, 3, 40)
    out = orc.verify(qz, pz, draft, u, rule, 1.0, 1.0)
    assert (out["accept_len"] == 3).all()
    assert (out["defer"] == 0).all()
    for b in range(100):
        cdf = np.cumsum(_softmax64(qz[b, 3]))
        assert out["next_token"][b] == np.searchsorted(cdf / cdf[-1], np.float64(u[b, 3]),
                                                       side="right")


@pytest.mark.parametrize("rule,alpha,T,seed", [
    (V1, 0.1, 1.0, 140), (V2, 0.05, 1.0, 141), (V3, 0.3, 1.0, 142), (V3, 0.6, 0.7, 143)])
def test_token_emitted_token_law_is_target(orc, rule, alpha, T, seed):
    """The first emitted token is distributed as pi_Token (Alg. 4 with the
    target of Alg. 6), the extra token as pi_{t+gamma}; the rejection
    probability of a draft x ~ q is D_TV(pi, q) = sum max(0, q - pi)."""
    r = _rng(seed)
    V = 6
    pz = r.normal(0, 1.5, (1, 2, V))
    qz = r.normal(0, 1.5, (1, 2, V))
    law, bonus, _ = _first_token_law(orc, qz, pz, rule, alpha, T)
    q0, p0 = _softmax64(qz[0, 0], T), _softmax64(pz[0, 0], T)
    q1, p1 = _softmax64(qz[0, 1], T), _softmax64(pz[0, 1], T)
    r0, r1 = _r_independent(rule, alpha, q0, p0), _r_independent(rule, alpha, q1, p1)
    pi0 = q0 * (1 - r0) + p0 * (r0 * q0).sum()
    pi1 = q1 * (1 - r1) + p1 * (r1 * q1).sum()
    N = 1 << 14
    np.testing.assert_allclose(law, pi0, atol=3.0 / N)
    np.testing.assert_allclose(bonus, pi1, atol=2.0 / N)
    # rejection probability of a q-distributed draft
    acc = np.minimum(1.0, pi0 / q0)
    assert float((q0 * (1 - acc)).sum()) == pytest.approx(np.maximum(0, q0 - pi0).sum(),
                                                          abs=1e-14)


def test_token_greedy_v1_equals_diff(orc):
    """At temperature 0 the drafter's argmax carries q = max q, so TokenV1's
    verdict there, max q < max p - alpha, is the Diff rule."""
    r = _rng(150)
    B, gamma, V = 400, 4, 12
    pz = r.normal(0, 1, (B, gamma + 1, V))
    qz = pz + r.normal(0, 0.8, (B, gamma + 1, V))
    draft = np.argmax(qz[:, :gamma], -1).astype(np.int32)
    for alpha in (0.0, 0.05, 0.3):
        a = orc.greedy_verify(qz, pz, draft, V1, alpha)
        b = orc.greedy_verify(qz, pz, draft, DIFF, alpha)
        np.testing.assert_array_equal(a["accept_len"], b["accept_len"])
        np.testing.assert_array_equal(a["next_token"], b["next_token"])
        np.testing.assert_array_equal(a["defer"], b["defer"])


def test_token_greedy_hand_case(orc):
    """Two positions (gamma = 1), V = 3, T = 1 probabilities for the rule.
    Position 0: argmax q = 0, argmax p = 2; p(0) is small, so V2 and V3 reject
    the drafter's token and the one-hot target moves to argmax p."""
    qz = np.array([[[2.0, 0.0, 1.0], [0.0, 2.0, 0.0]]])
    pz = np.array([[[-2.0, 0.0, 3.0], [0.0, 3.0, 0.0]]])
    draft = np.array([[0]], np.int32)
    for rule in (V2, V3):
        out = orc.greedy_verify(qz, pz, draft, rule, 0.1)
        assert out["defer"][0, 0] == 1
        assert out["accept_len"][0] == 0 and out["next_token"][0] == 2
    # V1 at alpha = 0.9: max q < max p - 0.9 fails, so the draft is kept; at
    # the bonus position argmax q = argmax p = 1
    out = orc.greedy_verify(qz, pz, draft, V1, 0.9)
    assert out["accept_len"][0] == 1 and out["next_token"][0] == 1
