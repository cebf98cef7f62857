"""Pins of the fp64 oracle against what the paper and mathematics fix.

None of these compare the oracle with itself: each check uses a library
routine, a closed form worked out by hand, an invariant the paper proves, or
an independently written textbook procedure.
"""
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
RULES = {"chow": 0, "diff": 1, "opt": 2, "always": 3, "never": 4}


def _softmax64(z, T=1.0):
    return torch.softmax(torch.as_tensor(np.asarray(z, np.float64)) / T, dim=-1).numpy()


def _rng(seed):
    return np.random.default_rng(seed)


# ---------------------------------------------------------------- softmax rows

@pytest.mark.parametrize("T", [1.0, 0.5, 0.7, 2.0])
def test_softmax_matches_torch_float64(orc, T):
    """Row statistics vs torch.softmax / logsumexp in float64 (library pin)."""
    z = _rng(1).normal(0, 3, 777)
    prob, m, lse, maxprob, amax = orc.softmax_row(z, T)
    ref = _softmax64(z, T)
    np.testing.assert_allclose(prob, ref, rtol=1e-12, atol=1e-300)
    assert lse == pytest.approx(torch.logsumexp(torch.tensor(z / T), 0).item(), rel=1e-13)
    assert m == pytest.approx(z.max() / T, rel=1e-15)
    assert maxprob == pytest.approx(ref.max(), rel=1e-12)
    # maxprob = exp(m - lse) = 1 / Z
    assert maxprob == pytest.approx(math.exp(m - lse), rel=1e-12)
    assert amax == int(np.argmax(z))


def test_softmax_widening_f32_bf16(orc):
    """float32 and bfloat16 inputs widen exactly: same stats as the f64 copy."""
    z32 = _rng(2).normal(0, 2, 513).astype(np.float32)
    bf = torch.from_numpy(z32).to(torch.bfloat16)
    z_bf_bits = bf.view(torch.int16).numpy().view(np.uint16)
    z_bf_64 = bf.to(torch.float64).numpy()
    for raw, wide in ((z32, z32.astype(np.float64)), (z_bf_bits, z_bf_64)):
        a = orc.softmax_row(raw, 0.7)
        b = orc.softmax_row(wide, 0.7)
        np.testing.assert_array_equal(a[0], b[0])
        assert a[1:] == b[1:]


def test_argmax_ties_lowest_index(orc):
    z = np.array([1.0, 3.0, -2.0, 3.0, 3.0])
    assert orc.softmax_row(z, 1.0)[4] == 1
    z = np.full(9, -1.5)
    assert orc.softmax_row(z, 0.5)[4] == 0


def test_masked_logits(orc):
    """-inf logits get zero probability and never win the argmax."""
    z = np.array([-np.inf, 0.0, np.log(3.0), -np.inf])
    prob, m, lse, maxprob, amax = orc.softmax_row(z, 1.0)
    np.testing.assert_allclose(prob, [0, 0.25, 0.75, 0], rtol=1e-15)
    assert amax == 2


# ---------------------------------------------------------------------- TV

def test_tv_three_forms_and_range(orc):
    """Lemma 3: D_TV = sum max(0, p - q) = 1/2 sum |p - q| = 1 - sum min(p, q)."""
    r = _rng(3)
    for V in (2, 7, 1000):
        for _ in range(5):
            p = _softmax64(r.normal(0, 2, V))
            q = _softmax64(r.normal(0, 2, V))
            tv = orc.tv(p, q)
            assert tv == pytest.approx(0.5 * np.abs(p - q).sum(), abs=1e-13)
            assert tv == pytest.approx(1.0 - np.minimum(p, q).sum(), abs=1e-13)
            assert 0.0 <= tv <= 1.0
            assert tv == pytest.approx(orc.tv(q, p), abs=1e-13)  # symmetric
    p = _softmax64(r.normal(0, 1, 50))
    assert orc.tv(p, p) == 0.0
    a = np.array([0.5, 0.5, 0, 0])
    b = np.array([0, 0, 0.25, 0.75])
    assert orc.tv(a, b) == 1.0  # disjoint supports


# ------------------------------------------------------------ deferral rules

def _tok(s):
    return math.log(float(s[2:])) if s.startswith("ln") else float(s)


def _golden_defer_cases():
    rows = []
    with open(os.path.join(HERE, "golden", "defer_cases.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            head, qz, pz, vals, dl = [c.strip() for c in line.split("|")]
            rule, alpha, T = head.split()
            rows.append(dict(rule=rule, alpha=float(alpha), T=float(T),
                             qz=[_tok(t) for t in qz.split()], pz=[_tok(t) for t in pz.split()],
                             vals=[float(Fraction(v)) for v in vals.split()], delta=int(dl)))
    assert len(rows) >= 15
    return rows


@pytest.mark.parametrize("case", _golden_defer_cases(), ids=lambda c: f"{c['rule']}-{c['alpha']}")
def test_defer_hand_cases(orc, case):
    """Table 1 rules on hand-derived closed forms (tests/golden/defer_cases.txt)."""
    q, _, _, maxq, _ = orc.softmax_row(np.array(case["qz"]), case["T"])
    p, _, _, maxp, _ = orc.softmax_row(np.array(case["pz"]), case["T"])
    tv = orc.tv(p, q)
    emq, emp, etv = case["vals"]
    assert maxq == pytest.approx(emq, abs=1e-14)
    assert maxp == pytest.approx(emp, abs=1e-14)
    assert tv == pytest.approx(etv, abs=1e-14)
    d, mg = orc.defer(RULES[case["rule"]], case["alpha"], maxq, maxp, tv)
    assert d == case["delta"]
    # OPT on identical rows is an exact tie (maxq < maxp - alpha * 0), which the
    # strict inequality resolves to "keep"; every other case is far from a tie
    assert mg > 1e-4 or (case["rule"] == "opt" and etv == 0.0)


def test_defer_constant_rules_and_strictness(orc):
    assert orc.defer(RULES["always"], 0.3, 0.9, 0.1, 0.5)[0] == 1
    assert orc.defer(RULES["never"], 0.3, 0.1, 0.9, 0.5)[0] == 0
    # a tie does not defer (strict '<')
    assert orc.defer(RULES["chow"], 0.5, 0.5, 0.0, 0.0)[0] == 0
    assert orc.defer(RULES["diff"], 0.25, 0.5, 0.75, 0.0)[0] == 0
    assert orc.defer(RULES["opt"], 0.5, 0.5, 0.75, 0.5)[0] == 0
    assert orc.defer(99, 0.1, 0.5, 0.5, 0.0)[0] == -1


# ------------------------------------------------- target, accept, residual

def test_target_mixture(orc):
    r = _rng(4)
    q = _softmax64(r.normal(size=11))
    p = _softmax64(r.normal(size=11))
    np.testing.assert_array_equal(orc.target(0, q, p), q)
    np.testing.assert_array_equal(orc.target(1, q, p), p)


def test_accept_threshold(orc):
    """u < min(1, pi/q): pi = 0.3, q = 0.6 gives ratio 1/2; strict."""
    assert orc.accept(0.3, 0.6, 0.49)[0] == 1
    assert orc.accept(0.3, 0.6, 0.5)[0] == 0
    assert orc.accept(0.3, 0.6, 0.51)[0] == 0
    assert orc.accept(0.7, 0.6, 0.999999)[0] == 1   # pi >= q is always kept
    assert orc.accept(0.0, 0.6, 0.0)[0] == 0        # pi(x) = 0 is always rejected
    assert orc.accept(0.2, 0.0, 0.5)[0] == 1        # q(x) = 0 <= pi(x)
    a, mg = orc.accept(0.3, 0.6, 0.45)
    assert mg == pytest.approx(0.05, abs=1e-15)


def test_residual_is_distribution(orc):
    """P7: max(0, pi - q) is non-negative, zero where pi <= q, and W = D_TV."""
    r = _rng(5)
    for _ in range(10):
        q = _softmax64(r.normal(0, 2, 300))
        p = _softmax64(r.normal(0, 2, 300))
        w, W = orc.residual(p, q)
        assert (w >= 0).all()
        assert (w[p <= q] == 0).all()
        assert W == pytest.approx(w.sum(), rel=1e-15)
        assert W == pytest.approx(orc.tv(p, q), rel=1e-13)
        assert (w / W).sum() == pytest.approx(1.0, abs=1e-12)


def test_sample_inverse_cdf_vs_searchsorted(orc):
    """The smallest k with C_k / W > u == numpy searchsorted(side='right')."""
    r = _rng(6)
    for _ in range(20):
        w = r.random(64) * (r.random(64) < 0.6)
        cdf = np.cumsum(w) / w.sum()
        for u in r.random(50):
            k, mg = orc.sample(w, u)
            assert k == int(np.searchsorted(cdf, u, side="right"))
            assert w[k] > 0  # zero-mass tokens are never drawn
    # dyadic masses: C = (1/8, 3/8, 3/4, 1) exactly; a boundary u goes right
    w = np.array([0.125, 0.25, 0.375, 0.25])
    assert [orc.sample(w, u)[0] for u in (0.0, 0.124, 0.125, 0.374, 0.375, 0.749, 0.75, 0.9999)] \
        == [0, 0, 1, 1, 2, 2, 3, 3]
    assert orc.sample(np.array([0.0, 0.5, 0.0, 0.5, 0.0]), 0.5)[0] == 3
    assert orc.sample(np.zeros(5), 0.5)[0] == -1


# ----------------------------------------------------- full verify step pins

def _textbook_specdecode(qz, pz, draft, u, T):
    """Standard speculative sampling (Leviathan et al.), written independently:
    keep x_j with probability min(1, p(x)/q(x)); at the first rejection draw from
    norm(max(0, p - q)); if every draft is kept, draw the extra token from p."""
    B, G, V = qz.shape
    gamma = G - 1
    acc = np.empty(B, np.int32)
    tok = np.empty(B, np.int32)
    for b in range(B):
        qs = _softmax64(qz[b], T)
        ps = _softmax64(pz[b], T)
        n = gamma
        for j in range(gamma):
            x = draft[b, j]
            if not (u[b, j] < min(1.0, ps[j, x] / qs[j, x])):
                n = j
                break
        dist = np.maximum(0.0, ps[n] - qs[n]) if n < gamma else ps[gamma]
        cdf = np.cumsum(dist) / dist.sum()
        acc[b] = n
        tok[b] = np.searchsorted(cdf, np.float64(u[b, gamma]), side="right")
    return acc, tok


def _random_step(seed, B, gamma, V, T=1.0, noise=0.7):
    r = _rng(seed)
    pz = r.normal(0, 2, (B, gamma + 1, V))
    qz = pz + r.normal(0, noise, (B, gamma + 1, V))
    draft = np.empty((B, gamma), np.int32)
    for b in range(B):
        for j in range(gamma):
            draft[b, j] = r.choice(V, p=_softmax64(qz[b, j], T))
    u = r.random((B, gamma + 1)).astype(np.float32)
    return qz, pz, draft, u


@pytest.mark.parametrize("T", [1.0, 0.5])
def test_delta_one_is_speculative_decoding(orc, T):
    """P1: with delta == 1 (rule ALWAYS, or Chow with alpha < 0) Alg. 4 is Alg. 1."""
    qz, pz, draft, u = _random_step(7, 200, 4, 50, T)
    ref_acc, ref_tok = _textbook_specdecode(qz, pz, draft, u, T)
    for rule, alpha in ((RULES["always"], 0.0), (RULES["chow"], -0.5)):
        out = orc.verify(qz, pz, draft, u, rule, alpha, T)
        assert (out["defer"] == 1).all()
        ok = (out["accept_len"] == ref_acc) & (out["next_token"] == ref_tok)
        # a disagreement may only sit on a decision tied to ~1e-12
        for b in np.flatnonzero(~ok):
            m = min(out["accept_margin"][b].min(), out["sample_margin"][b])
            assert m < 1e-9, b
        assert ok.mean() > 0.99


def test_delta_zero_samples_drafter(orc):
    """delta == 0: pi = q, every draft is kept, the extra token comes from q_gamma."""
    qz, pz, draft, u = _random_step(8, 100, 3, 40)
    out = orc.verify(qz, pz, draft, u, RULES["never"], 0.0, 1.0)
    assert (out["accept_len"] == 3).all()
    for b in range(100):
        cdf = np.cumsum(_softmax64(qz[b, 3]))
        assert out["next_token"][b] == np.searchsorted(cdf / cdf[-1], np.float64(u[b, 3]),
                                                       side="right")


def test_identical_models_accept_everything(orc):
    """P5: p = q gives pi = q, D_TV = 0 and no rejection, for every rule."""
    qz, _, draft, u = _random_step(9, 40, 5, 64)
    for rule, alpha in ((0, 0.5), (1, 0.0), (1, 0.2), (2, 0.1), (3, 0.0)):
        out = orc.verify(qz, qz.copy(), draft, u, rule, alpha, 1.0)
        assert (out["accept_len"] == 5).all()
        assert (out["row_stats"][..., 6] == 0.0).all()
        if rule in (1, 2):
            assert (out["defer"] == 0).all()


def test_output_ranges(orc):
    """P3: at least one and at most gamma+1 tokens per call."""
    qz, pz, draft, u = _random_step(10, 300, 6, 30, noise=2.0)
    for rule in range(5):
        out = orc.verify(qz, pz, draft, u, rule, 0.1, 1.0)
        assert ((out["accept_len"] >= 0) & (out["accept_len"] <= 6)).all()
        assert ((out["next_token"] >= 0) & (out["next_token"] < 30)).all()
        assert (out["flags"] == 0).all()


def test_draft_out_of_range_is_rejected(orc):
    qz, pz, draft, u = _random_step(11, 4, 3, 16)
    draft[:, 1] = [-1, 16, 1 << 30, -(1 << 30)]
    u[:, 0] = 0.0  # position 0 kept whenever pi(x) > 0
    out = orc.verify(qz, pz, draft, u, RULES["always"], 0.0, 1.0)
    assert (out["accept_len"] <= 1).all()
    assert (out["flags"] & orc.FLAG_DRAFT_OUT_OF_RANGE).all()


def _first_token_law(orc, qz, pz, rule, alpha, T, N=1 << 14):
    """Law of the first emitted token for gamma = 1 by exhaustive grids:
    draft x over V weighted by q(x), accept uniform over an N-point midpoint grid,
    sample uniform over another; error <= 1/N per threshold."""
    V = qz.shape[-1]
    q0 = _softmax64(qz[0, 0], T)
    grid = ((np.arange(N) + 0.5) / N).astype(np.float32)
    law = np.zeros(V)
    # acceptance fraction per draft token
    acc = np.zeros(V)
    for x in range(V):
        B = N
        out = orc.verify(np.repeat(qz, B, 0), np.repeat(pz, B, 0), np.full((B, 1), x, np.int32),
                         np.stack([grid, np.zeros(B, np.float32)], 1), rule, alpha, T)
        acc[x] = (out["accept_len"] == 1).mean()
    # residual law: reject a draft that can be rejected, sweep the sample uniform
    res = np.zeros(V)
    rejectable = [x for x in range(V) if acc[x] < 1.0]
    if rejectable:
        x = rejectable[0]
        out = orc.verify(np.repeat(qz, N, 0), np.repeat(pz, N, 0), np.full((N, 1), x, np.int32),
                         np.stack([np.full(N, np.float32(1.0 - 2 ** -24)), grid], 1), rule,
                         alpha, T)
        assert (out["accept_len"] == 0).all()
        res = np.bincount(out["next_token"], minlength=V) / N
    for x in range(V):
        law[x] += q0[x] * acc[x]
        law += q0[x] * (1.0 - acc[x]) * res
    # the extra token after an acceptance
    out = orc.verify(np.repeat(qz, N, 0), np.repeat(pz, N, 0),
                     np.full((N, 1), int(np.argmax(q0)), np.int32),
                     np.stack([np.zeros(N, np.float32), grid], 1), rule, alpha, T)
    bonus = np.bincount(out["next_token"][out["accept_len"] == 1], minlength=V)
    bonus = bonus / max(1, bonus.sum())
    return law, bonus, out["defer"][0]


@pytest.mark.parametrize("rule,alpha,T,seed", [
    (RULES["chow"], 0.6, 1.0, 20), (RULES["diff"], 0.0, 1.0, 21), (RULES["opt"], 0.05, 0.5, 22),
    (RULES["always"], 0.0, 1.0, 23), (RULES["diff"], 0.3, 0.7, 24)])
def test_emitted_token_law_is_target(orc, rule, alpha, T, seed):
    """P2: the first emitted token is distributed as pi_t (Alg. 4 samples pi),
    and the extra token after a full acceptance as pi_{t+gamma}."""
    r = _rng(seed)
    V = 6
    pz = r.normal(0, 1.5, (1, 2, V))
    qz = r.normal(0, 1.5, (1, 2, V))
    law, bonus, defer = _first_token_law(orc, qz, pz, rule, alpha, T)
    pi0 = (1 - defer[0]) * _softmax64(qz[0, 0], T) + defer[0] * _softmax64(pz[0, 0], T)
    pi1 = (1 - defer[1]) * _softmax64(qz[0, 1], T) + defer[1] * _softmax64(pz[0, 1], T)
    N = 1 << 14
    np.testing.assert_allclose(law, pi0, atol=3.0 / N)
    np.testing.assert_allclose(bonus, pi1, atol=2.0 / N)


def test_rejection_probability_is_delta_tv(orc):
    """P4, Lemma 3: sum_x q(x) (1 - min(1, pi(x)/q(x))) = delta * D_TV(p, q)."""
    r = _rng(30)
    for rule, alpha in ((0, 0.4), (1, 0.05), (2, 0.1), (3, 0.0), (4, 0.0)):
        for _ in range(5):
            V = 200
            qz = r.normal(0, 2, (1, 2, V))
            pz = r.normal(0, 2, (1, 2, V))
            out = orc.verify(qz, pz, np.zeros((1, 1), np.int32),
                             np.zeros((1, 2), np.float32), rule, alpha, 1.0)
            d = int(out["defer"][0, 0])
            q = _softmax64(qz[0, 0])
            p = _softmax64(pz[0, 0])
            pi = orc.target(d, q, p)
            rej = float(np.sum(q * (1.0 - np.minimum(1.0, pi / q))))
            assert rej == pytest.approx(d * orc.tv(p, q), abs=1e-12)
            assert out["row_stats"][0, 0, 6] == pytest.approx(0.5 * np.abs(p - q).sum(), abs=1e-13)


def test_expected_accept_length(orc):
    """P9: E[j*] = sum_{k=1..gamma} prod_{j<k} min(1, pi_j(x_j)/q_j(x_j))."""
    qz, pz, draft, _ = _random_step(31, 1, 5, 20, noise=1.0)
    N = 40000
    u = _rng(32).random((N, 6)).astype(np.float32)
    for rule, alpha in ((1, 0.02), (3, 0.0), (0, 0.3)):
        out = orc.verify(np.repeat(qz, N, 0), np.repeat(pz, N, 0), np.repeat(draft, N, 0), u,
                         rule, alpha, 1.0)
        ratios = []
        for j in range(5):
            q = _softmax64(qz[0, j])
            p = _softmax64(pz[0, j])
            d = out["defer"][0, j]
            pi = (1 - d) * q + d * p
            ratios.append(min(1.0, pi[draft[0, j]] / q[draft[0, j]]))
        expect = sum(np.prod(ratios[:k]) for k in range(1, 6))
        mean = out["accept_len"].mean()
        sd = out["accept_len"].std() / math.sqrt(N)
        assert abs(mean - expect) < 5 * sd + 1e-9, (rule, mean, expect)


# -------------------------------------------------------------- greedy pins

def test_greedy_opt_equals_diff(orc):
    """P6, Lemma 6: at temperature 0, OPT and Diff emit the same tokens."""
    r = _rng(40)
    B, gamma, V = 500, 4, 12
    pz = r.normal(0, 1, (B, gamma + 1, V))
    qz = pz + r.normal(0, 0.8, (B, gamma + 1, V))
    draft = np.argmax(qz[:, :gamma], -1).astype(np.int32)
    means = []
    for alpha in (0.0, 0.05, 0.2, 0.6):
        a = orc.greedy_verify(qz, pz, draft, RULES["opt"], alpha)
        b = orc.greedy_verify(qz, pz, draft, RULES["diff"], alpha)
        np.testing.assert_array_equal(a["accept_len"], b["accept_len"])
        np.testing.assert_array_equal(a["next_token"], b["next_token"])
        means.append(a["accept_len"].mean())
    assert 0 < means[0] < gamma  # the case exercises rejections


def test_greedy_hand_cases(orc):
    """One-hot algebra on two positions (gamma = 1), V = 3.
    Position 0: q = softmax(0, ln3, 0) (argmax 1, maxq 3/5),
                p = softmax(ln8, 0, 0) (argmax 0, maxp 8/10).
    Diff alpha=0.1: 3/5 < 7/10 defers, pi~ = one-hot(0); the draft 1 is
    rejected and token 0 is emitted.  Diff alpha=0.3: 3/5 < 1/2 is false,
    the draft is kept and position 1 emits argmax q_1 = 2."""
    l3, l8 = math.log(3), math.log(8)
    qz = np.array([[[0, l3, 0], [0, 0, l3]]])
    pz = np.array([[[l8, 0, 0], [0, l8, 0]]])
    draft = np.array([[1]], np.int32)
    out = orc.greedy_verify(qz, pz, draft, RULES["diff"], 0.1)
    assert out["accept_len"][0] == 0 and out["next_token"][0] == 0
    assert out["row_stats"][0, 0, 2] == pytest.approx(0.6, abs=1e-15)
    assert out["row_stats"][0, 0, 5] == pytest.approx(0.8, abs=1e-15)
    assert out["row_stats"][0, 0, 6] == 1.0
    out = orc.greedy_verify(qz, pz, draft, RULES["diff"], 0.3)
    assert out["accept_len"][0] == 1 and out["next_token"][0] == 2
    # position 1 with Diff alpha=0.1: 3/5 < 7/10 defers, bonus = argmax p_1 = 1
    out = orc.greedy_verify(qz, pz, draft, RULES["always"], 0.0)
    assert out["accept_len"][0] == 0 and out["next_token"][0] == 0
    out = orc.greedy_verify(qz, pz, np.array([[0]], np.int32), RULES["always"], 0.0)
    assert out["accept_len"][0] == 1 and out["next_token"][0] == 1
    np.testing.assert_array_equal(out["argmax"][0], [[1, 0], [2, 1]])


def test_greedy_identical_models(orc):
    r = _rng(41)
    qz = r.normal(0, 1, (50, 4, 30))
    draft = np.argmax(qz[:, :3], -1).astype(np.int32)
    for rule in range(5):
        out = orc.greedy_verify(qz, qz.copy(), draft, rule, 0.1)
        assert (out["accept_len"] == 3).all()
        np.testing.assert_array_equal(out["next_token"], np.argmax(qz[:, 3], -1))


def test_argument_errors(orc):
    qz, pz, draft, u = _random_step(50, 2, 2, 8)
    with pytest.raises(ValueError):
        orc.verify(qz, pz, draft, u, 13, 0.1, 1.0)
    with pytest.raises(ValueError):  # the lossy target needs alpha < 1
        orc.verify(qz, pz, draft, u, 8, 1.0, 1.0)
    with pytest.raises(ValueError):
        orc.verify(qz, pz, draft, u, 1, 0.1, 0.0)
