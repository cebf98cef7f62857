"""Pins of the oracle's drafter sampling step (Alg. 4: x_{t+j} ~ q_{t+j}).

The token is the inverse CDF of softmax(z / T) at the row's uniform (the
smallest k whose cumulative mass exceeds u, in vocabulary order), or the
argmax of the raw logits at T = 0.  Checked against scipy's softmax with
numpy's searchsorted (library pins), the exact law of the token over a fine
grid of uniforms (it must be softmax(z / T) itself), numpy's argmax, masked
entries, and the argument checks.
"""
import numpy as np
import pytest
from scipy.special import softmax as scipy_softmax

import oracle


def _rng(seed):
    return np.random.default_rng(seed)


@pytest.mark.parametrize("T", [0.5, 1.0, 2.0])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_matches_library_inverse_cdf(T, dtype):
    rng = _rng(11)
    z = rng.normal(0.0, 2.0, size=(16, 300)).astype(np.float32)
    if dtype == "bf16":  # round to bfloat16; both sides read the stored values
        bits = (z.view(np.uint32) + 0x7FFF + ((z.view(np.uint32) >> 16) & 1)) >> 16
        zb = bits.astype(np.uint16)
        zw = (zb.astype(np.uint32) << 16).view(np.float32)
    else:
        zb = zw = z
    u = rng.random(16).astype(np.float32)
    tok, mg = oracle.draft_sample(zb, T, u)
    for b in range(16):
        p = scipy_softmax(zw[b].astype(np.float64) / T)
        c = np.cumsum(p) / p.sum()
        assert tok[b] == np.searchsorted(c, float(u[b]), side="right")
        assert mg[b] > 0


@pytest.mark.parametrize("T", [0.7, 1.0])
def test_token_law_is_the_softmax(T):
    """Over a fine midpoint grid of uniforms the oracle's token counts are
    softmax(z / T) itself: each token's count is the number of grid points in
    its cumulative-mass interval (scipy), up to one point per edge."""
    z = np.array([0.3, -1.2, 2.0, 0.0, -np.inf, 1.1, 0.5], np.float32)
    n = 100_000
    us = ((np.arange(n) + 0.5) / n).astype(np.float32)
    toks, _ = oracle.draft_sample(np.tile(z, (n, 1)), T, us)
    counts = np.bincount(toks, minlength=z.size)
    c = np.cumsum(scipy_softmax(z.astype(np.float64) / T))
    expect = np.diff(np.concatenate([[0], np.searchsorted(us.astype(np.float64), c,
                                                          side="right")]))
    assert counts[4] == 0  # the masked token
    np.testing.assert_allclose(counts, expect, atol=1)
    np.testing.assert_allclose(counts / n, np.diff(np.concatenate([[0.0], c])), atol=2.0 / n)


def test_masked_entries_never_drawn():
    rng = _rng(5)
    z = rng.normal(size=(64, 50)).astype(np.float32)
    z[:, ::3] = -np.inf
    u = rng.random(64).astype(np.float32)
    tok, _ = oracle.draft_sample(z, 1.0, u)
    assert np.all(tok % 3 != 0)


def test_greedy_is_first_argmax():
    rng = _rng(9)
    z = rng.integers(-3, 4, size=(32, 40)).astype(np.float32)  # many ties
    tok, mg = oracle.draft_sample(z, 0.0)
    np.testing.assert_array_equal(tok, np.argmax(z, axis=1))
    assert np.all(np.isinf(mg))


def test_per_row_temperature_mix():
    rng = _rng(3)
    z = rng.normal(0.0, 1.5, size=(8, 100)).astype(np.float32)
    T = np.array([0.0, 0.5, 1.0, 0.0, 2.0, 0.7, 0.0, 1.0], np.float32)
    u = rng.random(8).astype(np.float32)
    tok, _ = oracle.draft_sample(z, T, u)
    for b in range(8):
        if T[b] == 0:
            assert tok[b] == np.argmax(z[b])
        else:
            c = np.cumsum(scipy_softmax(z[b].astype(np.float64) / T[b]))
            assert tok[b] == np.searchsorted(c / c[-1], float(u[b]), side="right")


def test_argument_errors():
    z = np.zeros((2, 5), np.float32)
    with pytest.raises(ValueError):
        oracle.draft_sample(z, -1.0, np.zeros(2, np.float32))
    with pytest.raises(ValueError):
        oracle.draft_sample(z, 1.0, None)  # sampling needs uniforms
