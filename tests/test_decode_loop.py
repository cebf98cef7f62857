"""The decoding loop (GenSpecSample, Alg. 4, round after round) on the CPU with
the oracle backend: its bookkeeping against results with closed forms.

- Greedy speculative decoding with delta = 1 is greedy decoding of the
  verifier, so the loop must reproduce the verifier's own argmax chain.
- With drafter = verifier and delta = 1 every draft is kept, and the emitted
  tokens are plain auto-regressive sampling from p with the same uniforms
  (drafts from the drafting uniforms, the extra token from u[gamma]).
- With delta = 0 the target is q: every draft is kept and the extra token
  is drawn from q at position gamma.
"""
import numpy as np
import pytest
import torch

import oracle
from decode_oracle import OracleBackend, _host
from paper_2405_19261_amd import decode
from paper_2405_19261_amd import workloads as W

V, B, GAMMA = 300, 6, 4


def _models(seed=0, same=False):
    p = decode.SyntheticLM(V, rows=16, seed=seed, dtype=torch.float32, device="cpu")
    q = p if same else p.derive(scale=0.8, sigma=1.0, seed=seed + 1)
    return q, p


def _first(seed=3):
    return torch.randint(0, V, (B,), generator=torch.Generator().manual_seed(seed))


def test_greedy_always_is_greedy_decoding_of_p():
    q, p = _models()
    res = decode.spec_decode(q, p, _first(), rounds=6, gamma=GAMMA, rule=W.ALWAYS, alpha=0.0,
                             temperature=0.0, backend=OracleBackend())
    for b in range(B):
        last, pos, chain = int(_first()[b]), 0, []
        for _ in range(len(res.tokens[b])):
            z = p(torch.tensor([last]), torch.tensor([pos]))[0].numpy()
            last = int(np.argmax(z))
            chain.append(last)
            pos += 1
        assert res.tokens[b] == chain


def test_identical_models_always_is_autoregressive_sampling():
    q, p = _models(same=True)
    inputs = []
    res = decode.spec_decode(q, p, _first(), rounds=3, gamma=GAMMA, rule=W.ALWAYS, alpha=0.0,
                             temperature=1.0, backend=OracleBackend(), rounds_inputs=inputs)
    assert all(bool((a == GAMMA).all()) for a in res.accept_len)
    for b in range(B):
        last, pos, expect = int(_first()[b]), 0, []
        for rnd in inputs:
            for j in range(GAMMA + 1):
                u = rnd["u_draft"][j, b] if j < GAMMA else rnd["uniforms"][b, GAMMA]
                z = p(torch.tensor([last]), torch.tensor([pos]))
                tok, _ = oracle.draft_sample(_host(z), 1.0, np.array([float(u)], np.float32))
                last = int(tok[0])
                expect.append(last)
                pos += 1
        assert res.tokens[b] == expect


def test_never_defer_keeps_every_draft_and_samples_q_last():
    q, p = _models(seed=5)
    inputs = []
    res = decode.spec_decode(q, p, _first(7), rounds=3, gamma=GAMMA, rule=W.NEVER, alpha=0.0,
                             temperature=1.0, backend=OracleBackend(), rounds_inputs=inputs)
    assert all(bool((a == GAMMA).all()) for a in res.accept_len)
    k = 0
    for rnd in inputs:
        for b in range(B):
            got = res.tokens[b][k:k + GAMMA + 1]
            assert got[:GAMMA] == [int(t) for t in rnd["draft"][b]]
            zq = rnd["q"][b, GAMMA][None].contiguous()
            tok, _ = oracle.draft_sample(_host(zq), 1.0,
                                         np.array([float(rnd["uniforms"][b, GAMMA])], np.float32))
            assert got[GAMMA] == int(tok[0])
        k += GAMMA + 1


@pytest.mark.parametrize("rule,alpha", [(W.DIFF, 0.05), (W.OPT, 0.1), (W.TOKEN_V3, 0.3),
                                        (W.CHOWLOG, 4.0), (W.LOSSY, 0.3)])
def test_emitted_count_matches_accept_lengths(rule, alpha):
    q, p = _models(seed=11)
    res = decode.spec_decode(q, p, _first(2), rounds=4, gamma=GAMMA, rule=rule, alpha=alpha,
                             temperature=torch.tensor([1.0, 0.7, 0.0, 1.0, 0.5, 0.0]),
                             backend=OracleBackend())
    for b in range(B):
        assert len(res.tokens[b]) == sum(int(a[b]) + 1 for a in res.accept_len)
        assert all(0 <= t < V for t in res.tokens[b])
    assert 1.0 <= res.tokens_per_round() <= GAMMA + 1
