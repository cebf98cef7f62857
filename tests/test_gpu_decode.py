"""The drafter's sampling step and the decoding loop on the GPU, against the
fp64 oracle (needs an MI355X)."""
import numpy as np
import pytest
import torch

import oracle
import parity
from decode_oracle import OracleBackend, _host
from paper_2405_19261_amd import decode, spc
from paper_2405_19261_amd import workloads as W

pytestmark = pytest.mark.gpu
DEV = "cuda"
NEAR = parity.NEAR


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()


def _check_tokens(gpu_tok, o_tok, o_margin, rep):
    """Tokens must agree wherever the oracle's draw is not a near-tie."""
    for g, o, m in zip(gpu_tok, o_tok, o_margin):
        rep["draws"] += 1
        if g != o:
            assert m < NEAR, f"token gpu={g} oracle={o} margin={m:.3g}"
            rep["excused"] += 1


@pytest.mark.parametrize("cfg", [3, 2])
@pytest.mark.parametrize("T", [1.0, 0.5, 0.0, "mix"])
def test_draft_sample_parity(cfg, T):
    wl = W.WORKLOADS[cfg]
    rep = {"draws": 0, "excused": 0}
    for step in range(4 if cfg == 3 else 20):
        inp = W.generate(wl, 400 + step, DEV)
        z = inp["q"].reshape(-1, wl.V)[: 4 * wl.B].contiguous()  # [n, V] drafter rows
        n = z.shape[0]
        g = torch.Generator(device=DEV).manual_seed(77 + step)
        u = torch.rand(n, generator=g, device=DEV)
        if T == "mix":
            temps = torch.tensor([0.0, 0.5, 0.7, 1.0], device=DEV).repeat(n // 4)
            tok = spc.spc_draft_sample(z, 0.0, uniforms=u, temp_per_seq=temps)
            th = temps.cpu().numpy()
        else:
            tok = spc.spc_draft_sample(z, T, uniforms=u if T > 0 else None)
            th = np.full(n, T, np.float32)
        torch.cuda.synchronize()
        o_tok, o_mg = oracle.draft_sample(_host(z), th, u.cpu().numpy())
        _check_tokens(tok.cpu().numpy(), o_tok, o_mg, rep)
    print(f"[draft] cfg{cfg} T={T} {rep}", flush=True)


@pytest.mark.parametrize("dtype,V", [("bf16", 2), ("bf16", 1001), ("bf16", 16385),
                                     ("f32", 3), ("f32", 999), ("f32", 8193),
                                     ("bf16", 2000000), ("bf16", 1100001)])
def test_draft_sample_ragged_and_masked(dtype, V):
    wl = W.WORKLOADS[3].with_(B=16, V=V, dtype=dtype)
    inp = W.generate(wl, 5, DEV)
    z = inp["q"][:, 0].contiguous()
    g = torch.Generator(device=DEV).manual_seed(5)
    m = torch.rand(z.shape, generator=g, device=DEV) < 0.4
    m[:, 0] = False
    z[m[:, :]] = float("-inf")
    u = torch.rand(16, generator=g, device=DEV)
    for T in (1.0, 0.0):
        tok = spc.spc_draft_sample(z, T, uniforms=u)
        torch.cuda.synchronize()
        o_tok, o_mg = oracle.draft_sample(_host(z), np.full(16, T, np.float32), u.cpu().numpy())
        _check_tokens(tok.cpu().numpy(), o_tok, o_mg, {"draws": 0, "excused": 0})
        assert not m.gather(1, tok.long()[:, None]).any()  # never a masked token


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_draft_sample_maximum_rows(dtype):
    """The drafter at its row limit (32767 rows)."""
    B = 32767
    wl = W.WORKLOADS[3].with_(B=B, gamma=1, V=41, dtype=dtype)
    z = W.generate(wl, 9, DEV)["q"][:, 0].contiguous()
    g = torch.Generator(device=DEV).manual_seed(9)
    u = torch.rand(B, generator=g, device=DEV)
    for T in (1.0, 0.0):
        tok = spc.spc_draft_sample(z, T, uniforms=u)
        torch.cuda.synchronize()
        o_tok, o_mg = oracle.draft_sample(_host(z), np.full(B, T, np.float32), u.cpu().numpy())
        _check_tokens(tok.cpu().numpy(), o_tok, o_mg, {"draws": 0, "excused": 0})


def test_decode_loop_rounds_match_oracle():
    """Every round of the GPU loop, replayed through the oracle on the same
    inputs: the drafts are the oracle's draws from the drafter rows, and the
    verify outputs are the oracle's."""
    q_lm, p_lm = decode.synthetic_pair(V=256000, seed=4, dtype=torch.bfloat16, device=DEV)
    B, gamma = 16, 5
    first = torch.randint(0, 256000, (B,), generator=torch.Generator().manual_seed(1))
    temps = torch.tensor([1.0, 0.7, 0.5, 1.0] * 4)
    rules = torch.tensor([W.DIFF, W.OPT, W.TOKEN_V3, W.CHOW] * 4, dtype=torch.int32)
    alphas = torch.tensor([0.05, 0.1, 0.3, 0.4] * 4)
    inputs = []
    res = decode.spec_decode(q_lm, p_lm, first, rounds=4, gamma=gamma, rule=rules,
                             alpha=alphas, temperature=temps, seed=9, rounds_inputs=inputs)
    rep = {"draws": 0, "excused": 0}
    for rnd in inputs:
        for j in range(gamma):
            o_tok, o_mg = oracle.draft_sample(_host(rnd["q"][:, j].contiguous()),
                                              rnd["temperature"].cpu().numpy(),
                                              rnd["u_draft"][j].cpu().numpy())
            _check_tokens(rnd["draft"][:, j].cpu().numpy(), o_tok, o_mg, rep)
        g = parity.run_gpu(rnd)
        h = parity.host_inputs(rnd)
        parity.compare(g, parity.run_oracle(h), h, "bf16")
    print(f"[decode] rounds {len(inputs)} tokens/round {res.tokens_per_round():.2f} {rep}",
          flush=True)


@pytest.mark.parametrize("mode", ["mixed", "greedy"])
def test_graph_decode_equals_eager(mode):
    """One captured round replayed per round emits exactly the eager loop's
    tokens and accept lengths; every round's output feeds the next replay, and
    eager copies run between the replays."""
    q_lm, p_lm = decode.synthetic_pair(V=256000, seed=4, dtype=torch.bfloat16, device=DEV)
    B, gamma = 16, 5
    first = torch.randint(0, 256000, (B,), generator=torch.Generator().manual_seed(3))
    if mode == "mixed":
        kw = dict(rule=torch.tensor([W.DIFF, W.OPT, W.TOKEN_V3, W.BILD] * 4, dtype=torch.int32),
                  alpha=torch.tensor([0.05, 0.1, 0.3, 2.5] * 4),
                  temperature=torch.tensor([1.0, 0.7, 0.5, 0.0] * 4))
    else:
        kw = dict(rule=W.DIFF, alpha=0.05, temperature=0.0)
    eager = decode.spec_decode(q_lm, p_lm, first, rounds=7, gamma=gamma, seed=21, **kw)
    for _ in range(2):
        torch.cuda.synchronize()
        graphed = decode.spec_decode(q_lm, p_lm, first, rounds=7, gamma=gamma, seed=21,
                                     graph=True, **kw)
        assert graphed.tokens == eager.tokens
        for a, b in zip(graphed.accept_len, eager.accept_len):
            assert torch.equal(a, b)
    print(f"[decode-graph] {mode} tokens/round {eager.tokens_per_round():.2f}", flush=True)


@pytest.mark.parametrize("rule,alpha", [(W.DIFF, 0.05), (W.OPT, 0.1), (W.TOKEN_V1, 0.05),
                                        (W.BILD, 2.5), (W.LOSSY, 0.3)])
def test_greedy_decode_loop_equals_oracle_loop(rule, alpha):
    """Temperature 0 end to end: the GPU loop and the oracle loop emit the same
    tokens round after round."""
    q_lm, p_lm = decode.synthetic_pair(V=50000, seed=6, dtype=torch.bfloat16, device=DEV)
    first = torch.randint(0, 50000, (12,), generator=torch.Generator().manual_seed(2))
    kw = dict(rounds=5, gamma=4, rule=rule, alpha=alpha, temperature=0.0, seed=3)
    a = decode.spec_decode(q_lm, p_lm, first, **kw)
    b = decode.spec_decode(q_lm, p_lm, first, backend=OracleBackend(), **kw)
    assert a.tokens == b.tokens
    for x, y in zip(a.accept_len, b.accept_len):
        np.testing.assert_array_equal(x.numpy(), y.cpu().numpy())


def test_draft_sample_invalid_row_temperatures():
    """A per-row temperature that is negative or not finite gives that row
    token -1; the other rows draw as with valid temperatures alone."""
    wl = W.WORKLOADS[3].with_(B=8, V=30000)
    z = W.generate(wl, 6, DEV)["q"][:, 0].contiguous()
    u = torch.rand(8, generator=torch.Generator(device=DEV).manual_seed(6), device=DEV)
    temps = torch.tensor([1.0, float("nan"), 0.7, -1.0, 0.0, float("inf"), 2.0, 1.0],
                         device=DEV)
    tok = spc.spc_draft_sample(z, 0.0, uniforms=u, temp_per_seq=temps).cpu().numpy()
    bad = [1, 3, 5]
    assert (tok[bad] == -1).all()
    ok = [b for b in range(8) if b not in bad]
    t_ok = temps[ok].cpu().numpy()
    o_tok, o_mg = oracle.draft_sample(_host(z[ok]), t_ok, u[ok].cpu().numpy())
    _check_tokens(tok[ok], o_tok, o_mg, {"draws": 0, "excused": 0})
