"""Speculative-cascade decoding: GenSpecSample (Alg. 4) run round after round.

Each round, for every sequence b of the batch:

  1. drafts gamma tokens auto-regressively from the drafter,
     x_{t+j} ~ q(.|x_{<t+j}), j = 0..gamma-1 (``spc_draft_sample``), and takes
     the drafter's logits at the extra position t+gamma as well (the target
     at that position needs q_{t+gamma});
  2. scores the gamma+1 prefixes x_{<t}, ..., x_{<t+gamma} with the verifier
     in one batch;
  3. verifies the block (``spc_verify`` with the chosen target): the first
     rejection j*, and the token that replaces it (or the extra token when
     every draft is kept);
  4. emits x_t .. x_{t+j*-1} and the new token, and rolls back to t+j*+1:
     the drafts past j* are discarded, and the next round starts from the
     emitted token.

Models are callables ``logits_for(last_tokens, positions) -> [n, V]``: the
next-token logits given the last token and its position.  A real language
model conditions on the whole prefix through its KV cache; rolling back is
then truncating that cache to t + j* + 1.  ``SyntheticLM`` is such a callable
with seeded logits, standing in for the paper's drafter/verifier pairs,
whose weights are not used here.

The backend does the sampling and verification.  ``GpuBackend`` calls the C
library; a test may pass any object with the same two methods.
"""
from dataclasses import dataclass, field

import torch

from . import spc


class SyntheticLM:
    """Seeded next-token logits that depend on (last token, position):
    ``rows`` logit rows, each a Zipf(s) ranking over a per-row random
    permutation of the vocabulary plus N(0, noise^2), and the row for a
    context chosen by a hash of (token, position).  ``derive`` makes a model
    whose rows are ``scale`` times this model's rows plus fresh N(0, sigma^2)
    noise, i.e. a drafter that mostly agrees with its verifier."""

    def __init__(self, V, rows=64, s=1.2, noise=1.0, seed=0, dtype=torch.bfloat16,
                 device="cuda", table=None):
        self.V, self.rows, self.dtype, self.device = V, rows, dtype, torch.device(device)
        if table is None:
            g = torch.Generator(device="cpu").manual_seed(seed)
            rank = torch.argsort(torch.rand(rows, V, generator=g), dim=1).float() + 1.0
            table = -s * torch.log(rank) + noise * torch.randn(rows, V, generator=g)
        self.table = table.to(self.device, torch.float32)
        self.logits_table = self.table.to(dtype).contiguous()

    def derive(self, scale=0.8, sigma=1.0, seed=1):
        g = torch.Generator(device="cpu").manual_seed(seed)
        t = scale * self.table.cpu() + sigma * torch.randn(self.rows, self.V, generator=g)
        return SyntheticLM(self.V, self.rows, dtype=self.dtype, device=self.device, table=t)

    def __call__(self, last_tokens, positions):
        h = (last_tokens.long() * 1000003 + positions.long() * 7919) % self.rows
        return self.logits_table.index_select(0, h.to(self.device))


class GpuBackend:
    """Sampling and verification through libspeccascade."""

    def draft_sample(self, logits, temperature, uniforms):
        return spc.spc_draft_sample(logits, 0.0, uniforms=uniforms, temp_per_seq=temperature)

    def verify(self, q, p, drafts, uniforms, rule, alpha, temperature):
        acc, tok, _ = spc.spc_verify_ex(q, p, drafts, uniforms, 0, 0.0, 1.0, rule_per_seq=rule,
                                        alpha_per_seq=alpha, temp_per_seq=temperature)
        return acc, tok


@dataclass
class DecodeResult:
    tokens: list                      # per sequence: the emitted tokens, in order
    accept_len: list = field(default_factory=list)  # per round: [B] int tensor (j*)

    def tokens_per_round(self):
        """Mean emitted tokens per sequence and round (j* + 1)."""
        n = sum(int(a.sum()) + a.numel() for a in self.accept_len)
        return n / (len(self.accept_len) * self.accept_len[0].numel())


def spec_decode(drafter, verifier, first_tokens, rounds, gamma, rule, alpha, temperature,
                seed=0, backend=None, rounds_inputs=None):
    """Run ``rounds`` rounds of GenSpecSample for B sequences whose last
    prefix token is ``first_tokens`` [B] (at position 0).  ``rule``,
    ``alpha`` and ``temperature`` are scalars or [B] tensors (temperature 0:
    greedy).  Uniforms come from a torch.Generator seeded with ``seed``;
    ``rounds_inputs`` (a list), when given, receives each round's inputs so a
    test can replay them through another backend.

    The rounds run without waiting for the device: emitted tokens are
    scattered into a device buffer (a round writes its gamma+1 candidates at
    the sequence's length and advances the length by j* + 1, so the
    candidates past j* are overwritten by the next round), and the host reads
    the buffer and the accept lengths once, after the last round."""
    backend = backend or GpuBackend()
    dev = verifier.device
    B = first_tokens.numel()
    g1 = gamma + 1

    def per_seq(x, dtype):
        t = torch.as_tensor(x, dtype=dtype, device=dev)
        return t.expand(B).contiguous() if t.dim() == 0 else t.to(dev).contiguous()

    rule_t = per_seq(rule, torch.int32)
    alpha_t = per_seq(alpha, torch.float32)
    temp_t = per_seq(temperature, torch.float32)
    gen = torch.Generator(device=dev).manual_seed(seed)
    # round state, updated in place by every round
    last = first_tokens.to(dev, torch.int32).clone()
    pos = torch.zeros(B, dtype=torch.int64, device=dev)
    buf = torch.zeros(B, rounds * g1 + g1, dtype=torch.int32, device=dev)
    length = torch.zeros(B, dtype=torch.int64, device=dev)
    acc_out = torch.zeros(B, dtype=torch.int64, device=dev)
    ar = torch.arange(g1, device=dev)

    def one_round(u_draft, u):
        # 1. draft gamma tokens from q, and q's logits at the extra position
        q_rows, drafts = [], []
        tok = last
        for j in range(g1):
            zq = drafter(tok, pos + j).contiguous()
            q_rows.append(zq)
            if j < gamma:
                tok = backend.draft_sample(zq, temp_t, u_draft[j].contiguous())
                drafts.append(tok)
        q = torch.stack(q_rows, dim=1).contiguous()            # [B, gamma+1, V]
        x = torch.stack(drafts, dim=1).to(torch.int32).contiguous()  # [B, gamma]
        # 2. score the gamma+1 prefixes with p in one batch
        ctx = torch.cat([last[:, None], x], dim=1)             # last tokens of x_{<t+j}
        p = verifier(ctx.reshape(-1), (pos[:, None] + ar).reshape(-1))
        p = p.reshape(B, g1, -1).contiguous()
        # 3. verify
        if rounds_inputs is not None:
            rounds_inputs.append(dict(q=q, p=p, draft=x, uniforms=u, u_draft=u_draft,
                                      rule=rule_t, alpha=alpha_t, temperature=temp_t))
        acc, nxt = backend.verify(q, p, x, u, rule_t, alpha_t, temp_t)
        # 4. emit x_t .. x_{t+j*-1} and the new token, roll back to t + j* + 1
        acc = acc.to(dev).long()
        nxt = nxt.to(dev, torch.int32)
        j = acc.clamp(min=0)
        cand = torch.cat([x, nxt[:, None]], dim=1)
        cand = torch.where(ar[None, :] == j[:, None], nxt[:, None], cand)
        buf.scatter_(1, length[:, None] + ar[None, :], cand)
        length.add_(j + 1)
        pos.add_(j + 1)
        last.copy_(nxt)
        acc_out.copy_(acc)

    def uniforms():
        return (torch.rand(gamma, B, generator=gen, device=dev),
                torch.rand(B, g1, generator=gen, device=dev))

    accs = torch.zeros(rounds, B, dtype=torch.int64, device=dev)
    for r in range(rounds):
        one_round(*uniforms())
        accs[r].copy_(acc_out)
    acc_h = accs.cpu()
    bad = (acc_h < 0).nonzero()
    if bad.numel():
        raise RuntimeError(f"sequence {int(bad[0, 1])}: invalid parameters (accept_len -1)")
    buf_h, len_h = buf.cpu(), length.cpu()
    res = DecodeResult(tokens=[buf_h[b, :int(len_h[b])].tolist() for b in range(B)])
    res.accept_len = [a.to(torch.int32) for a in acc_h]
    return res


def synthetic_pair(V, seed=0, dtype=torch.bfloat16, device="cuda", rows=64):
    """A verifier SyntheticLM and a drafter derived from it as the Gemma-vocab
    workload's drafter (0.8 x verifier + N(0, 1))."""
    p = SyntheticLM(V, rows=rows, s=1.2, noise=1.0, seed=seed, dtype=dtype, device=device)
    return p.derive(scale=0.8, sigma=1.0, seed=seed + 1), p


__all__ = ["SyntheticLM", "GpuBackend", "DecodeResult", "spec_decode", "synthetic_pair"]
