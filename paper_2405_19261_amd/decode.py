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
    """Sampling and verification through libspeccascade.

    ``prepare`` (called once by ``spec_decode`` before the rounds) reads the
    per-sequence parameters on the host.  When every sequence shares one
    rule, alpha and temperature the calls take the scalar forms, so the
    library launches only the kernels that rule needs (no argmax at T > 0);
    otherwise the per-sequence arrays go with the ``rules_present`` mask of
    the rules they hold."""

    def __init__(self):
        self._scalar = None
        self._rules_present = 0

    def prepare(self, rule, alpha, temperature):
        r, a, t = rule.cpu(), alpha.cpu(), temperature.cpu()
        self._rules_present = sum(1 << int(x) for x in set(r.tolist()) if 0 <= x < 31)
        same = bool((r == r[0]).all() and (a == a[0]).all() and (t == t[0]).all())
        self._scalar = (int(r[0]), float(a[0]), float(t[0])) if same else None

    def draft_sample(self, logits, temperature, uniforms):
        if self._scalar is not None:
            T = self._scalar[2]
            return spc.spc_draft_sample(logits, T, uniforms=uniforms if T > 0 else None)
        return spc.spc_draft_sample(logits, 0.0, uniforms=uniforms, temp_per_seq=temperature)

    def verify(self, q, p, drafts, uniforms, rule, alpha, temperature):
        if self._scalar is not None:
            acc, tok, _ = spc.spc_verify_ex(q, p, drafts, uniforms, *self._scalar)
        else:
            acc, tok, _ = spc.spc_verify_ex(q, p, drafts, uniforms, 0, 0.0, 1.0,
                                            rule_per_seq=rule, alpha_per_seq=alpha,
                                            temp_per_seq=temperature,
                                            rules_present=self._rules_present)
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
                seed=0, backend=None, rounds_inputs=None, graph=False):
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
    the buffer and the accept lengths once, after the last round.

    ``graph=True`` captures one round (the 2*gamma+1 model and sampling calls,
    the verification and the emission) into a HIP graph and replays it once
    per round, so a round costs one launch instead of dozens.  The round's
    uniforms are drawn up front in the eager order and copied into the
    graph's input buffers before each replay, so the tokens equal the eager
    loop's.  The models and the backend must be capturable (no host syncs,
    no allocation outside torch's allocator); one eager round, whose effects
    are undone, sizes the library's workspace before the capture."""
    backend = backend or GpuBackend()
    if graph and rounds_inputs is not None:
        raise ValueError("rounds_inputs needs the eager loop (graph=False)")
    dev = verifier.device
    B = first_tokens.numel()
    g1 = gamma + 1

    def per_seq(x, dtype):
        t = torch.as_tensor(x, dtype=dtype, device=dev)
        return t.expand(B).contiguous() if t.dim() == 0 else t.to(dev).contiguous()

    rule_t = per_seq(rule, torch.int32)
    alpha_t = per_seq(alpha, torch.float32)
    temp_t = per_seq(temperature, torch.float32)
    if hasattr(backend, "prepare"):
        backend.prepare(rule_t, alpha_t, temp_t)
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
    if graph:
        drawn = [uniforms() for _ in range(rounds)]
        ud_in, u_in = torch.empty_like(drawn[0][0]), torch.empty_like(drawn[0][1])
        # warm-up on a side stream (the library sizes its workspace here);
        # the round state is restored afterwards
        state = [t.clone() for t in (last, pos, buf, length, acc_out)]
        side = torch.cuda.Stream(device=dev)
        side.wait_stream(torch.cuda.current_stream(dev))
        with torch.cuda.stream(side):
            ud_in.copy_(drawn[0][0])
            u_in.copy_(drawn[0][1])
            one_round(ud_in, u_in)
            for t, t0 in zip((last, pos, buf, length, acc_out), state):
                t.copy_(t0)
        torch.cuda.current_stream(dev).wait_stream(side)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            one_round(ud_in, u_in)
        for r in range(rounds):
            ud_in.copy_(drawn[r][0])
            u_in.copy_(drawn[r][1])
            g.replay()
            accs[r].copy_(acc_out)
        torch.cuda.current_stream(dev).synchronize()
        del g
    else:
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
