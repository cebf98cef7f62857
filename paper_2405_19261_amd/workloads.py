"""Seeded synthetic inputs for the verify step.

This module only *draws* inputs: logits, draft tokens, uniforms and the
per-sequence parameters.  It contains none of the verify arithmetic and
imports nothing from the GPU library or from the oracle, so both sides can be
fed the same bytes.

The five workloads stand in for the paper's T5 (vocabulary ~32k) and Gemma
(vocabulary 256k) drafter/verifier pairs, whose weights and datasets are not
used here.  Logits are made in float32 and, for bfloat16 workloads, rounded
to bfloat16 (round to nearest even); the stored tensor is what both the GPU
and the oracle read.  Each row of a "Zipf" base gets logit ``-s * ln(rank)``
with ranks 1..V scattered by a per-row seeded permutation.

Seeds: logits ``1000*cfg + step``, uniforms ``+1_000_000``, drafts
``+2_000_000``, each on its own ``torch.Generator`` on the target device.
"""
from dataclasses import dataclass, replace
import math

import torch

# Rule codes (same numbering as the C interface).
CHOW, DIFF, OPT, ALWAYS, NEVER = 0, 1, 2, 3, 4
TOKEN_V1, TOKEN_V2, TOKEN_V3 = 5, 6, 7
LOSSY, BILD, CHOWLOG, DIFFLOG, OPTLOG = 8, 9, 10, 11, 12
RULE_NAMES = {CHOW: "chow", DIFF: "diff", OPT: "opt", ALWAYS: "always", NEVER: "never",
              TOKEN_V1: "token-v1", TOKEN_V2: "token-v2", TOKEN_V3: "token-v3",
              LOSSY: "lossy", BILD: "bild", CHOWLOG: "chowlog", DIFFLOG: "difflog",
              OPTLOG: "optlog"}


@dataclass(frozen=True)
class Workload:
    cfg: int
    name: str
    B: int
    gamma: int
    V: int
    dtype: str            # "f32" or "bf16"
    rule: int             # -1: per-sequence mix
    alpha: float
    temperature: float    # 0.0: greedy
    steps: int

    @property
    def rows(self):
        return self.B * (self.gamma + 1)

    @property
    def elem_bytes(self):
        return 4 if self.dtype == "f32" else 2

    @property
    def greedy(self):
        return self.temperature == 0.0

    def logit_bytes(self):
        """q and p, each read once."""
        return 2 * self.rows * self.V * self.elem_bytes

    def algorithmic_bytes(self):
        """Logits + drafts + uniforms + outputs of one step."""
        B, g = self.B, self.gamma
        uni = 0 if self.greedy else 4 * B * (g + 1)
        return self.logit_bytes() + 4 * B * g + uni + 4 * B + 4 * B + B * (g + 1)

    def with_(self, **kw):
        return replace(self, **kw)


WORKLOADS = {
    1: Workload(1, "tiny B=1 gamma=4 V=1000 f32 chow", 1, 4, 1000, "f32", CHOW, 0.5, 1.0, 1000),
    2: Workload(2, "t5-vocab B=8 gamma=5 V=32128 f32 opt", 8, 5, 32128, "f32", OPT, 0.1, 1.0,
                10000),
    3: Workload(3, "gemma-vocab B=32 gamma=7 V=256000 bf16 diff", 32, 7, 256000, "bf16", DIFF,
                0.05, 1.0, 100),
    4: Workload(4, "greedy B=128 gamma=4 V=256000 bf16 opt T=0", 128, 4, 256000, "bf16", OPT,
                0.1, 0.0, 50),
    5: Workload(5, "stress-mix B=256 gamma=8 V=256000 bf16 mixed", 256, 8, 256000, "bf16", -1,
                0.0, 1.0, 20),
}

CFG5_TEMPS = (0.5, 0.7, 1.0)
CFG5_RULES = ((CHOW, 0.4), (DIFF, 0.05), (OPT, 0.1))


def _gen(device, seed):
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def _normal(shape, std, g, device):
    return torch.randn(shape, generator=g, device=device, dtype=torch.float32) * std


def _zipf_rows(R, V, s, g, device, rows_per_chunk=256):
    """-s * ln(rank) with ranks 1..V scattered by a per-row random permutation."""
    out = torch.empty((R, V), device=device, dtype=torch.float32)
    base = -s * torch.log(torch.arange(1, V + 1, device=device, dtype=torch.float64))
    base = base.to(torch.float32)
    for r0 in range(0, R, rows_per_chunk):
        r1 = min(R, r0 + rows_per_chunk)
        perm = torch.argsort(torch.rand((r1 - r0, V), generator=g, device=device), dim=1)
        out[r0:r1] = base[perm]
        del perm
    return out


def _pick_rows(R, frac, g, device):
    n = math.ceil(frac * R)
    return torch.randperm(R, generator=g, device=device)[:n]


def generate(wl: Workload, step: int, device="cpu"):
    """Inputs of one verify step of workload ``wl`` on ``device``.

    Returns a dict of tensors: q, p [B, gamma+1, V] (float32 or bfloat16),
    draft [B, gamma] int32, uniforms [B, gamma+1] float32 in [0, 1),
    rule [B] int32, alpha [B] float32, temperature [B] float32.
    """
    device = torch.device(device)
    B, g1, V = wl.B, wl.gamma + 1, wl.V
    R = B * g1
    gl = _gen(device, 1000 * wl.cfg + step)
    gu = _gen(device, 1000 * wl.cfg + step + 1_000_000)
    gd = _gen(device, 1000 * wl.cfg + step + 2_000_000)

    rule = torch.full((B,), wl.rule, dtype=torch.int32, device=device)
    alpha = torch.full((B,), wl.alpha, dtype=torch.float32, device=device)
    temp = torch.full((B,), wl.temperature, dtype=torch.float32, device=device)

    if wl.cfg == 1:
        p = _normal((R, V), 2.0, gl, device)
        q = p + _normal((R, V), 0.5, gl, device)
    elif wl.cfg == 2:
        p = _zipf_rows(R, V, 1.1, gl, device) + _normal((R, V), 1.0, gl, device)
        q = p + _normal((R, V), 0.8, gl, device)
    elif wl.cfg in (3, 4):
        p = _zipf_rows(R, V, 1.2, gl, device) + _normal((R, V), 1.0, gl, device)
        q = 0.8 * p + _normal((R, V), 1.0, gl, device)
        noisy = _pick_rows(R, 0.10, gl, device)
        q[noisy] += _normal((noisy.numel(), V), math.sqrt(3.0), gl, device)
    elif wl.cfg == 5:
        p = _zipf_rows(R, V, 1.2, gl, device) + _normal((R, V), 1.0, gl, device)
        q = 0.8 * p + _normal((R, V), 1.0, gl, device)
        seq_perm = torch.randperm(B, generator=gl, device=device)
        n_same, n_indep = B // 4, B // 4
        same = seq_perm[:n_same]
        indep = seq_perm[n_same:n_same + n_indep]
        mixed = seq_perm[n_same + n_indep:]
        # config-3 recipe on the remaining half, incl. the extra-noise rows
        mixed_rows = (mixed[:, None] * g1 + torch.arange(g1, device=device)[None, :]).reshape(-1)
        noisy = mixed_rows[_pick_rows(mixed_rows.numel(), 0.10, gl, device)]
        q[noisy] += _normal((noisy.numel(), V), math.sqrt(3.0), gl, device)
        q = q.view(B, g1, V)
        p3 = p.view(B, g1, V)
        q[indep] = _normal((indep.numel(), g1, V), 2.0, gl, device)
        q[same] = p3[same]
        q = q.view(R, V)
        temp = torch.tensor(CFG5_TEMPS, dtype=torch.float32, device=device)[
            torch.randint(0, len(CFG5_TEMPS), (B,), generator=gl, device=device)]
        pick = torch.randint(0, len(CFG5_RULES), (B,), generator=gl, device=device)
        rule = torch.tensor([r for r, _ in CFG5_RULES], dtype=torch.int32, device=device)[pick]
        alpha = torch.tensor([a for _, a in CFG5_RULES], dtype=torch.float32,
                             device=device)[pick]
    else:
        raise ValueError(f"unknown workload {wl.cfg}")

    dt = torch.float32 if wl.dtype == "f32" else torch.bfloat16
    q = q.view(B, g1, V).to(dt).contiguous()
    p = p.view(B, g1, V).to(dt).contiguous()
    if wl.cfg == 5:
        # the identical-drafter sequences must stay bit-identical after rounding
        q[same] = p[same]

    uniforms = torch.rand((B, g1), generator=gu, device=device, dtype=torch.float32)
    draft = draw_drafts(q, temp, gd)
    return dict(q=q, p=p, draft=draft, uniforms=uniforms, rule=rule, alpha=alpha,
                temperature=temp)


def draw_drafts(q, temperature, g):
    """Draft tokens x_{t+j} ~ softmax(q_{t+j} / T) for j < gamma, or the argmax
    (first maximal index) where T == 0.  Uses torch's own softmax/multinomial."""
    B, g1, V = q.shape
    gamma = g1 - 1
    z = q[:, :gamma, :].float()
    out = torch.empty((B, gamma), dtype=torch.int32, device=q.device)
    greedy = temperature == 0
    for b in range(B):
        if bool(greedy[b]):
            out[b] = torch.argmax(z[b], dim=-1).to(torch.int32)
        else:
            probs = torch.softmax(z[b] / temperature[b], dim=-1)
            out[b] = torch.multinomial(probs, 1, generator=g).view(-1).to(torch.int32)
    return out
