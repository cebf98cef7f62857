"""An oracle-backed backend for the decoding loop (test infrastructure): the
same two calls as decode.GpuBackend, answered by the fp64 CPU oracle."""
import numpy as np
import torch

import oracle


def _host(t):
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


class OracleBackend:
    def __init__(self):
        self.margins = []  # per call: the oracle's decision margins

    def draft_sample(self, logits, temperature, uniforms):
        T = temperature.cpu().numpy()
        tok, mg = oracle.draft_sample(_host(logits), T, uniforms.cpu().numpy())
        self.margins.append(("draft", mg))
        return torch.as_tensor(tok, device=logits.device)

    def verify(self, q, p, drafts, uniforms, rule, alpha, temperature):
        hq, hp = _host(q), _host(p)
        x, u = drafts.cpu().numpy(), uniforms.cpu().numpy()
        r, a, T = rule.cpu().numpy(), alpha.cpu().numpy(), temperature.cpu().numpy()
        B = hq.shape[0]
        acc = np.empty(B, np.int32)
        tok = np.empty(B, np.int32)
        for greedy in (True, False):
            sel = (T == 0) if greedy else (T > 0)
            if not sel.any():
                continue
            if greedy:
                o = oracle.greedy_verify(hq[sel], hp[sel], x[sel], r[sel], a[sel])
            else:
                o = oracle.verify(hq[sel], hp[sel], x[sel], u[sel], r[sel], a[sel], T[sel])
                self.margins.append(("verify", o))
            acc[sel], tok[sel] = o["accept_len"], o["next_token"]
        dev = q.device
        return torch.as_tensor(acc, device=dev), torch.as_tensor(tok, device=dev)
