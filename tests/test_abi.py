"""The C interface loads, exports every function include/speccascade.h
declares, and rejects bad arguments before any HIP call (CPU only: every call
here fails its argument checks, so nothing is launched)."""
import ctypes
import os
import re

import pytest

from paper_2405_19261_amd import spc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "speccascade.h")

FAKE = ctypes.c_void_p(0x10000)      # never dereferenced: every call below fails first
FAKE_ODD = ctypes.c_void_p(0x10008)  # 8- but not 16-byte aligned


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(spc_\w+)\s*\(", text)))


def test_exports_every_declared_symbol():
    L = spc.lib()
    names = _declared()
    assert {"spc_verify", "spc_greedy_verify", "spc_verify_ex", "spc_workspace_bytes",
            "spc_last_error", "spc_release", "spc_version"} <= set(names)
    for n in names:
        assert hasattr(L, n), n
    assert "gfx950" in spc.spc_version()


def _verify(**kw):
    a = dict(q=FAKE, p=FAKE, dtype=spc.SPC_BF16, draft=FAKE, u=FAKE, B=2, gamma=3, V=100,
             rule=spc.SPC_RULE_DIFF, alpha=0.1, T=1.0, acc=FAKE, tok=FAKE, dm=FAKE)
    a.update(kw)
    return spc.lib().spc_verify(a["q"], a["p"], a["dtype"], a["draft"], a["u"], a["B"],
                                a["gamma"], a["V"], a["rule"], a["alpha"], a["T"], a["acc"],
                                a["tok"], a["dm"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(q=None), -1), (dict(p=None), -1), (dict(draft=None), -1), (dict(u=None), -1),
    (dict(acc=None), -1), (dict(tok=None), -1), (dict(dm=None), -1),
    (dict(B=0), -2), (dict(gamma=0), -2), (dict(gamma=64), -2), (dict(V=1), -2),
    (dict(rule=13), -3), (dict(rule=-1), -3), (dict(rule=8, alpha=1.0), -4),
    (dict(alpha=float("nan")), -4), (dict(alpha=float("inf")), -4),
    (dict(T=0.0), -4), (dict(T=-1.0), -4), (dict(T=float("nan")), -4),
    (dict(T=float("inf")), -4), (dict(dtype=7), -4),
    (dict(q=FAKE_ODD), -5), (dict(p=FAKE_ODD), -5),
])
def test_argument_errors(kw, status):
    assert _verify(**kw) == status
    assert spc.spc_last_error() != ""


@pytest.mark.parametrize("kw", [
    dict(B=10000, gamma=7),      # 80000 rows: consecutive launches of whole sequences
    dict(B=2_000_000, gamma=63),
    dict(T=1e-30), dict(T=1.17549435e-38), dict(T=1e-45),  # tiny positive temperatures
])
def test_accepted_shapes_and_temperatures(kw):
    """Large batches and tiny positive temperatures pass every shape and
    parameter check: the call stops at the misaligned logits instead."""
    assert _verify(q=FAKE_ODD, **kw) == -5


def test_greedy_argument_errors():
    L = spc.lib()
    # no uniforms needed; bad rule / shape still rejected
    assert L.spc_greedy_verify(FAKE, FAKE, 1, FAKE, 2, 3, 100, 13, 0.1, FAKE, FAKE, FAKE,
                               None) == -3
    assert L.spc_greedy_verify(FAKE, FAKE, 1, FAKE, 2, 0, 100, 1, 0.1, FAKE, FAKE, FAKE,
                               None) == -2
    assert L.spc_greedy_verify(FAKE, FAKE, 1, None, 2, 3, 100, 1, 0.1, FAKE, FAKE, FAKE,
                               None) == -1


def test_workspace_errors_and_sizes():
    L = spc.lib()
    n = spc.spc_workspace_bytes(32, 7, 256000, spc.SPC_BF16)
    z = spc.spc_workspace_zero_bytes(32, 7, 256000, spc.SPC_BF16)
    assert 0 < z < n and n % 256 == 0 and z % 256 == 0
    assert spc.spc_workspace_bytes(0, 7, 256000, spc.SPC_BF16) == 0
    ex = spc.ExArgs()
    ex.workspace = ctypes.c_void_p(0x100000)
    ex.workspace_bytes = n - 1
    st = L.spc_verify_ex(FAKE, FAKE, 1, FAKE, FAKE, 32, 7, 256000, 1, 0.05, 1.0, FAKE, FAKE,
                         FAKE, ctypes.byref(ex), None)
    assert st == -6
    ex.workspace = ctypes.c_void_p(0x100010)  # misaligned
    ex.workspace_bytes = n
    st = L.spc_verify_ex(FAKE, FAKE, 1, FAKE, FAKE, 32, 7, 256000, 1, 0.05, 1.0, FAKE, FAKE,
                         FAKE, ctypes.byref(ex), None)
    assert st == -6


def test_ex_per_sequence_arrays_skip_scalar_checks():
    """With per-sequence arrays the scalar rule/alpha/temperature are not used,
    so only the remaining checks apply (here: a misaligned q)."""
    L = spc.lib()
    ex = spc.ExArgs()
    ex.rule_per_seq = FAKE
    ex.alpha_per_seq = FAKE
    ex.temp_per_seq = FAKE
    st = L.spc_verify_ex(FAKE_ODD, FAKE, 1, FAKE, FAKE, 4, 3, 1000, 99, float("nan"), 0.0,
                         FAKE, FAKE, FAKE, ctypes.byref(ex), None)
    assert st == -5


@pytest.mark.parametrize("kw,status", [
    (dict(z=None), -1), (dict(tok=None), -1), (dict(u=None), -1),
    (dict(B=0), -2), (dict(V=1), -2),
    (dict(T=-0.5), -4), (dict(T=float("nan")), -4), (dict(T=float("inf")), -4),
    (dict(dtype=3), -4), (dict(z=FAKE_ODD), -5),
])
def test_draft_sample_argument_errors(kw, status):
    a = dict(z=FAKE, dtype=spc.SPC_BF16, B=4, V=1000, T=1.0, tps=None, u=FAKE, tok=FAKE)
    a.update(kw)
    st = spc.lib().spc_draft_sample(a["z"], a["dtype"], a["B"], a["V"], a["T"], a["tps"],
                                    a["u"], a["tok"], None)
    assert st == status
    assert spc.spc_last_error() != ""


def test_draft_sample_greedy_needs_no_uniforms():
    """T = 0 takes no uniforms: the call gets past every argument check (here
    it stops at the misaligned logits, before any HIP call)."""
    st = spc.lib().spc_draft_sample(FAKE_ODD, spc.SPC_BF16, 4, 1000, 0.0, None, None, FAKE, None)
    assert st == -5


def test_draft_workspace_errors_and_sizes():
    L = spc.lib()
    n = spc.spc_draft_workspace_bytes(32, 256000, spc.SPC_BF16)
    z = spc.spc_workspace_zero_bytes(1, 1, 2, spc.SPC_BF16)
    assert 0 < z < n and n % 256 == 0
    assert spc.spc_draft_workspace_bytes(0, 256000, spc.SPC_BF16) == 0
    for ws, nb in ((0x100000, n - 1), (0x100010, n)):  # too small; misaligned
        st = L.spc_draft_sample_ws(FAKE, spc.SPC_BF16, 32, 256000, 1.0, None, FAKE, FAKE,
                                   ctypes.c_void_p(ws), nb, None)
        assert st == -6
        assert spc.spc_last_error() != ""
    # a large batch passes the shape check (consecutive launches)
    st = L.spc_draft_sample_ws(FAKE_ODD, spc.SPC_BF16, 100000, 1000, 1.0, None, FAKE, FAKE,
                               None, 0, None)
    assert st == -5
