"""ctypes binding of the fp64 CPU oracle (``oracle/spc_oracle.c``).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, the smoke check and the
benchmark's CPU-baseline leg, never by the GPU library.  Arrays are numpy;
logits may be float32, float64, or uint16 (raw bfloat16 bits).
"""
import ctypes
import os

import numpy as np

from .build import LIB, build

_lib = None

F32, BF16, F64 = 0, 1, 2
CHOW, DIFF, OPT, ALWAYS, NEVER = 0, 1, 2, 3, 4
TOKEN_V1, TOKEN_V2, TOKEN_V3 = 5, 6, 7
LOSSY, BILD, CHOWLOG, DIFFLOG, OPTLOG = 8, 9, 10, 11, 12
FLAG_DRAFT_OUT_OF_RANGE, FLAG_EMPTY_RESIDUAL = 1, 2

_P = ctypes.c_void_p
_I32, _I64, _D = ctypes.c_int32, ctypes.c_int64, ctypes.c_double


class RowStats(ctypes.Structure):
    _fields_ = [("m", ctypes.c_double), ("lse", ctypes.c_double),
                ("maxprob", ctypes.c_double), ("argmax", ctypes.c_int32)]


def lib():
    """Load the oracle library, compiling it first if it is not built."""
    global _lib
    if _lib is None:
        # SPC_ORACLE_LIB: another build of the oracle (e.g. with sanitizers)
        path = os.environ.get("SPC_ORACLE_LIB") or LIB
        if path == LIB and not os.path.exists(LIB):
            build()
        L = ctypes.CDLL(path)
        L.orc_softmax_row.argtypes = [_P, ctypes.c_int, _I64, _D, _P, ctypes.POINTER(RowStats)]
        L.orc_softmax_row.restype = None
        L.orc_tv.argtypes = [_P, _P, _I64]
        L.orc_tv.restype = _D
        L.orc_defer.argtypes = [ctypes.c_int, _D, _D, _D, _D, ctypes.POINTER(_D)]
        L.orc_defer.restype = ctypes.c_int
        L.orc_target.argtypes = [ctypes.c_int, _P, _P, _I64, _P]
        L.orc_target.restype = None
        L.orc_accept.argtypes = [_D, _D, _D, ctypes.POINTER(_D)]
        L.orc_accept.restype = ctypes.c_int
        L.orc_residual.argtypes = [_P, _P, _I64, _P]
        L.orc_residual.restype = _D
        L.orc_token_r.argtypes = [ctypes.c_int, _D, _D, _D, _D, ctypes.POINTER(_D)]
        L.orc_token_r.restype = ctypes.c_int
        L.orc_token_target.argtypes = [ctypes.c_int, _D, _P, _P, _I64, _D, _P, ctypes.POINTER(_D)]
        L.orc_token_target.restype = _D
        L.orc_entropy_row.argtypes = [_P, ctypes.c_int, _I64, _D, ctypes.POINTER(RowStats)]
        L.orc_entropy_row.restype = _D
        L.orc_cross_entropy_row.argtypes = [_P, _P, ctypes.c_int, _I64, _D,
                                            ctypes.POINTER(RowStats), ctypes.POINTER(RowStats)]
        L.orc_cross_entropy_row.restype = _D
        L.orc_log_defer.argtypes = [_D, _D, _D, ctypes.POINTER(_D)]
        L.orc_log_defer.restype = ctypes.c_int
        L.orc_lossy_target.argtypes = [_D, _P, _P, _I64, _P]
        L.orc_lossy_target.restype = None
        L.orc_sample.argtypes = [_P, _I64, _D, ctypes.POINTER(_D)]
        L.orc_sample.restype = _I32
        L.orc_draft_sample.argtypes = [_P, ctypes.c_int, _I32, _I64, _P, _P, _P, _P]
        L.orc_draft_sample.restype = ctypes.c_int
        L.orc_verify.argtypes = [_P, _P, ctypes.c_int, _P, _P, _I32, _I32, _I64, _P, _P, _P,
                                 _P, _P, _P, _P, _P, _P, _P, _P, _P]
        L.orc_verify.restype = ctypes.c_int
        L.orc_greedy_verify.argtypes = [_P, _P, ctypes.c_int, _P, _I32, _I32, _I64, _P, _P,
                                        _P, _P, _P, _P, _P, _P, _P]
        L.orc_greedy_verify.restype = ctypes.c_int
        L.orc_num_threads.argtypes = []
        L.orc_num_threads.restype = ctypes.c_int
        L.orc_set_num_threads.argtypes = [ctypes.c_int]
        L.orc_set_num_threads.restype = None
        _lib = L
    return _lib


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def _logits(a):
    a = np.ascontiguousarray(a)
    if a.dtype == np.float32:
        return a, F32
    if a.dtype == np.float64:
        return a, F64
    if a.dtype in (np.uint16, np.int16):
        return a.view(np.uint16), BF16
    raise TypeError(f"unsupported logit dtype {a.dtype}")


def _per_seq(x, B, dtype):
    a = np.asarray(x, dtype=dtype)
    if a.ndim == 0:
        a = np.full(B, a, dtype=dtype)
    assert a.shape == (B,)
    return np.ascontiguousarray(a)


def num_threads():
    return lib().orc_num_threads()


def set_num_threads(n):
    lib().orc_set_num_threads(int(n))


def softmax_row(z, T=1.0):
    """(prob, m, lse, maxprob, argmax) of softmax(z / T) for one row."""
    z, dt = _logits(z)
    V = z.shape[-1]
    prob = np.empty(V, np.float64)
    st = RowStats()
    lib().orc_softmax_row(_ptr(z), dt, V, float(T), _ptr(prob), ctypes.byref(st))
    return prob, st.m, st.lse, st.maxprob, st.argmax


def _row_stats(z, dt, T):
    st = RowStats()
    lib().orc_softmax_row(_ptr(z), dt, z.shape[-1], float(T), None, ctypes.byref(st))
    return st


def entropy_row(z, T=1.0):
    """H(softmax(z / T)) in nats."""
    z, dt = _logits(z)
    st = _row_stats(z, dt, T)
    return lib().orc_entropy_row(_ptr(z), dt, z.shape[-1], float(T), ctypes.byref(st))


def cross_entropy_row(zq, zp, T=1.0):
    """-sum_v q(v) log p(v) for q = softmax(zq / T), p = softmax(zp / T)."""
    zq, dt = _logits(zq)
    zp, dt2 = _logits(zp)
    assert dt == dt2 and zq.shape == zp.shape
    sq, sp = _row_stats(zq, dt, T), _row_stats(zp, dt, T)
    return lib().orc_cross_entropy_row(_ptr(zq), _ptr(zp), dt, zq.shape[-1], float(T),
                                       ctypes.byref(sq), ctypes.byref(sp))


def log_defer(s, threshold, mag=None):
    mg = _D()
    d = lib().orc_log_defer(float(s), float(threshold), float(s if mag is None else mag),
                            ctypes.byref(mg))
    return d, mg.value


def lossy_target(alpha, q, p):
    q = np.ascontiguousarray(q, np.float64)
    p = np.ascontiguousarray(p, np.float64)
    pi = np.empty_like(q)
    lib().orc_lossy_target(float(alpha), _ptr(q), _ptr(p), q.size, _ptr(pi))
    return pi


def tv(p, q):
    p = np.ascontiguousarray(p, np.float64)
    q = np.ascontiguousarray(q, np.float64)
    return lib().orc_tv(_ptr(p), _ptr(q), p.size)


def defer(rule, alpha, maxq, maxp, tv_=0.0):
    mg = _D()
    d = lib().orc_defer(rule, float(alpha), float(maxq), float(maxp), float(tv_), ctypes.byref(mg))
    return d, mg.value


def target(delta, q, p):
    q = np.ascontiguousarray(q, np.float64)
    p = np.ascontiguousarray(p, np.float64)
    pi = np.empty_like(q)
    lib().orc_target(int(delta), _ptr(q), _ptr(p), q.size, _ptr(pi))
    return pi


def token_r(rule, alpha, qv, pv, maxp):
    mg = _D()
    r = lib().orc_token_r(rule, float(alpha), float(qv), float(pv), float(maxp), ctypes.byref(mg))
    return r, mg.value


def token_target(rule, alpha, q, p, maxp):
    """(pi, eta, rmargin) of the token-specific target for one row."""
    q = np.ascontiguousarray(q, np.float64)
    p = np.ascontiguousarray(p, np.float64)
    pi = np.empty_like(q)
    mg = _D()
    eta = lib().orc_token_target(rule, float(alpha), _ptr(q), _ptr(p), q.size, float(maxp),
                                 _ptr(pi), ctypes.byref(mg))
    return pi, eta, mg.value


def accept(pi_x, q_x, u):
    mg = _D()
    a = lib().orc_accept(float(pi_x), float(q_x), float(u), ctypes.byref(mg))
    return a, mg.value


def residual(pi, q):
    pi = np.ascontiguousarray(pi, np.float64)
    q = np.ascontiguousarray(q, np.float64)
    w = np.empty_like(q)
    W = lib().orc_residual(_ptr(pi), _ptr(q), q.size, _ptr(w))
    return w, W


def sample(w, u):
    w = np.ascontiguousarray(w, np.float64)
    mg = _D()
    k = lib().orc_sample(_ptr(w), w.size, float(u), ctypes.byref(mg))
    return k, mg.value


def verify(q, p, draft, uniforms, rule, alpha, temperature):
    """One verify step for B sequences.  q, p: [B, gamma+1, V]; draft: [B, gamma];
    uniforms: [B, gamma+1]; rule/alpha/temperature: scalars or [B]."""
    q, dt = _logits(q)
    p, dt2 = _logits(p)
    assert dt == dt2 and q.shape == p.shape and q.ndim == 3
    B, G, V = q.shape
    gamma = G - 1
    draft = np.ascontiguousarray(draft, np.int32)
    uniforms = np.ascontiguousarray(uniforms, np.float32)
    assert draft.shape == (B, gamma) and uniforms.shape == (B, G)
    rule = _per_seq(rule, B, np.int32)
    alpha = _per_seq(alpha, B, np.float32)
    temperature = _per_seq(temperature, B, np.float32)
    out = dict(
        accept_len=np.empty(B, np.int32), next_token=np.empty(B, np.int32),
        defer=np.empty((B, G), np.uint8), row_stats=np.empty((B, G, 8), np.float64),
        defer_margin=np.empty((B, G)), accept_margin=np.empty((B, gamma)),
        sample_margin=np.empty(B), sample_norm=np.empty(B), flags=np.empty(B, np.int32))
    rc = lib().orc_verify(
        _ptr(q), _ptr(p), dt, _ptr(draft), _ptr(uniforms), B, gamma, V, _ptr(rule),
        _ptr(alpha), _ptr(temperature), _ptr(out["accept_len"]), _ptr(out["next_token"]),
        _ptr(out["defer"]), _ptr(out["row_stats"]), _ptr(out["defer_margin"]),
        _ptr(out["accept_margin"]), _ptr(out["sample_margin"]), _ptr(out["sample_norm"]),
        _ptr(out["flags"]))
    if rc != 0:
        raise ValueError("orc_verify rejected its arguments")
    return out


def greedy_verify(q, p, draft, rule, alpha):
    """The temperature-0 step (Lemma 6) for B sequences."""
    q, dt = _logits(q)
    p, dt2 = _logits(p)
    assert dt == dt2 and q.shape == p.shape and q.ndim == 3
    B, G, V = q.shape
    gamma = G - 1
    draft = np.ascontiguousarray(draft, np.int32)
    assert draft.shape == (B, gamma)
    rule = _per_seq(rule, B, np.int32)
    alpha = _per_seq(alpha, B, np.float32)
    out = dict(
        accept_len=np.empty(B, np.int32), next_token=np.empty(B, np.int32),
        defer=np.empty((B, G), np.uint8), row_stats=np.empty((B, G, 8), np.float64),
        argmax=np.empty((B, G, 2), np.int32), defer_margin=np.empty((B, G)),
        flags=np.empty(B, np.int32))
    rc = lib().orc_greedy_verify(
        _ptr(q), _ptr(p), dt, _ptr(draft), B, gamma, V, _ptr(rule), _ptr(alpha),
        _ptr(out["accept_len"]), _ptr(out["next_token"]), _ptr(out["defer"]),
        _ptr(out["row_stats"]), _ptr(out["argmax"]), _ptr(out["defer_margin"]),
        _ptr(out["flags"]))
    if rc != 0:
        raise ValueError("orc_greedy_verify rejected its arguments")
    return out


def draft_sample(logits, temperature, uniforms=None):
    """The drafter's sampling step: one token per row of ``logits`` [B, V]
    from softmax(z / T_b) by the inverse CDF at ``uniforms[b]``, or the argmax
    where T_b = 0.  Returns (tokens [B] int32, margins [B])."""
    z, dt = _logits(logits)
    B, V = z.shape
    T = np.ascontiguousarray(np.broadcast_to(np.asarray(temperature, np.float32), (B,)))
    u = None if uniforms is None else np.ascontiguousarray(uniforms, np.float32)
    tok = np.empty(B, np.int32)
    mg = np.empty(B, np.float64)
    rc = lib().orc_draft_sample(_ptr(z), dt, B, V, _ptr(T), None if u is None else _ptr(u),
                                _ptr(tok), _ptr(mg))
    if rc != 0:
        raise ValueError("orc_draft_sample: bad arguments")
    return tok, mg
