"""Python binding of libspeccascade (the C interface in include/speccascade.h).

Argument marshalling only: every step of the verify path runs in the gfx950
kernels of ``libspeccascade.so``.  Functions carry the C names; tensors are
torch tensors on the current HIP device (PyTorch supplies device memory and
streams, nothing else).  A missing or unloadable library raises -- there is no
fallback implementation.
"""
import ctypes
import os

import torch

# SPC_LIB_PATH selects another build of the library (e.g. a tuning variant)
LIB_PATH = os.environ.get("SPC_LIB_PATH") or os.path.join(
    os.path.dirname(os.path.abspath(__file__)), "libspeccascade.so")

SPC_F32, SPC_BF16 = 0, 1
SPC_RULE_CHOW, SPC_RULE_DIFF, SPC_RULE_OPT, SPC_RULE_ALWAYS, SPC_RULE_NEVER = range(5)
SPC_RULE_TOKEN_V1, SPC_RULE_TOKEN_V2, SPC_RULE_TOKEN_V3 = 5, 6, 7
SPC_RULE_LOSSY, SPC_RULE_BILD, SPC_RULE_CHOWLOG, SPC_RULE_DIFFLOG, SPC_RULE_OPTLOG = range(8, 13)
SPC_MAX_GAMMA = 63
STATUS = {0: "SPC_OK", -1: "SPC_E_NULL", -2: "SPC_E_SHAPE", -3: "SPC_E_RULE",
          -4: "SPC_E_PARAM", -5: "SPC_E_ALIGN", -6: "SPC_E_WORKSPACE", -7: "SPC_E_HIP"}

_P = ctypes.c_void_p
_I32 = ctypes.c_int32


class ExArgs(ctypes.Structure):
    """spc_verify_ex_args."""
    _fields_ = [("rule_per_seq", _P), ("alpha_per_seq", _P), ("temp_per_seq", _P),
                ("out_row_stats", _P), ("out_argmax", _P), ("out_sample_norm", _P),
                ("workspace", _P), ("workspace_bytes", ctypes.c_size_t),
                ("rules_present", ctypes.c_uint32), ("ev_tiles_begin", _P),
                ("ev_tiles_end", _P)]


class SpcError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


_lib = None


def lib():
    """The loaded shared library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built: run `python -m "
                               "paper_2405_19261_amd.build` (or __graft_entry__.build())")
        L = ctypes.CDLL(LIB_PATH)
        common = [_P, _P, ctypes.c_int]
        L.spc_verify.argtypes = common + [_P, _P, _I32, _I32, _I32, _I32, ctypes.c_float,
                                          ctypes.c_float, _P, _P, _P, _P]
        L.spc_verify.restype = ctypes.c_int
        L.spc_greedy_verify.argtypes = common + [_P, _I32, _I32, _I32, _I32, ctypes.c_float,
                                                 _P, _P, _P, _P]
        L.spc_greedy_verify.restype = ctypes.c_int
        L.spc_verify_ex.argtypes = common + [_P, _P, _I32, _I32, _I32, _I32, ctypes.c_float,
                                             ctypes.c_float, _P, _P, _P,
                                             ctypes.POINTER(ExArgs), _P]
        L.spc_verify_ex.restype = ctypes.c_int
        L.spc_verify_noalloc.argtypes = L.spc_verify_ex.argtypes
        L.spc_verify_noalloc.restype = ctypes.c_int
        L.spc_noalloc_scratch_bytes.argtypes = []
        L.spc_noalloc_scratch_bytes.restype = ctypes.c_size_t
        L.spc_draft_sample.argtypes = [_P, ctypes.c_int, _I32, _I32, ctypes.c_float, _P, _P, _P,
                                       _P]
        L.spc_draft_sample.restype = ctypes.c_int
        L.spc_draft_sample_ws.argtypes = [_P, ctypes.c_int, _I32, _I32, ctypes.c_float, _P, _P,
                                          _P, _P, ctypes.c_size_t, _P]
        L.spc_draft_sample_ws.restype = ctypes.c_int
        L.spc_draft_workspace_bytes.argtypes = [_I32, _I32, ctypes.c_int]
        L.spc_draft_workspace_bytes.restype = ctypes.c_size_t
        L.spc_workspace_bytes.argtypes = [_I32, _I32, _I32, ctypes.c_int]
        L.spc_workspace_bytes.restype = ctypes.c_size_t
        L.spc_workspace_zero_bytes.argtypes = [_I32, _I32, _I32, ctypes.c_int]
        L.spc_workspace_zero_bytes.restype = ctypes.c_size_t
        L.spc_last_error.argtypes = []
        L.spc_last_error.restype = ctypes.c_char_p
        L.spc_release.argtypes = []
        L.spc_release.restype = None
        L.spc_version.argtypes = []
        L.spc_version.restype = ctypes.c_char_p
        _lib = L
    return _lib


def _dtype_code(t):
    if t.dtype == torch.float32:
        return SPC_F32
    if t.dtype == torch.bfloat16:
        return SPC_BF16
    raise TypeError(f"logits must be float32 or bfloat16, not {t.dtype}")


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _check(status):
    if status != 0:
        raise SpcError(status, lib().spc_last_error().decode())


def _outputs(q, B, gamma, out):
    if out is not None:
        return out
    dev = q.device
    return (torch.empty(B, dtype=torch.int32, device=dev),
            torch.empty(B, dtype=torch.int32, device=dev),
            torch.empty((B, gamma + 1), dtype=torch.uint8, device=dev))


def _shape(q, p, draft):
    if q.dim() != 3 or q.shape != p.shape or q.dtype != p.dtype:
        raise ValueError("q and p must both be [B, gamma+1, V] of one dtype")
    if not (q.is_contiguous() and p.is_contiguous()):
        raise ValueError("inputs must be contiguous")
    if p.device != q.device:
        raise ValueError("q and p must be on one device")
    B, g1, V = q.shape
    _check_arg("draft", draft, torch.int32, q.device, (B, g1 - 1))
    return B, g1 - 1, V


def _check_arg(name, t, dtype, device, shape=None):
    """Raise unless t is a contiguous tensor of dtype on device (of shape)."""
    if t is None:
        return
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, not {t.dtype}")
    if t.device != device:
        raise ValueError(f"{name} must be on {device}, not {t.device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, not {tuple(t.shape)}")


def spc_verify(q, p, draft, uniforms, rule, alpha, temperature, out=None, stream=None):
    """One verify step; returns (accept_len [B], next_token [B], defer_mask [B, gamma+1])."""
    B, gamma, V = _shape(q, p, draft)
    _check_arg("uniforms", uniforms, torch.float32, q.device, (B, gamma + 1))
    acc, tok, dm = _outputs(q, B, gamma, out)
    _check(lib().spc_verify(_ptr(q), _ptr(p), _dtype_code(q), _ptr(draft), _ptr(uniforms), B,
                            gamma, V, int(rule), float(alpha), float(temperature), _ptr(acc),
                            _ptr(tok), _ptr(dm), _stream(stream)))
    return acc, tok, dm


def spc_greedy_verify(q, p, draft, rule, alpha, out=None, stream=None):
    """The temperature-0 step; returns (accept_len, next_token, defer_mask)."""
    B, gamma, V = _shape(q, p, draft)
    acc, tok, dm = _outputs(q, B, gamma, out)
    _check(lib().spc_greedy_verify(_ptr(q), _ptr(p), _dtype_code(q), _ptr(draft), B, gamma, V,
                                   int(rule), float(alpha), _ptr(acc), _ptr(tok), _ptr(dm),
                                   _stream(stream)))
    return acc, tok, dm


def _verify_ex(entry, q, p, draft, uniforms, rule, alpha, temperature, rule_per_seq=None,
               alpha_per_seq=None, temp_per_seq=None, out_row_stats=None, out_argmax=None,
               out_sample_norm=None, workspace=None, rules_present=0, ev_tiles=None, out=None,
               stream=None):
    """spc_verify with per-sequence parameters and optional outputs.
    rules_present: bitmask of the rule ids rule_per_seq may hold (0 = any).
    ev_tiles: for profiling, a pair of raw hipEvent_t handles (integers)
    recorded around the statistics kernel of the call's first launch."""
    B, gamma, V = _shape(q, p, draft)
    dev = q.device
    _check_arg("uniforms", uniforms, torch.float32, dev, (B, gamma + 1))
    _check_arg("rule_per_seq", rule_per_seq, torch.int32, dev, (B,))
    _check_arg("alpha_per_seq", alpha_per_seq, torch.float32, dev, (B,))
    _check_arg("temp_per_seq", temp_per_seq, torch.float32, dev, (B,))
    _check_arg("out_row_stats", out_row_stats, torch.float32, dev, (B, gamma + 1, 8))
    _check_arg("out_argmax", out_argmax, torch.int32, dev, (B, gamma + 1, 2))
    _check_arg("out_sample_norm", out_sample_norm, torch.float32, dev, (B,))
    acc, tok, dm = _outputs(q, B, gamma, out)
    ex = ExArgs()
    ex.rule_per_seq = _ptr(rule_per_seq)
    ex.alpha_per_seq = _ptr(alpha_per_seq)
    ex.temp_per_seq = _ptr(temp_per_seq)
    ex.out_row_stats = _ptr(out_row_stats)
    ex.out_argmax = _ptr(out_argmax)
    ex.out_sample_norm = _ptr(out_sample_norm)
    if workspace is not None:
        if workspace.device != dev or not workspace.is_contiguous():
            raise ValueError("workspace must be a contiguous tensor on the logits' device")
        ex.workspace = _ptr(workspace)
        ex.workspace_bytes = workspace.numel() * workspace.element_size()
    ex.rules_present = int(rules_present)
    if ev_tiles is not None:
        ex.ev_tiles_begin, ex.ev_tiles_end = int(ev_tiles[0]), int(ev_tiles[1])
    _check(getattr(lib(), entry)(_ptr(q), _ptr(p), _dtype_code(q), _ptr(draft), _ptr(uniforms), B,
                                  gamma, V, int(rule), float(alpha), float(temperature),
                                  _ptr(acc), _ptr(tok), _ptr(dm), ctypes.byref(ex),
                                  _stream(stream)))
    return acc, tok, dm


def spc_verify_ex(q, p, draft, uniforms, rule, alpha, temperature, **kw):
    """spc_verify with per-sequence parameters and optional outputs (keyword
    arguments of _verify_ex: rule_per_seq, alpha_per_seq, temp_per_seq,
    out_row_stats, out_argmax, out_sample_norm, workspace, rules_present,
    ev_tiles, out, stream); returns (accept_len, next_token, defer_mask)."""
    return _verify_ex("spc_verify_ex", q, p, draft, uniforms, rule, alpha, temperature, **kw)


def spc_verify_noalloc(q, p, draft, uniforms, rule, alpha, temperature, **kw):
    """spc_verify_ex on the library's static scratch: no device allocation
    (``workspace`` must be None)."""
    return _verify_ex("spc_verify_noalloc", q, p, draft, uniforms, rule, alpha, temperature,
                      **kw)


def spc_noalloc_scratch_bytes():
    return lib().spc_noalloc_scratch_bytes()


def spc_draft_sample(logits, temperature, uniforms=None, temp_per_seq=None, out=None,
                     workspace=None, stream=None):
    """The drafter's sampling step: one token per row of ``logits`` [B, V]
    (float32 or bfloat16, contiguous) from softmax(z / T), T = 0 giving the
    argmax.  Returns the tokens [B] int32 (``out`` if given).  ``workspace``:
    an optional caller workspace (a uint8 tensor of at least
    spc_draft_workspace_bytes bytes, zeroed before its first use)."""
    if logits.dim() != 2 or not logits.is_contiguous():
        raise ValueError("logits must be a contiguous [B, V] tensor")
    B, V = logits.shape
    dev = logits.device
    _check_arg("uniforms", uniforms, torch.float32, dev, (B,))
    _check_arg("temp_per_seq", temp_per_seq, torch.float32, dev, (B,))
    tok = out if out is not None else torch.empty(B, dtype=torch.int32, device=dev)
    _check_arg("out", tok, torch.int32, dev, (B,))
    if workspace is None:
        _check(lib().spc_draft_sample(_ptr(logits), _dtype_code(logits), B, V, float(temperature),
                                      _ptr(temp_per_seq), _ptr(uniforms), _ptr(tok),
                                      _stream(stream)))
    else:
        if workspace.device != dev or not workspace.is_contiguous():
            raise ValueError("workspace must be a contiguous tensor on the logits' device")
        _check(lib().spc_draft_sample_ws(_ptr(logits), _dtype_code(logits), B, V,
                                         float(temperature), _ptr(temp_per_seq), _ptr(uniforms),
                                         _ptr(tok), _ptr(workspace),
                                         workspace.numel() * workspace.element_size(),
                                         _stream(stream)))
    return tok


def spc_workspace_bytes(B, gamma, V, dtype_code):
    return lib().spc_workspace_bytes(B, gamma, V, dtype_code)


def spc_workspace_zero_bytes(B, gamma, V, dtype_code):
    return lib().spc_workspace_zero_bytes(B, gamma, V, dtype_code)


def spc_draft_workspace_bytes(B, V, dtype_code):
    return lib().spc_draft_workspace_bytes(B, V, dtype_code)


def spc_last_error():
    return lib().spc_last_error().decode()


def spc_release():
    lib().spc_release()


def spc_version():
    return lib().spc_version().decode()
