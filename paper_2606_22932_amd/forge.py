"""Python binding of the C ABI in ``include/forge.h`` (argument marshalling only).

Every function here has the name of the C entry point it calls.  Tensors are torch
tensors on the current HIP device; their data pointers, shapes and the current torch
stream are passed through ctypes.  All arithmetic runs in the HIP kernels of
``libforge.so``; there is no fallback: if the library is not built, calls raise.
"""
from __future__ import annotations

import ctypes
import os
import re
import threading

from . import build as _build

FORGE_MOMENT_F32, FORGE_MOMENT_BF16, FORGE_MOMENT_I8, FORGE_MOMENT_I8_ROW64, FORGE_MOMENT_FP8 = 0, 1, 2, 3, 4
AMAX_SLOTS = 4
FORGE_GRAD_BF16, FORGE_GRAD_F32 = 0, 1

STATUS = {
    0: "FORGE_OK", 1: "FORGE_ERR_NULL_POINTER", 2: "FORGE_ERR_INVALID_SHAPE",
    3: "FORGE_ERR_UNSUPPORTED_SHAPE", 4: "FORGE_ERR_INVALID_HYPERPARAM",
    5: "FORGE_ERR_INVALID_DTYPE", 6: "FORGE_ERR_MISALIGNED", 7: "FORGE_ERR_ALIASING",
    8: "FORGE_ERR_NO_DEVICE", 9: "FORGE_ERR_LAUNCH", 10: "FORGE_ERR_INVALID_OPTIMIZER",
    11: "FORGE_ERR_SCRATCH_LIMIT",
}
# bytes of the library's fixed device buffer (FORGE_SCRATCH_BYTES)
FORGE_SCRATCH_BYTES = 64 << 20
# forge_optimizer codes of include/forge.h
OPTIMIZERS = {"adamw": 0, "sgd": 1, "sgd_momentum": 2, "adagrad": 3, "rmsprop": 4, "lion": 5, "nadam": 6,
              "radam": 7, "adamax": 8, "muon_accumulate": 9}
# state tensors each update rule reads and writes
OPTIMIZER_STATES = {"adamw": 2, "sgd": 0, "sgd_momentum": 1, "adagrad": 1, "rmsprop": 1, "lion": 1, "nadam": 2,
                    "radam": 2, "adamax": 2, "muon_accumulate": 1}
HEADER = os.path.join(_build.ROOT, "include", "forge.h")


class ForgeError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        self.name = STATUS.get(code, "unknown")
        super().__init__(f"{where}: {forge_status_string(code)}")


_lock = threading.Lock()
_lib = None

_P, _I64, _I32, _F = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_float
FORGE_MAX_GROUP = 8


class forge_hparams(ctypes.Structure):
    """``forge_hparams`` of ``include/forge.h``."""
    _fields_ = [("lr", _F), ("beta1", _F), ("beta2", _F), ("eps", _F), ("weight_decay", _F),
                ("lr_decay", _F), ("momentum_decay", _F)]


class forge_matrix(ctypes.Structure):
    """``forge_matrix`` of ``include/forge.h``: one matrix of a grouped step."""
    _fields_ = [("X", _P), ("dY", _P), ("W", _P), ("m", _P), ("v", _P), ("m_scale", _P),
                ("v_scale", _P), ("d_in", _I64), ("d_out", _I64)]


_SIGS = {
    "forge_linear_step": [_P, _P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _I32, _F, _F, _F, _F, _F, _I64, _P],
    "forge_linear_step_grouped": [ctypes.POINTER(forge_matrix), _I32, _I64, _I32, _F, _F, _F, _F, _F,
                                  _I64, _P],
    "forge_linear_step_opt": [_P, _P, _P, _P, _P, _I64, _I64, _I64, _I32, _I32, ctypes.POINTER(forge_hparams),
                              _I64, _P],
    "forge_linear_step_wfp8": [_P, _P, _P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _I32, _F, _F, _F, _F, _F, _I64,
                               _P],
    "forge_input_grad": [_P, _P, _P, _I64, _I64, _I64, _P],
    "forge_linear_backward": [_P, _P, _P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _I32, _F, _F, _F, _F, _F,
                              _I64, _P],
    "forge_linear_backward_grouped": [ctypes.POINTER(forge_matrix), _I32, _I64, _P, _I32, _F, _F, _F, _F,
                                      _F, _I64, _P],
    "forge_wgrad": [_P, _P, _P, _I64, _I64, _I64, _I32, _P],
    "forge_adamw": [_P, _I32, _P, _P, _P, _P, _P, _I64, _I64, _I32, _F, _F, _F, _F, _F, _I64, _P],
    "forge_linear_step_unfused": [_P, _P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _I32, _F, _F, _F, _F,
                                  _F, _I64, _P, _I32, _P],
    "forge_linear_step_unfused_noalloc": [_P, _P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _I32, _F, _F, _F, _F,
                                          _F, _I64, _I32, _P],
    "forge_status_string": [_I32],
    "forge_query_tile": [_I64, _I64, _I64, _I32, ctypes.POINTER(_I32), ctypes.POINTER(_I32),
                         ctypes.POINTER(_I32)],
}


def lib():
    """The loaded ``libforge.so`` (raises if it has not been built)."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_build.LIB):
                raise RuntimeError(
                    f"{_build.LIB} is not built: run `python -m paper_2606_22932_amd.build` "
                    "(or __graft_entry__.build()) first; there is no non-HIP fallback")
            L = ctypes.CDLL(_build.LIB)
            for name, args in _SIGS.items():
                fn = getattr(L, name)
                fn.argtypes = args
                fn.restype = ctypes.c_char_p if name == "forge_status_string" else ctypes.c_int32
            _lib = L
    return _lib


def header_functions():
    """Names of the functions ``include/forge.h`` declares."""
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(forge_[a-z_0-9]+)\s*\(", text)))


def forge_status_string(code: int) -> str:
    return lib().forge_status_string(int(code)).decode()


def forge_query_tile(T: int, d_in: int, d_out: int, moment_dtype: int):
    r, c, t = _I32(), _I32(), _I32()
    st = lib().forge_query_tile(int(T), int(d_in), int(d_out), int(moment_dtype), ctypes.byref(r),
                                ctypes.byref(c), ctypes.byref(t))
    _check(st, "forge_query_tile")
    return r.value, c.value, t.value


# ----------------------------------------------------------------------------- marshalling

def _check(status: int, where: str):
    if status != 0:
        raise ForgeError(status, where)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream, ref):
    if stream is not None:
        return ctypes.c_void_p(int(stream))
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream(ref.device).cuda_stream)


def _moment_code(m, m_scale=None):
    """Moment dtype code; int8 moments name their layout through the scale tensor's shape:
    [ceil(d_out/256), d_in] (256-row column blocks) or [d_out, ceil(d_in/64)] (64-wide row
    blocks)."""
    import torch
    codes = {torch.float32: FORGE_MOMENT_F32, torch.bfloat16: FORGE_MOMENT_BF16,
             torch.float8_e4m3fn: FORGE_MOMENT_FP8}
    if m.dtype in codes:
        if m.dtype == torch.float8_e4m3fn and (m_scale is None or m_scale.numel() != AMAX_SLOTS):
            raise ValueError(f"fp8 moments need amax rings of {AMAX_SLOTS} float32 (m_scale, v_scale)")
        return codes[m.dtype]
    if m.dtype != torch.int8:
        raise TypeError(f"moments must be float32, bfloat16 or int8, got {m.dtype}")
    if m_scale is None:
        raise ValueError("int8 moments need their scale tensors")
    d_out, d_in = m.shape
    if tuple(m_scale.shape) == ((d_out + 255) // 256, d_in):
        return FORGE_MOMENT_I8
    if tuple(m_scale.shape) == (d_out, (d_in + 63) // 64):
        return FORGE_MOMENT_I8_ROW64
    raise ValueError(f"int8 scale shape {tuple(m_scale.shape)} matches neither layout for moments {tuple(m.shape)}")


def _grad_code(G):
    import torch
    codes = {torch.bfloat16: FORGE_GRAD_BF16, torch.float32: FORGE_GRAD_F32}
    if G.dtype not in codes:
        raise TypeError(f"gradient must be bfloat16 or float32, got {G.dtype}")
    return codes[G.dtype]


def _dev(*ts):
    for t in ts:
        if t is not None:
            if not t.is_cuda:
                raise ValueError("forge tensors must live on a HIP device")
            if not t.is_contiguous():
                raise ValueError("forge tensors must be contiguous")


def _shapes(X, dY, W):
    import torch
    if W.dtype != torch.bfloat16 or X.dtype != torch.bfloat16 or dY.dtype != torch.bfloat16:
        raise TypeError("X, dY and W must be bfloat16")
    T, d_in = X.shape
    T2, d_out = dY.shape
    if T2 != T or tuple(W.shape) != (d_out, d_in):
        raise ValueError(f"shape mismatch: X {tuple(X.shape)}, dY {tuple(dY.shape)}, W {tuple(W.shape)}")
    return T, d_in, d_out


def forge_linear_step(X, dY, W, m, v, m_scale=None, v_scale=None, *, lr, beta1, beta2, eps,
                      weight_decay, step, stream=None):
    """The fused step: W, m, v (and int8 scales) updated in place; G is never stored."""
    _dev(X, dY, W, m, v, m_scale, v_scale)
    T, d_in, d_out = _shapes(X, dY, W)
    st = lib().forge_linear_step(_ptr(X), _ptr(dY), _ptr(W), _ptr(m), _ptr(v), _ptr(m_scale),
                                 _ptr(v_scale), T, d_in, d_out, _moment_code(m, m_scale), lr, beta1, beta2,
                                 eps, weight_decay, int(step), _stream(stream, W))
    _check(st, "forge_linear_step")


def forge_linear_step_opt(X, dY, W, s1=None, s2=None, *, optimizer, lr, beta1=0.0, beta2=0.0, eps=1e-8,
                          weight_decay=0.0, lr_decay=0.0, momentum_decay=0.004, step, stream=None):
    """The fused step with update rule ``optimizer`` (a key of OPTIMIZERS) on fp32 or bf16
    state tensors s1, s2 (as many as the rule has).  W may be None for 'muon_accumulate'."""
    import torch
    if optimizer not in OPTIMIZERS:
        raise ValueError(f"unknown optimizer {optimizer!r}; one of {sorted(OPTIMIZERS)}")
    ns = OPTIMIZER_STATES[optimizer]
    states = [t for t in (s1, s2)[:ns]]
    if any(t is None for t in states):
        raise ValueError(f"{optimizer} needs {ns} state tensor(s)")
    _dev(X, dY, W, *states)
    if X.dtype != torch.bfloat16 or dY.dtype != torch.bfloat16:
        raise TypeError("X and dY must be bfloat16")
    T, d_in = X.shape
    T2, d_out = dY.shape
    if T2 != T:
        raise ValueError("X and dY disagree on T")
    for t in ([W] if W is not None else []):
        if t.dtype != torch.bfloat16 or tuple(t.shape) != (d_out, d_in):
            raise ValueError("W must be bfloat16 [d_out, d_in]")
    code = FORGE_MOMENT_BF16
    if states:
        if states[0].dtype == torch.int8:
            raise ValueError("forge_linear_step_opt takes float32 or bfloat16 state")
        code = _moment_code(states[0])
        if any(t.dtype != states[0].dtype or tuple(t.shape) != (d_out, d_in)
                                          for t in states):
            raise ValueError("state tensors must all be float32 or all bfloat16, [d_out, d_in]")
    hp = forge_hparams(lr, beta1, beta2, eps, weight_decay, lr_decay, momentum_decay)
    ref = W if W is not None else dY
    st = lib().forge_linear_step_opt(_ptr(X), _ptr(dY), _ptr(W), _ptr(s1 if ns >= 1 else None),
                                     _ptr(s2 if ns >= 2 else None), T, d_in, d_out, OPTIMIZERS[optimizer], code,
                                     ctypes.byref(hp), int(step), _stream(stream, ref))
    _check(st, "forge_linear_step_opt")


def forge_linear_step_wfp8(X, dY, W, w_amax, m, v, m_amax=None, v_amax=None, *, lr, beta1, beta2, eps,
                           weight_decay, step, stream=None):
    """The fused step with W in fp8 (float8_e4m3fn codes, amax ring ``w_amax`` of 4 float32)
    and bf16 moments, or fp8 moments (float8_e4m3fn codes of m and sqrt(v) with their rings)."""
    import torch
    _dev(X, dY, W, w_amax, m, v, m_amax, v_amax)
    if X.dtype != torch.bfloat16 or dY.dtype != torch.bfloat16 or W.dtype != torch.float8_e4m3fn:
        raise TypeError("X, dY must be bfloat16 and W float8_e4m3fn")
    T, d_in = X.shape
    T2, d_out = dY.shape
    if T2 != T or tuple(W.shape) != (d_out, d_in):
        raise ValueError(f"shape mismatch: X {tuple(X.shape)}, dY {tuple(dY.shape)}, W {tuple(W.shape)}")
    if w_amax.dtype != torch.float32 or w_amax.numel() != AMAX_SLOTS:
        raise ValueError(f"w_amax must be {AMAX_SLOTS} float32")
    code = _moment_code(m, m_amax)
    if code not in (FORGE_MOMENT_BF16, FORGE_MOMENT_FP8):
        raise TypeError("moments must be bfloat16 or float8_e4m3fn")
    st = lib().forge_linear_step_wfp8(_ptr(X), _ptr(dY), _ptr(W), _ptr(w_amax), _ptr(m), _ptr(v), _ptr(m_amax),
                                      _ptr(v_amax), T, d_in, d_out, code, lr, beta1, beta2, eps, weight_decay,
                                      int(step), _stream(stream, W))
    _check(st, "forge_linear_step_wfp8")


def _group(mats):
    """ctypes array of forge_matrix for (X, dY, W, m, v[, m_scale, v_scale]) tuples, T, dtype code."""
    mats = [tuple(x) + (None,) * (7 - len(x)) for x in mats]
    if not mats:
        raise ValueError("empty group")
    arr = (forge_matrix * len(mats))()
    T = code = None
    for i, (X, dY, W, m, v, ms, vs) in enumerate(mats):
        _dev(X, dY, W, m, v, ms, vs)
        Ti, d_in, d_out = _shapes(X, dY, W)
        ci = _moment_code(m, ms)
        if T is None:
            T, code = Ti, ci
        elif Ti != T or ci != code:
            raise ValueError("all matrices of a group share T and the moment dtype")
        arr[i] = forge_matrix(X.data_ptr(), dY.data_ptr(), W.data_ptr(), m.data_ptr(), v.data_ptr(),
                              None if ms is None else ms.data_ptr(), None if vs is None else vs.data_ptr(),
                              d_in, d_out)
    return arr, len(mats), T, code, mats[0][2]


def forge_linear_step_grouped(mats, *, lr, beta1, beta2, eps, weight_decay, step, stream=None):
    """The fused step on several independent matrices in one launch.

    ``mats``: sequence of ``(X, dY, W, m, v)`` or ``(X, dY, W, m, v, m_scale, v_scale)``
    tuples sharing the token count T and the moment dtype (at most FORGE_MAX_GROUP).
    """
    arr, n, T, code, ref = _group(mats)
    st = lib().forge_linear_step_grouped(arr, n, T, code, lr, beta1, beta2, eps, weight_decay,
                                         int(step), _stream(stream, ref))
    _check(st, "forge_linear_step_grouped")


def _dx(dX, T, d_in):
    import torch
    _dev(dX)
    if dX.dtype != torch.bfloat16 or tuple(dX.shape) != (T, d_in):
        raise ValueError(f"dX must be bfloat16 [{T}, {d_in}], got {dX.dtype} {tuple(dX.shape)}")


def forge_input_grad(dY, W, dX, *, stream=None):
    """dX = dY W (bf16 out, fp32 accumulation): the layer's input gradient."""
    import torch
    _dev(dY, W)
    if dY.dtype != torch.bfloat16 or W.dtype != torch.bfloat16:
        raise TypeError("dY and W must be bfloat16")
    T, d_out = dY.shape
    if W.shape[0] != d_out:
        raise ValueError(f"shape mismatch: dY {tuple(dY.shape)}, W {tuple(W.shape)}")
    d_in = W.shape[1]
    _dx(dX, T, d_in)
    st = lib().forge_input_grad(_ptr(dY), _ptr(W), _ptr(dX), T, d_in, d_out, _stream(stream, dX))
    _check(st, "forge_input_grad")


def forge_linear_backward(X, dY, W, m, v, m_scale=None, v_scale=None, *, dX, lr, beta1, beta2, eps,
                          weight_decay, step, stream=None):
    """The layer-level backward: dX = dY W from the pre-update W, then the fused step."""
    _dev(X, dY, W, m, v, m_scale, v_scale)
    T, d_in, d_out = _shapes(X, dY, W)
    _dx(dX, T, d_in)
    st = lib().forge_linear_backward(_ptr(X), _ptr(dY), _ptr(W), _ptr(m), _ptr(v), _ptr(m_scale),
                                     _ptr(v_scale), _ptr(dX), T, d_in, d_out, _moment_code(m, m_scale), lr, beta1,
                                     beta2, eps, weight_decay, int(step), _stream(stream, W))
    _check(st, "forge_linear_backward")


def forge_linear_backward_grouped(mats, *, dX, lr, beta1, beta2, eps, weight_decay, step, stream=None):
    """Backward of several projections of one input: dX = sum_i dY_i W_i (pre-update
    weights, one launch), then the grouped fused step.  ``mats`` as for
    ``forge_linear_step_grouped``; all share d_in."""
    arr, n, T, code, ref = _group(mats)
    _dx(dX, T, arr[0].d_in)
    st = lib().forge_linear_backward_grouped(arr, n, T, _ptr(dX), code, lr, beta1, beta2, eps,
                                             weight_decay, int(step), _stream(stream, ref))
    _check(st, "forge_linear_backward_grouped")


def forge_wgrad(X, dY, G, *, stream=None):
    """G = dY^T X stored in G's dtype (bfloat16 or float32)."""
    _dev(X, dY, G)
    T, d_in = X.shape
    d_out = dY.shape[1]
    if tuple(G.shape) != (d_out, d_in):
        raise ValueError("G must be [d_out, d_in]")
    st = lib().forge_wgrad(_ptr(X), _ptr(dY), _ptr(G), T, d_in, d_out, _grad_code(G), _stream(stream, G))
    _check(st, "forge_wgrad")


def forge_adamw(G, W, m, v, m_scale=None, v_scale=None, *, lr, beta1, beta2, eps, weight_decay,
                step, stream=None):
    """The stand-alone optimizer kernel over a materialised gradient G."""
    _dev(G, W, m, v, m_scale, v_scale)
    d_out, d_in = W.shape
    if tuple(G.shape) != (d_out, d_in):
        raise ValueError("G must match W")
    st = lib().forge_adamw(_ptr(G), _grad_code(G), _ptr(W), _ptr(m), _ptr(v), _ptr(m_scale),
                           _ptr(v_scale), d_in, d_out, _moment_code(m, m_scale), lr, beta1, beta2, eps,
                           weight_decay, int(step), _stream(stream, W))
    _check(st, "forge_adamw")


def forge_linear_step_unfused(X, dY, W, m, v, m_scale=None, v_scale=None, *, G_ws, lr, beta1,
                              beta2, eps, weight_decay, step, stream=None):
    """GEMM writes G into G_ws, then the optimizer kernel reads it (same stream)."""
    _dev(X, dY, W, m, v, m_scale, v_scale, G_ws)
    T, d_in, d_out = _shapes(X, dY, W)
    if G_ws.numel() < d_in * d_out:
        raise ValueError("G_ws too small")
    st = lib().forge_linear_step_unfused(_ptr(X), _ptr(dY), _ptr(W), _ptr(m), _ptr(v),
                                         _ptr(m_scale), _ptr(v_scale), T, d_in, d_out,
                                         _moment_code(m, m_scale), lr, beta1, beta2, eps, weight_decay,
                                         int(step), _ptr(G_ws), _grad_code(G_ws), _stream(stream, W))
    _check(st, "forge_linear_step_unfused")


def forge_linear_step_unfused_noalloc(X, dY, W, m, v, m_scale=None, v_scale=None, *, grad_dtype, lr, beta1,
                                      beta2, eps, weight_decay, step, stream=None):
    """forge_linear_step_unfused with G in the library's fixed device buffer: allocates
    nothing.  grad_dtype: "bf16" or "f32"."""
    _dev(X, dY, W, m, v, m_scale, v_scale)
    T, d_in, d_out = _shapes(X, dY, W)
    gd = {"bf16": FORGE_GRAD_BF16, "f32": FORGE_GRAD_F32}[grad_dtype]
    st = lib().forge_linear_step_unfused_noalloc(_ptr(X), _ptr(dY), _ptr(W), _ptr(m), _ptr(v),
                                                 _ptr(m_scale), _ptr(v_scale), T, d_in, d_out,
                                                 _moment_code(m, m_scale), lr, beta1, beta2, eps, weight_decay,
                                                 int(step), gd, _stream(stream, W))
    _check(st, "forge_linear_step_unfused_noalloc")
