"""CPU oracle for the fused weight-gradient + AdamW step (FORGE, Sec. 2.2, Algorithm 1).

TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the benchmark's
CPU-baseline leg may import this package.  It shares no code with the HIP library and
imports nothing from it.

The arithmetic lives in ``forge_oracle.c`` (plain fp64 C loops, OpenMP over rows);
this module compiles it with gcc, loads it with ctypes and marshals numpy arrays.
bf16 tensors are passed as ``numpy.uint16`` bit patterns.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "forge_oracle.c")
_LIB = os.path.join(_HERE, "libforge_oracle.so")

MOMENT_F32, MOMENT_BF16, MOMENT_I8, MOMENT_I8_ROW64 = 0, 1, 2, 3
ROW_BLOCK = 64
# Update rules (forge_oracle_rule_step); AdamW is ``adamw``.
OPT_ADAMW, OPT_SGD, OPT_SGD_MOMENTUM, OPT_ADAGRAD, OPT_RMSPROP, OPT_LION = 0, 1, 2, 3, 4, 5
OPT_NADAM, OPT_RADAM, OPT_ADAMAX, OPT_MUON = 6, 7, 8, 9
# state tensors of each rule, and whether it updates W
RULE_STATES = {OPT_ADAMW: 2, OPT_SGD: 0, OPT_SGD_MOMENTUM: 1, OPT_ADAGRAD: 1, OPT_RMSPROP: 1, OPT_LION: 1,
               OPT_NADAM: 2, OPT_RADAM: 2, OPT_ADAMAX: 2, OPT_MUON: 1}
I8_BLOCK = 256

_lock = threading.Lock()
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle into ``oracle/libforge_oracle.so`` with gcc (-O3, OpenMP, no fast-math)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.check_call(
            ["gcc", "-O3", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall",
             "-fno-fast-math", "-ffp-contract=off", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
                build(force=True)
            lib = ctypes.CDLL(_LIB)
            P, I64, F32, I32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_float, ctypes.c_int
            lib.forge_oracle_bf16_to_f64.argtypes = [ctypes.c_uint16]
            lib.forge_oracle_bf16_to_f64.restype = ctypes.c_double
            lib.forge_oracle_f64_to_bf16.argtypes = [ctypes.c_double]
            lib.forge_oracle_f64_to_bf16.restype = ctypes.c_uint16
            lib.forge_oracle_wgrad.argtypes = [P, P, I64, I64, I64, P]
            lib.forge_oracle_wgrad.restype = None
            lib.forge_oracle_f64_to_bf16_array.argtypes = [P, I64, P]
            lib.forge_oracle_f64_to_bf16_array.restype = None
            lib.forge_oracle_quantize_i8_row64.argtypes = [P, I64, I64, I32, P, P, P]
            lib.forge_oracle_quantize_i8_row64.restype = None
            lib.forge_oracle_adamw_i8row.argtypes = [P, P, P, P, P, P, I64, I64, F32, F32, F32, F32, F32, I64,
                                                     P, P, P, P, P]
            lib.forge_oracle_adamw_i8row.restype = None
            lib.forge_oracle_e4m3_decode.argtypes = [ctypes.c_uint8]
            lib.forge_oracle_e4m3_decode.restype = ctypes.c_double
            lib.forge_oracle_e4m3_encode_array.argtypes = [P, I64, P]
            lib.forge_oracle_e4m3_encode_array.restype = None
            lib.forge_oracle_adamw_fp8.argtypes = [P, P, I32, P, P, P, I32, P, P, I64, I64, F32, F32, F32, F32, F32,
                                                   I64, P, P, P, P, P, P]
            lib.forge_oracle_adamw_fp8.restype = None
            lib.forge_oracle_input_grad.argtypes = [P, P, I64, I64, I64, P]
            lib.forge_oracle_input_grad.restype = None
            lib.forge_oracle_quantize_i8.argtypes = [P, I64, I64, I32, P, P]
            lib.forge_oracle_quantize_i8.restype = None
            lib.forge_oracle_adamw.argtypes = [P, P, P, P, P, P, I64, I64, I32, F32, F32, F32, F32,
                                               F32, I64, I32, P, P, P, P, P]
            lib.forge_oracle_adamw.restype = None
            lib.forge_oracle_rule_step.argtypes = [P, P, P, P, I64, I64, I32, I32, F32, F32, F32, F32, F32,
                                                   F32, F32, I64, P, P, P, P]
            lib.forge_oracle_rule_step.restype = None
            lib.forge_oracle_num_threads.argtypes = []
            lib.forge_oracle_num_threads.restype = I32
            lib.forge_oracle_set_num_threads.argtypes = [I32]
            lib.forge_oracle_set_num_threads.restype = None
            _lib = lib
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    a = np.ascontiguousarray(a)
    if a.dtype != dtype:
        raise TypeError(f"expected {dtype}, got {a.dtype}")
    return a


def num_threads() -> int:
    """OpenMP threads the oracle runs with (OMP_NUM_THREADS, else all host cores)."""
    return int(_load().forge_oracle_num_threads())


def set_num_threads(n: int) -> None:
    """Threads for the oracle's parallel loops from now on (n >= 1; used by timing runs)."""
    _load().forge_oracle_set_num_threads(int(n))


# ----------------------------------------------------------------------------- rounding

def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> exact fp64 values (bf16 is the top half of an fp32)."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def f64_to_bf16_bits(x) -> np.ndarray:
    """fp64 -> bf16 bit patterns, round to nearest even in one step (the oracle's C routine)."""
    x = np.ascontiguousarray(np.asarray(x, dtype=np.float64))
    out = np.empty(x.shape, dtype=np.uint16)
    _load().forge_oracle_f64_to_bf16_array(_ptr(x), x.size, _ptr(out))
    return out


# ----------------------------------------------------------------------------- the method

def wgrad(X: np.ndarray, dY: np.ndarray) -> np.ndarray:
    """G = dY^T X in fp64 (Eq. wgrad): X bf16 bits [T, d_in], dY bf16 bits [T, d_out] -> [d_out, d_in]."""
    X, dY = _c(X, np.uint16), _c(dY, np.uint16)
    T, d_in = X.shape
    T2, d_out = dY.shape
    if T != T2:
        raise ValueError("X and dY disagree on T")
    G = np.empty((d_out, d_in), dtype=np.float64)
    _load().forge_oracle_wgrad(_ptr(X), _ptr(dY), T, d_in, d_out, _ptr(G))
    return G


def input_grad(dY: np.ndarray, W: np.ndarray) -> np.ndarray:
    """dX = dY W in fp64 (Algorithm 1, first line): dY bf16 bits [T, d_out], W bf16 bits
    [d_out, d_in] -> [T, d_in].  The layer-level backward forms it from the pre-update W."""
    dY, W = _c(dY, np.uint16), _c(W, np.uint16)
    T, d_out = dY.shape
    d_out2, d_in = W.shape
    if d_out != d_out2:
        raise ValueError("dY and W disagree on d_out")
    dX = np.empty((T, d_in), dtype=np.float64)
    _load().forge_oracle_input_grad(_ptr(dY), _ptr(W), T, d_in, d_out, _ptr(dX))
    return dX


def quantize_i8(x: np.ndarray, second_moment: bool):
    """Block-absmax int8 quantizer (App. B scheme, 256-row blocks along d_out).

    ``x`` is fp64 [d_out, d_in]; for the second moment it holds v and sqrt(v) is stored.
    Returns (codes int8 [d_out, d_in], scales fp32 [ceil(d_out/256), d_in]).
    """
    x = _c(x, np.float64)
    d_out, d_in = x.shape
    codes = np.empty((d_out, d_in), dtype=np.int8)
    scales = np.empty(((d_out + I8_BLOCK - 1) // I8_BLOCK, d_in), dtype=np.float32)
    _load().forge_oracle_quantize_i8(_ptr(x), d_in, d_out, int(second_moment), _ptr(codes), _ptr(scales))
    return codes, scales


def quantize_i8_row64(x: np.ndarray, second_moment: bool):
    """The paper's int8 layout (App. B): one scale per 64 consecutive elements of a row,
    v quantised directly (no square root), its codes floored at 1 in non-zero blocks.
    ``x`` fp64 [d_out, d_in] -> (codes int8 [d_out, d_in], scales fp32 [d_out, ceil(d_in/64)])."""
    x = _c(x, np.float64)
    d_out, d_in = x.shape
    codes = np.empty((d_out, d_in), dtype=np.int8)
    scales = np.empty((d_out, (d_in + ROW_BLOCK - 1) // ROW_BLOCK), dtype=np.float32)
    _load().forge_oracle_quantize_i8_row64(_ptr(x), d_in, d_out, int(second_moment), _ptr(codes), _ptr(scales),
                                           None)
    return codes, scales


def dequantize_i8_row64(codes: np.ndarray, scales: np.ndarray) -> np.ndarray:
    """Decode the 64-wide row-block layout: x = s * q (for v as well: v is stored directly)."""
    d_in = codes.shape[1]
    s = np.repeat(scales.astype(np.float64), ROW_BLOCK, axis=1)[:, :d_in]
    return s * codes.astype(np.float64)


def dequantize_i8(codes: np.ndarray, scales: np.ndarray, second_moment: bool) -> np.ndarray:
    """Decode int8 moments to fp64: m = s*q, v = (s*q)^2 (the stored quantity is sqrt(v))."""
    d_out = codes.shape[0]
    s = np.repeat(scales.astype(np.float64), I8_BLOCK, axis=0)[:d_out]
    x = s * codes.astype(np.float64)
    return x * x if second_moment else x


def adamw(G, W, m, v, *, moment_dtype, lr, beta1, beta2, eps, weight_decay, step,
          m_scale=None, v_scale=None, round_grad_to_bf16=False, want_quotients=False):
    """One AdamW step (Algorithm 1) on an fp64 gradient; inputs are not modified.

    W: bf16 bits [d_out, d_in].  m, v: float32 / bf16 bits / int8 codes per ``moment_dtype``.
    Returns a dict with the rounded new state (W, m, v, m_scale, v_scale), the unrounded
    fp64 values W64, m64, v64 (and the int8 quotients qm, qv when asked) and the step.
    """
    G = _c(G, np.float64)
    d_out, d_in = G.shape
    if moment_dtype == MOMENT_I8_ROW64:
        return _adamw_i8row(G, W, m, v, m_scale, v_scale, lr=lr, beta1=beta1, beta2=beta2, eps=eps,
                            weight_decay=weight_decay, step=step, want_quotients=want_quotients)
    W = _c(W, np.uint16).copy()
    mdt = {MOMENT_F32: np.float32, MOMENT_BF16: np.uint16, MOMENT_I8: np.int8}[moment_dtype]
    m, v = _c(m, mdt).copy(), _c(v, mdt).copy()
    for a in (W, m, v):
        if a.shape != (d_out, d_in):
            raise ValueError("state shape mismatch")
    if moment_dtype == MOMENT_I8:
        m_scale = _c(m_scale, np.float32).copy()
        v_scale = _c(v_scale, np.float32).copy()
    else:
        m_scale = v_scale = None
    W64, m64, v64 = (np.empty((d_out, d_in), dtype=np.float64) for _ in range(3))
    qm = qv = None
    if want_quotients and moment_dtype == MOMENT_I8:
        qm, qv = np.empty((d_out, d_in), np.float64), np.empty((d_out, d_in), np.float64)
    _load().forge_oracle_adamw(
        _ptr(G), _ptr(W), _ptr(m), _ptr(v), _ptr(m_scale), _ptr(v_scale), d_in, d_out,
        int(moment_dtype), float(lr), float(beta1), float(beta2), float(eps), float(weight_decay),
        int(step), int(bool(round_grad_to_bf16)), _ptr(W64), _ptr(m64), _ptr(v64), _ptr(qm), _ptr(qv))
    out = dict(W=W, m=m, v=v, m_scale=m_scale, v_scale=v_scale, W64=W64, m64=m64, v64=v64, step=int(step))
    if qm is not None:
        out.update(qm=qm, qv=qv)
    return out


def adamw_f64(G, W, m, v, *, lr, beta1, beta2, eps, weight_decay, step):
    """Algorithm 1 on fp64 arrays with no rounding to any storage type: the reference the
    fidelity experiment (App. E) measures weight error against.  Returns (W', m', v')."""
    f = lambda x: float(np.float32(x))            # hyper-parameters as the GPU receives them
    b1, b2, eta, ep, lam = f(beta1), f(beta2), f(lr), f(eps), f(weight_decay)
    m1 = b1 * m + (1.0 - b1) * G
    v1 = b2 * v + (1.0 - b2) * G * G
    mhat = m1 / (1.0 - b1 ** step)
    vhat = v1 / (1.0 - b2 ** step)
    W1 = (1.0 - eta * lam) * W - eta * mhat / (np.sqrt(vhat) + ep)
    return W1, m1, v1


def rule_step(G, W, s1=None, s2=None, *, opt, state_dtype, lr, beta1=0.0, beta2=0.0, eps=1e-8,
              weight_decay=0.0, lr_decay=0.0, momentum_decay=0.004, step):
    """One step of update rule ``opt`` (not AdamW) on an fp64 gradient; inputs are not modified.

    W: bf16 bits [d_out, d_in]; s1, s2: float32 or bf16-bits state per ``state_dtype`` (None
    for states the rule does not have).  Returns W, s1, s2 rounded to storage, their fp64
    values W64, s1_64, s2_64, and ``aux`` (Lion: the argument of the sign).
    """
    if opt == OPT_ADAMW:
        raise ValueError("AdamW: use adamw()")
    G = _c(G, np.float64)
    d_out, d_in = G.shape
    W = _c(W, np.uint16).copy()
    sdt = np.float32 if state_dtype == MOMENT_F32 else np.uint16
    ns = RULE_STATES[opt]
    s1 = _c(s1, sdt).copy() if ns >= 1 else None
    s2 = _c(s2, sdt).copy() if ns >= 2 else None
    W64, S1, S2, AUX = (np.zeros((d_out, d_in), np.float64) for _ in range(4))
    _load().forge_oracle_rule_step(
        _ptr(G), _ptr(W), _ptr(s1), _ptr(s2), d_in, d_out, int(opt), int(state_dtype), float(lr),
        float(beta1), float(beta2), float(eps), float(weight_decay), float(lr_decay), float(momentum_decay),
        int(step), _ptr(W64), _ptr(S1), _ptr(S2), _ptr(AUX))
    return dict(W=W, s1=s1, s2=s2, W64=W64, s1_64=S1, s2_64=S2, aux=AUX)


def _adamw_i8row(G, W, m, v, m_scale, v_scale, *, lr, beta1, beta2, eps, weight_decay, step, want_quotients):
    d_out, d_in = G.shape
    W = _c(W, np.uint16).copy()
    m, v = _c(m, np.int8).copy(), _c(v, np.int8).copy()
    m_scale, v_scale = _c(m_scale, np.float32).copy(), _c(v_scale, np.float32).copy()
    W64, m64, v64 = (np.empty((d_out, d_in), dtype=np.float64) for _ in range(3))
    qm = qv = None
    if want_quotients:
        qm, qv = np.empty((d_out, d_in), np.float64), np.empty((d_out, d_in), np.float64)
    _load().forge_oracle_adamw_i8row(_ptr(G), _ptr(W), _ptr(m), _ptr(v), _ptr(m_scale), _ptr(v_scale), d_in, d_out,
                                     float(lr), float(beta1), float(beta2), float(eps), float(weight_decay), int(step),
                                     _ptr(W64), _ptr(m64), _ptr(v64), _ptr(qm), _ptr(qv))
    out = dict(W=W, m=m, v=v, m_scale=m_scale, v_scale=v_scale, W64=W64, m64=m64, v64=v64, step=int(step))
    if qm is not None:
        out.update(qm=qm, qv=qv)
    return out


def e4m3_decode(codes: np.ndarray) -> np.ndarray:
    """E4M3 (OCP) codes -> fp64 values."""
    lib = _load()
    c = np.ascontiguousarray(codes, dtype=np.uint8)
    return np.array([lib.forge_oracle_e4m3_decode(int(x)) for x in c.reshape(-1)]).reshape(c.shape)


def e4m3_encode(x) -> np.ndarray:
    """fp32 values within [-448, 448] -> nearest E4M3 codes, ties to even."""
    x = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    out = np.empty(x.shape, dtype=np.uint8)
    _load().forge_oracle_e4m3_encode_array(_ptr(x), x.size, _ptr(out))
    return out


def adamw_fp8(G, W, m, v, *, w_fp8, m_fp8, w_ring=None, m_ring=None, v_ring=None, lr, beta1, beta2, eps,
              weight_decay, step):
    """One AdamW step with fp8 (E4M3, per-tensor delayed scale) weights and / or moments.

    W: E4M3 codes (uint8) when ``w_fp8``, else bf16 bits; m, v: E4M3 codes of m and sqrt(v)
    when ``m_fp8``, else bf16 bits; rings: fp32 [4] amax slots.  Inputs are not modified.
    Returns the new W, m, v, rings, the fp64 W64, m64, v64 and the encoded fp32 quotients
    qw, qm, qv.
    """
    G = _c(G, np.float64)
    d_out, d_in = G.shape
    W = _c(W, np.uint8 if w_fp8 else np.uint16).copy()
    m = _c(m, np.uint8 if m_fp8 else np.uint16).copy()
    v = _c(v, np.uint8 if m_fp8 else np.uint16).copy()
    rings = [_c(r, np.float32).copy() if r is not None else None for r in (w_ring, m_ring, v_ring)]
    W64, m64, v64, qw, qm, qv = (np.empty((d_out, d_in), dtype=np.float64) for _ in range(6))
    _load().forge_oracle_adamw_fp8(_ptr(G), _ptr(W), int(bool(w_fp8)), _ptr(rings[0]), _ptr(m), _ptr(v),
                                   int(bool(m_fp8)), _ptr(rings[1]), _ptr(rings[2]), d_in, d_out, float(lr),
                                   float(beta1), float(beta2), float(eps), float(weight_decay), int(step),
                                   _ptr(W64), _ptr(m64), _ptr(v64), _ptr(qw), _ptr(qm), _ptr(qv))
    return dict(W=W, m=m, v=v, w_ring=rings[0], m_ring=rings[1], v_ring=rings[2], W64=W64, m64=m64, v64=v64,
                qw=qw, qm=qm, qv=qv)


def linear_step(X, dY, W, m, v, **kw):
    """The whole fused step by definition: G = dY^T X (fp64), then ``adamw``. Also returns G."""
    G = wgrad(X, dY)
    out = adamw(G, W, m, v, **kw)
    out["G"] = G
    return out


def linear_backward(X, dY, W, m, v, **kw):
    """The layer-level backward: dX = dY W from the weight before the step (fp64, key
    ``dX``), then ``linear_step``.  Sec. 2.2 and the ordering remark of App. A."""
    dX = input_grad(dY, W)
    out = linear_step(X, dY, W, m, v, **kw)
    out["dX"] = dX
    return out
