"""Tolerance checks between the HIP path and the oracle.

The bar (fused step, every config):
* W: within 1 bf16 ulp of the oracle's rounded W' on >= 99.9% of elements;
* m, v: |gpu - ora| <= 1e-3 |ora| + 1e-6 max|ora| per element.  For bf16 moments one
  ulp (2^-8 relative) is wider than 1e-3, so a neighbouring bf16 value is also accepted
  when the oracle's unrounded fp64 value lies within the kernel's own error bound of the
  midpoint between the two: there the kernel's fp32 value may legitimately round the
  other way.  The bound is derived from the arithmetic: the fp32 accumulation of G in any
  order errs by at most E_G = T 2^-24 (|dY|^T |X|) (the only discrepancy App. A's
  floating-point remark admits), which the moment recurrences scale by (1-beta1) and
  (1-beta2) 2|G|, plus a few fp32 roundings of the epilogue.  Every such allowance is
  counted and reported;
* int8 codes: equal, except +-1 where the oracle's fp32 quotient x/s lies within
  max(1e-3, error bound of x / s) of a half-integer (a rounding tie); scales within 1e-5
  relative.
"""

from __future__ import annotations

import numpy as np

U32 = 2.0 ** -24


def moment_windows(ora: dict, hp: dict):
    """Per-element absolute error bounds of the kernel's fp32 m' and v' (see module doc)."""
    if "EG" not in ora:
        return None, None
    G, EG = ora["G"], ora["EG"]
    c1 = 1.0 - float(np.float32(hp["beta1"]))
    c2 = 1.0 - float(np.float32(hp["beta2"]))
    wm = c1 * EG + 4 * U32 * (2 * np.abs(ora["m64"]) + 2 * c1 * np.abs(G))
    wv = c2 * (2 * np.abs(G) * EG + EG * EG) + 4 * U32 * (2 * np.abs(ora["v64"]) + 2 * c2 * G * G)
    return wm, wv


def bf16_key(bits: np.ndarray) -> np.ndarray:
    """Monotone integer key of bf16 bit patterns (adjacent values differ by 1; +0 == -0)."""
    b = bits.astype(np.int32)
    return np.where(b & 0x8000, -(b & 0x7FFF), b)


def bf16_f64(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def check_weight(W_gpu: np.ndarray, W_ora: np.ndarray, frac: float = 0.999, max_ulp=None):
    ulps = np.abs(bf16_key(W_gpu) - bf16_key(W_ora))
    n = ulps.size
    within = int((ulps <= 1).sum())
    stats = dict(n=n, within1=within, frac_within1=within / max(n, 1), max_ulp=int(ulps.max(initial=0)),
                 exact=int((ulps == 0).sum()))
    assert within >= frac * n, f"W: only {within}/{n} within 1 ulp ({stats})"
    if max_ulp is not None:
        assert stats["max_ulp"] <= max_ulp, f"W: max ulp {stats['max_ulp']} > {max_ulp}"
    return stats


def check_moment(gpu: np.ndarray, ora: np.ndarray, ora64: np.ndarray, kind: str, name: str,
                 window=None):
    """kind 'f32' (float arrays) or 'bf16' (bit patterns); `window`: the kernel's error bound."""
    if kind == "bf16":
        g, o = bf16_f64(gpu), bf16_f64(ora)
    else:
        g, o = gpu.astype(np.float64), ora.astype(np.float64)
    tol = 1e-3 * np.abs(o) + 1e-6 * np.abs(o).max(initial=0.0)
    bad = np.abs(g - o) > tol
    allowed = np.zeros_like(bad)
    if kind == "bf16" and bad.any():
        kg, ko = bf16_key(gpu), bf16_key(ora)
        adjacent = np.abs(kg - ko) == 1
        mid = 0.5 * (g + o)
        win = 2.0 ** -16 * np.abs(mid) if window is None else np.maximum(window, 4 * U32 * np.abs(mid))
        near_mid = np.abs(ora64 - mid) <= win
        allowed = bad & adjacent & near_mid
    fail = bad & ~allowed
    stats = dict(n=int(gpu.size), allowance_hits=int(allowed.sum()), failures=int(fail.sum()))
    if fail.any():
        idx = np.argwhere(fail)[:5]
        ex = [(tuple(i), float(g[tuple(i)]), float(o[tuple(i)]), float(ora64[tuple(i)])) for i in idx]
        raise AssertionError(f"{name}: {int(fail.sum())} elements out of tolerance, e.g. {ex}")
    return stats


def half_integer_tie(quot: np.ndarray, window=1e-3) -> np.ndarray:
    return np.abs(np.abs(quot - np.floor(quot)) - 0.5) <= window


def check_codes(gpu: np.ndarray, ora: np.ndarray, quot: np.ndarray, name: str, window=None):
    d = gpu.astype(np.int32) - ora.astype(np.int32)
    ties = half_integer_tie(quot, 1e-3 if window is None else np.maximum(1e-3, window))
    fail = (d != 0) & ~((np.abs(d) == 1) & ties)
    stats = dict(n=int(gpu.size), tie_flips=int(((d != 0) & ~fail).sum()), failures=int(fail.sum()))
    if fail.any():
        idx = np.argwhere(fail)[:5]
        ex = [(tuple(i), int(gpu[tuple(i)]), int(ora[tuple(i)]), float(quot[tuple(i)])) for i in idx]
        raise AssertionError(f"{name}: {int(fail.sum())} codes differ beyond ties, e.g. {ex}")
    return stats


def check_scales(gpu: np.ndarray, ora: np.ndarray, name: str, rtol: float = 1e-5):
    g, o = gpu.astype(np.float64), ora.astype(np.float64)
    bad = np.abs(g - o) > rtol * np.abs(o)
    assert not bad.any(), f"{name}: {int(bad.sum())} scales differ by more than {rtol} relative"
    return dict(n=int(gpu.size), max_rel=float((np.abs(g - o) / np.maximum(np.abs(o), 1e-300)).max(initial=0)))


def _per_row_scale(scale: np.ndarray, d_out: int) -> np.ndarray:
    return np.repeat(scale.astype(np.float64), 256, axis=0)[:d_out]


def check_step(gpu: dict, ora: dict, moment: str, w_frac: float = 0.999, hp: dict = None):
    """Compare a whole step: dicts with W, m, v (and m_scale, v_scale) as numpy arrays.

    With `hp` (hyper-parameters) and the oracle's gradient G and its fp32 error bound EG
    in `ora`, the rounding-boundary allowances use the derived error bounds.
    """
    out = {"W": check_weight(gpu["W"], ora["W"], frac=w_frac)}
    wm, wv = moment_windows(ora, hp) if hp is not None else (None, None)
    if moment == "i8":
        qwm = qwv = None
        if wm is not None:
            d_out = gpu["m"].shape[0]
            sm = _per_row_scale(ora["m_scale"], d_out)
            sv = _per_row_scale(ora["v_scale"], d_out)
            with np.errstate(divide="ignore", invalid="ignore"):
                # sqrt(v') moves by at most wv / (2 sqrt(v')) when v' moves by wv
                root = np.sqrt(np.maximum(ora["v64"], 1e-300))
                qwm = np.where(sm > 0, wm / sm, 0.0)
                qwv = np.where(sv > 0, np.minimum(wv / (2 * root), np.sqrt(wv)) / sv, 0.0)
        out["m"] = check_codes(gpu["m"], ora["m"], ora["qm"], "m codes", qwm)
        out["v"] = check_codes(gpu["v"], ora["v"], ora["qv"], "v codes", qwv)
        out["m_scale"] = check_scales(gpu["m_scale"], ora["m_scale"], "m scales")
        out["v_scale"] = check_scales(gpu["v_scale"], ora["v_scale"], "v scales")
    elif moment == "i8r64":
        qwm = qwv = None
        if wm is not None:
            d_in = gpu["m"].shape[1]
            sm = np.repeat(ora["m_scale"].astype(np.float64), 64, axis=1)[:, :d_in]
            sv = np.repeat(ora["v_scale"].astype(np.float64), 64, axis=1)[:, :d_in]
            with np.errstate(divide="ignore", invalid="ignore"):
                qwm = np.where(sm > 0, wm / sm, 0.0)
                qwv = np.where(sv > 0, wv / sv, 0.0)        # v itself is quantised
        out["m"] = check_codes(gpu["m"], ora["m"], ora["qm"], "m codes", qwm)
        out["v"] = check_codes(gpu["v"], ora["v"], ora["qv"], "v codes", qwv)
        out["m_scale"] = check_scales(gpu["m_scale"], ora["m_scale"], "m scales")
        out["v_scale"] = check_scales(gpu["v_scale"], ora["v_scale"], "v scales")
    else:
        out["m"] = check_moment(gpu["m"], ora["m"], ora["m64"], moment, "m", wm)
        out["v"] = check_moment(gpu["v"], ora["v"], ora["v64"], moment, "v", wv)
    return out


# ----------------------------------------------------------------------------- other update rules

def rule_windows(opt: int, ora: dict, hp: dict, G: np.ndarray, EG: np.ndarray, W64: np.ndarray,
                 s1: np.ndarray, s2: np.ndarray):
    """Per-element bounds on the kernel's fp32 states of update rule `opt` (codes of the
    oracle), as for AdamW: the gradient's accumulation error E_G carried through the rule's
    recurrence, plus a few fp32 roundings of the terms (see moment_windows)."""
    import oracle as o
    f = lambda x: float(np.float32(x))
    b1, b2, wd = f(hp.get("beta1", 0)), f(hp.get("beta2", 0)), f(hp.get("weight_decay", 0))
    gg = G + wd * W64
    a, b = (np.abs(x) if x is not None else 0.0 for x in (s1, s2))
    E = EG
    sq = 2 * np.abs(gg) * E + E * E
    if opt in (o.OPT_SGD_MOMENTUM,):
        return E + 4 * U32 * (b1 * a + 2 * np.abs(gg) + np.abs(wd * W64)), None
    if opt == o.OPT_ADAGRAD:
        return sq + 4 * U32 * (a + 2 * gg * gg), None
    if opt == o.OPT_RMSPROP:
        return (1 - b2) * sq + 4 * U32 * (b2 * a + 2 * (1 - b2) * gg * gg), None
    if opt == o.OPT_LION:
        return (1 - b2) * E + 4 * U32 * (b2 * a + 2 * (1 - b2) * np.abs(G)), None
    if opt == o.OPT_MUON:
        return E + 4 * U32 * (b1 * a + 2 * np.abs(G)), None
    if opt in (o.OPT_NADAM, o.OPT_RADAM, o.OPT_ADAMAX):
        w1 = (1 - b1) * E + 4 * U32 * (b1 * a + 2 * (1 - b1) * np.abs(gg) + np.abs(wd * W64))
        if opt == o.OPT_ADAMAX:
            w2 = E + 4 * U32 * (b2 * b + np.abs(gg) + f(hp.get("eps", 0)))
        else:
            w2 = (1 - b2) * sq + 4 * U32 * (b2 * b + 2 * (1 - b2) * gg * gg)
        return w1, w2
    return None, None


def lion_ambiguous(ora: dict, hp: dict, G: np.ndarray, EG: np.ndarray, s1: np.ndarray) -> np.ndarray:
    """Elements whose Lion sign argument c lies within its error bound of zero: there the
    kernel's fp32 c may take the other sign, and W may differ by up to 2 lr."""
    b1 = float(np.float32(hp["beta1"]))
    win = (1 - b1) * EG + 4 * U32 * (b1 * np.abs(s1) + 2 * (1 - b1) * np.abs(G))
    return np.abs(ora["aux"]) <= win


def check_rule_step(gpu: dict, ora: dict, opt: int, kind: str, hp: dict, G, EG, W64, s1_in, s2_in,
                    w_frac: float = 0.999):
    """W within 1 bf16 ulp on >= w_frac of the elements (Lion: outside its sign ties, where W
    must match one of the sign alternatives); states as check_moment with rule_windows."""
    import oracle as o
    out = {}
    if opt == o.OPT_MUON:
        assert np.array_equal(gpu["W"], ora["W"]), "W changed under the momentum accumulate"
    elif opt == o.OPT_LION:
        amb = lion_ambiguous(ora, hp, G, EG, s1_in)
        out["W"] = check_weight(gpu["W"][~amb], ora["W"][~amb], frac=w_frac)
        if amb.any():
            lr, wd = float(np.float32(hp["lr"])), float(np.float32(hp["weight_decay"]))
            base = W64[amb] * (1 - lr * wd)
            keys = [bf16_key(o.f64_to_bf16_bits(base + d)) for d in (-lr, 0.0, lr)]
            kg = bf16_key(gpu["W"][amb])
            ok = np.zeros(kg.shape, bool)
            for k in keys:
                ok |= np.abs(kg - k) <= 1
            assert ok.all(), f"W: {int((~ok).sum())} sign-tie elements match no sign alternative"
        out["lion_sign_ties"] = int(amb.sum())
    else:
        out["W"] = check_weight(gpu["W"], ora["W"], frac=w_frac)
    w1, w2 = rule_windows(opt, ora, hp, G, EG, W64, s1_in, s2_in)
    ns = o.RULE_STATES[opt]
    if ns >= 1:
        out["s1"] = check_moment(gpu["s1"], ora["s1"], ora["s1_64"], kind, "s1", w1)
    if ns >= 2:
        out["s2"] = check_moment(gpu["s2"], ora["s2"], ora["s2_64"], kind, "s2", w2)
    return out
