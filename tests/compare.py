"""Tolerance checks between the HIP path and the oracle.

The bar (fused step, every config):
* W: within 1 bf16 ulp of the oracle's rounded W' on >= 99.9% of elements;
* m, v: |gpu - ora| <= 1e-3 |ora| + 1e-6 max|ora| per element.  For bf16 moments one
  ulp (2^-8 relative) is wider than 1e-3, so a neighbouring bf16 value is also accepted
  when the oracle's unrounded fp64 value lies within the kernel's own error bound of the
  midpoint between the two: there the kernel's fp32 value may legitimately round the
  other way.  The bf16 rounding of the exact value's fp32 rounding is accepted as well
  (double rounding through fp32, which any fp32 kernel that stores bf16 does).  The bound is derived from the arithmetic: the fp32 accumulation of G in any
  order errs by at most E_G = T 2^-24 (|dY|^T |X|) (the only discrepancy App. A's
  floating-point remark admits), which the moment recurrences scale by (1-beta1) and
  (1-beta2) 2|G|, plus a few fp32 roundings of the epilogue.  Every such allowance is
  counted and reported;
  At most ALLOWANCE_CAP of the elements of a tensor may use it;
* W, in addition: every element is the bf16 rounding of a value within the derived bound
  of the oracle's unrounded W' (E_G carried through the update, plus the epilogue's fp32
  roundings), so a weight that is off by one ulp for any other reason fails;
* int8 codes: equal, except +-1 where the oracle's fp32 quotient x/s lies within the
  derived bound of a half-integer (a rounding tie): the state's own window divided by the
  scale, the scales' difference, and the kernel's reciprocal product (it rounds x * RN(1/s)
  where the oracle divides, a few 2^-24 relative).  At most TIE_FLIP_CAP of the codes may
  flip.  Scales agree within the bound that the block absmax's window gives them.
"""

from __future__ import annotations

import numpy as np

U32 = 2.0 ** -24
# Largest share of a tensor's elements that may use a rounding allowance (bf16 state next
# to a midpoint, int8 codes at a tie).  The fp32 accumulation of G errs far less than its
# worst-case bound, so in practice well under 0.1 % of elements use one.
ALLOWANCE_CAP = 0.005
TIE_FLIP_CAP = 0.005
CAP_SLACK = 3          # a few uses are allowed in any tensor, however small


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


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 values -> bf16 bit patterns, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def bf16_f64(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _key_f64(k: np.ndarray) -> np.ndarray:
    """Inverse of bf16_key, as fp64 values."""
    k = k.astype(np.int64)
    b = np.where(k >= 0, k, 0x8000 | (-k)).astype(np.uint32)
    return bf16_f64(b)


def bf16_half_gap(bits: np.ndarray) -> np.ndarray:
    """Half the larger of the gaps between a bf16 value and its two neighbours: the most a
    value that rounds (to nearest) to it can differ from it."""
    k = bf16_key(bits).astype(np.int64)
    x = _key_f64(k)
    return 0.5 * np.maximum(np.abs(_key_f64(k + 1) - x), np.abs(x - _key_f64(k - 1)))


def weight_window(ora: dict, hp: dict, wm: np.ndarray, wv: np.ndarray) -> np.ndarray:
    """Per-element bound on |W'_kernel - W'| for AdamW (Algorithm 1): the errors wm, wv of the
    kernel's fp32 m', v' carried through W' = wdf W - lr/bc1 m' / (sqrt(v'/bc2) + eps), plus
    the epilogue's fp32 roundings (products, the fma, sqrt and reciprocal: 16 units of 2^-24
    of |W'| and of twice the update, which is generous)."""
    f = lambda x: float(np.float32(x))
    t = int(ora["step"])
    b1, b2, lr, eps = f(hp["beta1"]), f(hp["beta2"]), f(hp["lr"]), f(hp["eps"])
    lr_bc1 = lr / (1.0 - b1 ** t)
    isb = 1.0 / np.sqrt(1.0 - b2 ** t)
    m1 = np.abs(ora["m64"])
    rv = np.sqrt(np.maximum(ora["v64"], 0.0))
    with np.errstate(divide="ignore", invalid="ignore"):
        drv = np.where(rv > 0, np.minimum(wv / (2 * rv), np.sqrt(wv)), np.sqrt(wv))
    D = rv * isb + eps
    dD = isb * drv
    D_lo = np.maximum(D - dD, eps)
    upd = lr_bc1 * m1 / D
    dupd = lr_bc1 * (wm / D_lo + m1 * dD / (D * D_lo))
    return dupd + 16 * U32 * (np.abs(ora["W64"]) + 2 * upd)


def check_weight(W_gpu: np.ndarray, W_ora: np.ndarray, frac: float = 0.999, max_ulp=None,
                 W64: np.ndarray = None, window: np.ndarray = None):
    """W within 1 bf16 ulp of the oracle's rounded W' on >= frac of the elements, at most
    max_ulp anywhere; with the oracle's unrounded W64 and the derived window, also every
    element within half a bf16 gap of W64 plus the window (the kernel rounds a value that
    lies within the window of W64)."""
    ulps = np.abs(bf16_key(W_gpu) - bf16_key(W_ora))
    n = ulps.size
    within = int((ulps <= 1).sum())
    stats = dict(n=n, within1=within, frac_within1=within / max(n, 1), max_ulp=int(ulps.max(initial=0)),
                 exact=int((ulps == 0).sum()))
    assert within >= frac * n, f"W: only {within}/{n} within 1 ulp ({stats})"
    if max_ulp is not None:
        assert stats["max_ulp"] <= max_ulp, f"W: max ulp {stats['max_ulp']} > {max_ulp}"
    if W64 is not None:
        err = np.abs(bf16_f64(W_gpu) - W64)
        lim = bf16_half_gap(W_gpu) * (1 + 2.0 ** -20) + window
        bad = err > lim
        stats["max_err_over_limit"] = float((err / lim).max(initial=0.0))
        if bad.any():
            idx = np.argwhere(bad)[:5]
            ex = [(tuple(i), float(bf16_f64(W_gpu)[tuple(i)]), float(W64[tuple(i)]), float(window[tuple(i)]))
                  for i in idx]
            raise AssertionError(f"W: {int(bad.sum())} elements are not a rounding of a value within "
                                 f"the derived window of the oracle's W', e.g. {ex}")
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
    double_rounded = np.zeros_like(bad)
    if kind == "bf16" and bad.any():
        # the kernel stores bf16 of an fp32 value: bf16(fp32(exact)) is what exact fp32
        # arithmetic gives, and it differs from bf16(exact) where the fp32 rounding lands on a
        # bf16 midpoint (structurally common, e.g. 0.9 * m with a bf16 m at G = 0)
        double_rounded = bad & (gpu == f32_to_bf16_bits(ora64.astype(np.float32)))
        bad = bad & ~double_rounded
        kg, ko = bf16_key(gpu), bf16_key(ora)
        adjacent = np.abs(kg - ko) == 1
        mid = 0.5 * (g + o)
        win = 2.0 ** -16 * np.abs(mid) if window is None else np.maximum(window, 4 * U32 * np.abs(mid))
        near_mid = np.abs(ora64 - mid) <= win
        allowed = bad & adjacent & near_mid
    fail = bad & ~allowed
    if kind == "f32" and window is not None:
        # fp32 state is stored as computed: it must lie within the derived window of the exact
        # value (a much tighter bar than 1e-3 relative)
        fail |= np.abs(g - ora64) > window + U32 * np.abs(ora64)
    stats = dict(n=int(gpu.size), allowance_hits=int(allowed.sum()), double_rounded=int(double_rounded.sum()),
                 failures=int(fail.sum()))
    if fail.any():
        idx = np.argwhere(fail)[:5]
        ex = [(tuple(i), float(g[tuple(i)]), float(o[tuple(i)]), float(ora64[tuple(i)])) for i in idx]
        raise AssertionError(f"{name}: {int(fail.sum())} elements out of tolerance, e.g. {ex}")
    assert stats["allowance_hits"] <= ALLOWANCE_CAP * gpu.size + CAP_SLACK, \
        f"{name}: {stats['allowance_hits']} of {gpu.size} elements needed the rounding allowance"
    return stats


def half_integer_tie(quot: np.ndarray, window) -> np.ndarray:
    return np.abs(np.abs(quot - np.floor(quot)) - 0.5) <= window


# The kernel's quotient x * RN(1/s) against the oracle's fp32 x / s: the reciprocal (1 ulp),
# the product and the oracle's division (half an ulp each) -- 2^-21 relative covers them.
RECIP_REL = 2.0 ** -21


def check_codes(gpu: np.ndarray, ora: np.ndarray, quot: np.ndarray, name: str, window):
    """int8 codes: equal, or +-1 where the oracle's quotient is within `window` of a tie."""
    d = gpu.astype(np.int32) - ora.astype(np.int32)
    ties = half_integer_tie(quot, window)
    fail = (d != 0) & ~((np.abs(d) == 1) & ties)
    stats = dict(n=int(gpu.size), tie_flips=int(((d != 0) & ~fail).sum()), failures=int(fail.sum()))
    if fail.any():
        idx = np.argwhere(fail)[:5]
        ex = [(tuple(i), int(gpu[tuple(i)]), int(ora[tuple(i)]), float(quot[tuple(i)])) for i in idx]
        raise AssertionError(f"{name}: {int(fail.sum())} codes differ beyond ties, e.g. {ex}")
    assert stats["tie_flips"] <= TIE_FLIP_CAP * gpu.size + CAP_SLACK, \
        f"{name}: {stats['tie_flips']} of {gpu.size} codes flipped at ties"
    return stats


def check_scales(gpu: np.ndarray, ora: np.ndarray, name: str, window: np.ndarray = None, rtol: float = 1e-5):
    """Scales within `window` (absolute, per scale) of the oracle's, else within rtol."""
    g, o = gpu.astype(np.float64), ora.astype(np.float64)
    lim = rtol * np.abs(o) if window is None else window
    bad = np.abs(g - o) > lim
    assert not bad.any(), f"{name}: {int(bad.sum())} scales differ by more than their bound"
    return dict(n=int(gpu.size), max_rel=float((np.abs(g - o) / np.maximum(np.abs(o), 1e-300)).max(initial=0)))


def _block_max_col256(x: np.ndarray) -> np.ndarray:
    """Max over 256-row blocks of each column: [ceil(d_out/256), d_in]."""
    d_out, d_in = x.shape
    nb = (d_out + 255) // 256
    pad = np.full((nb * 256, d_in), -np.inf)
    pad[:d_out] = x
    return pad.reshape(nb, 256, d_in).max(axis=1)


def _block_max_row64(x: np.ndarray) -> np.ndarray:
    """Max over 64-wide blocks of each row: [d_out, ceil(d_in/64)]."""
    d_out, d_in = x.shape
    nb = (d_in + 63) // 64
    pad = np.full((d_out, nb * 64), -np.inf)
    pad[:, :d_in] = x
    return pad.reshape(d_out, nb, 64).max(axis=2)


def _per_row_scale(scale: np.ndarray, d_out: int) -> np.ndarray:
    return np.repeat(scale.astype(np.float64), 256, axis=0)[:d_out]


def _per_col_scale(scale: np.ndarray, d_in: int) -> np.ndarray:
    return np.repeat(scale.astype(np.float64), 64, axis=1)[:, :d_in]


def _int8_checks(gpu: dict, ora: dict, layout: str, wm, wv) -> dict:
    """Codes and scales of both int8 moments against the oracle with derived windows."""
    out = {}
    if layout == "col256":
        d_out = gpu["m"].shape[0]
        expand = lambda s: _per_row_scale(s, d_out)
        block_max = _block_max_col256
        # sqrt(v') is stored: it moves by at most wv / (2 sqrt(v')) (or sqrt(wv)) when v' moves by wv
        root = np.sqrt(np.maximum(ora["v64"], 0.0))
        with np.errstate(divide="ignore", invalid="ignore"):
            wr = np.where(root > 0, np.minimum(wv / (2 * root), np.sqrt(wv)), np.sqrt(wv))
        stored = {"m": (np.abs(ora["m64"]), wm), "v": (root, wr)}
    else:
        d_in = gpu["m"].shape[1]
        expand = lambda s: _per_col_scale(s, d_in)
        block_max = _block_max_row64
        stored = {"m": (np.abs(ora["m64"]), wm), "v": (np.abs(ora["v64"]), wv)}   # v itself is stored
    for k in ("m", "v"):
        val, w = stored[k]
        so, sg = ora[f"{k}_scale"].astype(np.float64), gpu[f"{k}_scale"].astype(np.float64)
        swin = block_max(w + U32 * val) / 127.0 + 2 * U32 * np.abs(so)
        out[f"{k}_scale"] = check_scales(gpu[f"{k}_scale"], ora[f"{k}_scale"], f"{k} scales", window=swin)
        s_e, sg_e = expand(so), expand(sg)
        quot = ora[f"q{k}"]
        with np.errstate(divide="ignore", invalid="ignore"):
            qwin = np.where(s_e > 0, w / s_e + np.abs(quot) * (RECIP_REL + np.abs(sg_e - s_e) / s_e), 0.0)
        out[k] = check_codes(gpu[k], ora[k], quot, f"{k} codes", qwin)
    return out


def check_step(gpu: dict, ora: dict, moment: str, w_frac: float = 0.999, hp: dict = None):
    """Compare a whole AdamW step: dicts with W, m, v (and m_scale, v_scale) as numpy arrays.

    With `hp` (hyper-parameters) and the oracle's gradient G and its fp32 error bound EG
    in `ora`, the rounding allowances use the derived error bounds and W is held to its
    derived window; without them W must stay within 2 ulp everywhere.
    """
    wm, wv = moment_windows(ora, hp) if hp is not None else (None, None)
    if wm is not None and "step" in ora:
        # the window is the stricter bar; it also admits the elements whose W' cancels to a
        # small value, where the fp32 roundings of the two terms span several bf16 ulps of it
        out = {"W": check_weight(gpu["W"], ora["W"], frac=w_frac, W64=ora["W64"],
                                 window=weight_window(ora, hp, wm, wv))}
    else:
        out = {"W": check_weight(gpu["W"], ora["W"], frac=w_frac, max_ulp=2)}
    if moment in ("i8", "i8r64"):
        if wm is None:
            raise ValueError("int8 state is compared with derived windows: pass hp and the oracle's EG")
        out.update(_int8_checks(gpu, ora, "col256" if moment == "i8" else "row64", wm, wv))
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


def rule_weight_window(ora: dict, W64: np.ndarray, W_at) -> np.ndarray:
    """Per-element bound on |W'_kernel - W'| for an update rule: the kernel's G lies within
    E_G of the exact G, so its W' lies between the oracle's W' at G - E_G and at G + E_G
    (`W_at(sign)` returns those) -- doubled as a margin for curvature over that short
    interval -- plus the epilogue's fp32 roundings (16 units of 2^-24 of |W'| and of twice
    the update |W - W'|)."""
    lo, hi = W_at(-1), W_at(+1)
    sens = 2 * np.maximum(np.abs(hi - ora["W64"]), np.abs(lo - ora["W64"]))
    return sens + 16 * U32 * (np.abs(ora["W64"]) + 2 * np.abs(W64 - ora["W64"]))


def check_rule_step(gpu: dict, ora: dict, opt: int, kind: str, hp: dict, G, EG, W64, s1_in, s2_in,
                    w_frac: float = 0.999, W_at=None):
    """W within 1 bf16 ulp on >= w_frac of the elements and, with `W_at` (the oracle's W' at
    G -+ E_G), every element within half a bf16 gap plus rule_weight_window of the oracle's
    unrounded W' (Lion: outside its sign ties, where W must match one of the sign
    alternatives); states as check_moment with rule_windows."""
    import oracle as o
    out = {}
    win = rule_weight_window(ora, W64, W_at) if W_at is not None else None
    if opt == o.OPT_MUON:
        assert np.array_equal(gpu["W"], ora["W"]), "W changed under the momentum accumulate"
    elif opt == o.OPT_LION:
        amb = lion_ambiguous(ora, hp, G, EG, s1_in)
        if win is None:
            out["W"] = check_weight(gpu["W"][~amb], ora["W"][~amb], frac=w_frac, max_ulp=2)
        else:
            out["W"] = check_weight(gpu["W"][~amb], ora["W"][~amb], frac=w_frac, W64=ora["W64"][~amb],
                                    window=win[~amb])
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
    elif win is None:
        out["W"] = check_weight(gpu["W"], ora["W"], frac=w_frac, max_ulp=2)
    else:
        out["W"] = check_weight(gpu["W"], ora["W"], frac=w_frac, W64=ora["W64"], window=win)
    w1, w2 = rule_windows(opt, ora, hp, G, EG, W64, s1_in, s2_in)
    ns = o.RULE_STATES[opt]
    if ns >= 1:
        out["s1"] = check_moment(gpu["s1"], ora["s1"], ora["s1_64"], kind, "s1", w1)
    if ns >= 2:
        out["s2"] = check_moment(gpu["s2"], ora["s2"], ora["s2_64"], kind, "s2", w2)
    return out
