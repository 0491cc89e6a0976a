"""Pins for the CPU oracle: each checks it against something other than itself.

Kinds of pin used here (a plausible mistake in the oracle -- a dropped term, a wrong
sign, a transposed operand, a wrong bias correction -- fails at least one):

* exact rational brute force of G = dY^T X and of dX = dY W on tiny non-square shapes;
* dX is the adjoint of the forward Y = X W^T, and <dX, X> = <G, W> ties it to G;
* the rank-one closed form of G;
* Prop. 1 (App. A): summing the oracle's G over any partition of the token axis gives G;
* closed forms of Algorithm 1's update (step 1 from zero state; zero gradient; beta = 0;
  lr = 0);
* torch.optim.AdamW in fp64 as an independent library implementation of the update;
* bf16 round-to-nearest-even against torch's fp32 -> bf16 cast and against brute force;
* the int8 block-absmax quantizer's invariants and App. B's accumulated-error bound.
"""
from fractions import Fraction
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import MOMENT_BF16, MOMENT_F32, MOMENT_I8

HP = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.1)


def f32(x):
    """The fp64 value of an fp32 hyper-parameter, as the oracle promotes it."""
    return float(np.float32(x))


def bf16_rand(shape, std, seed):
    g = torch.Generator().manual_seed(seed)
    t = (torch.randn(shape, generator=g) * std).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def to_bits(values):
    """Exact small values -> bf16 bit patterns (asserts exactness)."""
    t = torch.tensor(values, dtype=torch.float64)
    b = t.to(torch.float32).to(torch.bfloat16)
    assert torch.equal(b.to(torch.float64), t), "value not exactly representable in bf16"
    return b.view(torch.int16).numpy().view(np.uint16).copy()


# ------------------------------------------------------------------------- bf16 rounding

def test_bf16_rne_matches_torch_on_fp32_values():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.standard_normal(20000).astype(np.float32) * np.float32(10.0) ** rng.integers(-30, 30, 20000).astype(np.float32),
        # exact ties between neighbouring bf16 values: low 16 bits == 0x8000
        (rng.integers(0x00800000, 0x7F000000, 2000, dtype=np.uint32) & 0xFFFF0000 | 0x8000).view(np.float32),
        np.array([0x3F808000, 0x3F818000, 0xBF808000, 0x00008000, 0x7F7F8000], dtype=np.uint32).view(np.float32),
    ]).astype(np.float32)
    x = x[np.isfinite(x)]
    want = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = oracle.f64_to_bf16_bits(x.astype(np.float64))
    assert np.array_equal(got, want)
    # hand-made ties round to even
    assert oracle.f64_to_bf16_bits(np.array([1.0 + 2 ** -8]))[0] == 0x3F80
    assert oracle.f64_to_bf16_bits(np.array([1.0 + 3 * 2 ** -8]))[0] == 0x3F82


def test_bf16_rne_is_nearest_on_doubles():
    """Direct fp64 -> bf16: brute force over the two neighbouring bf16 values."""
    rng = np.random.default_rng(1)
    x = rng.standard_normal(3000) * 10.0 ** rng.integers(-20, 20, 3000)
    got = oracle.f64_to_bf16_bits(x)
    for xi, hi in zip(x, got):
        r = oracle.bf16_bits_to_f64(np.array([hi]))[0]
        # neighbours of r in bf16 (same sign): r +- one ulp
        up = oracle.bf16_bits_to_f64(np.array([hi + 1]))[0]
        dn = oracle.bf16_bits_to_f64(np.array([hi - 1]))[0]
        err = abs(xi - r)
        assert err <= abs(xi - up) and err <= abs(xi - dn)
        if err == abs(xi - up) or err == abs(xi - dn):      # a tie: result must be even
            assert hi % 2 == 0


# ------------------------------------------------------------------------- weight gradient

def test_wgrad_exact_rationals_nonsquare():
    T, d_in, d_out = 7, 5, 3
    X = bf16_rand((T, d_in), 1.0, 11)
    dY = bf16_rand((T, d_out), 0.01, 12)
    G = oracle.wgrad(X, dY)
    assert G.shape == (d_out, d_in)
    Xf = oracle.bf16_bits_to_f64(X)
    Yf = oracle.bf16_bits_to_f64(dY)
    for p in range(d_out):
        for q in range(d_in):
            exact = sum(Fraction(Yf[t, p]) * Fraction(Xf[t, q]) for t in range(T))
            bound = T * 2.0 ** -53 * sum(abs(Yf[t, p] * Xf[t, q]) for t in range(T))
            assert abs(G[p, q] - float(exact)) <= bound


def test_wgrad_integer_values_exact():
    """Small integers: every partial sum is exact in fp64, so G must equal the rational sum."""
    rng = np.random.default_rng(2)
    T, d_in, d_out = 9, 6, 4
    Xv = rng.integers(-8, 9, (T, d_in))
    Yv = rng.integers(-8, 9, (T, d_out))
    G = oracle.wgrad(to_bits(Xv.tolist()), to_bits(Yv.tolist()))
    want = Yv.T @ Xv                                   # [d_out, d_in], integer matmul
    assert np.array_equal(G, want.astype(np.float64))


def test_wgrad_rank_one_closed_form():
    """X[t,q] = a_t b_q, dY[t,p] = c_t d_p  =>  G[p,q] = (sum_t c_t a_t) d_p b_q."""
    a = np.array([1, -2, 0.5, 3, -1.5, 0.25])
    b = np.array([2, -1, 0.5, 4])
    c = np.array([0.5, 1, -1, 2, 0.75, -4])
    d = np.array([-1, 2, 0.25])
    G = oracle.wgrad(to_bits(np.outer(a, b).tolist()), to_bits(np.outer(c, d).tolist()))
    want = np.dot(c, a) * np.outer(d, b)
    assert np.array_equal(G, want)


@pytest.mark.parametrize("chunk", [1, 7, 64, 200])
def test_wgrad_token_partition_invariance(chunk):
    """Prop. 1: accumulating over any partition of the token axis gives G (fp64 rounding aside)."""
    T, d_in, d_out = 200, 24, 16
    X = bf16_rand((T, d_in), 1.0, 21)
    dY = bf16_rand((T, d_out), 0.01, 22)
    G = oracle.wgrad(X, dY)
    acc = np.zeros_like(G)
    for t0 in range(0, T, chunk):
        acc += oracle.wgrad(X[t0:t0 + chunk], dY[t0:t0 + chunk])
    # bound on fp64 rounding: |dY|^T |X| (a numpy product, used only as an error scale)
    scale = np.abs(oracle.bf16_bits_to_f64(dY)).T @ np.abs(oracle.bf16_bits_to_f64(X))
    assert np.all(np.abs(acc - G) <= 4 * T * 2.0 ** -53 * scale)


def test_wgrad_empty_token_axis():
    G = oracle.wgrad(np.zeros((0, 8), np.uint16), np.zeros((0, 3), np.uint16))
    assert G.shape == (3, 8) and not G.any()


# ------------------------------------------------------------------------- input gradient

def test_input_grad_exact_rationals_nonsquare():
    T, d_in, d_out = 6, 3, 5
    dY = bf16_rand((T, d_out), 0.01, 31)
    W = bf16_rand((d_out, d_in), 0.02, 32)
    dX = oracle.input_grad(dY, W)
    assert dX.shape == (T, d_in)
    Yf, Wf = oracle.bf16_bits_to_f64(dY), oracle.bf16_bits_to_f64(W)
    for t in range(T):
        for q in range(d_in):
            exact = sum(Fraction(Yf[t, p]) * Fraction(Wf[p, q]) for p in range(d_out))
            bound = d_out * 2.0 ** -53 * sum(abs(Yf[t, p] * Wf[p, q]) for p in range(d_out))
            assert abs(dX[t, q] - float(exact)) <= bound


def test_input_grad_integer_values_exact():
    rng = np.random.default_rng(3)
    T, d_in, d_out = 5, 7, 4
    Yv = rng.integers(-8, 9, (T, d_out))
    Wv = rng.integers(-8, 9, (d_out, d_in))
    dX = oracle.input_grad(to_bits(Yv.tolist()), to_bits(Wv.tolist()))
    assert np.array_equal(dX, (Yv @ Wv).astype(np.float64))


def test_input_grad_identity_weight_returns_dy():
    d = 8
    dY = bf16_rand((5, d), 1.0, 33)
    dX = oracle.input_grad(dY, to_bits(np.eye(d).tolist()))
    assert np.array_equal(dX, oracle.bf16_bits_to_f64(dY))


def test_input_grad_is_adjoint_of_forward():
    """<dX, X> = <dY, Y> for the forward Y = X W^T (Eq. fwd), for any X: the backward is
    the transpose of the forward map.  Square d_in = d_out with a non-symmetric W, so a
    transposed weight fails too."""
    T, d = 9, 12
    X = oracle.bf16_bits_to_f64(bf16_rand((T, d), 1.0, 34))
    W = bf16_rand((d, d), 0.02, 35)
    dY = bf16_rand((T, d), 0.01, 36)
    Wf, Yf = oracle.bf16_bits_to_f64(W), oracle.bf16_bits_to_f64(dY)
    assert not np.allclose(Wf, Wf.T)
    Y = np.array([[sum(X[t, q] * Wf[p, q] for q in range(d)) for p in range(d)] for t in range(T)])
    lhs = float(np.sum(oracle.input_grad(dY, W) * X))
    rhs = float(np.sum(Yf * Y))
    assert abs(lhs - rhs) <= 1e-12 * (np.abs(Yf) @ np.abs(Wf) * np.abs(X)).sum()


def test_input_grad_consistent_with_weight_gradient():
    """<dX, X> = <G, W> with G = dY^T X: both equal sum_{t,p,q} dY[t,p] W[p,q] X[t,q].
    Ties the input gradient to the separately pinned weight gradient."""
    T, d_in, d_out = 11, 16, 24
    X = bf16_rand((T, d_in), 1.0, 37)
    dY = bf16_rand((T, d_out), 0.01, 38)
    W = bf16_rand((d_out, d_in), 0.02, 39)
    Xf, Wf = oracle.bf16_bits_to_f64(X), oracle.bf16_bits_to_f64(W)
    a = float(np.sum(oracle.input_grad(dY, W) * Xf))
    b = float(np.sum(oracle.wgrad(X, dY) * Wf))
    scale = float((np.abs(oracle.bf16_bits_to_f64(dY)) @ np.abs(Wf) * np.abs(Xf)).sum())
    assert abs(a - b) <= 1e-12 * scale


def test_input_grad_empty_axes():
    assert not oracle.input_grad(np.zeros((4, 0), np.uint16), np.zeros((0, 8), np.uint16)).any()
    assert oracle.input_grad(np.zeros((4, 0), np.uint16), np.zeros((0, 8), np.uint16)).shape == (4, 8)
    assert oracle.input_grad(np.zeros((0, 8), np.uint16), np.zeros((8, 16), np.uint16)).shape == (0, 16)


def test_linear_backward_reads_pre_update_weight():
    """The ordering remark of App. A: dX comes from W before the step, not after it."""
    T, d_in, d_out = 16, 24, 8
    X = bf16_rand((T, d_in), 1.0, 40)
    dY = bf16_rand((T, d_out), 0.01, 41)
    W = bf16_rand((d_out, d_in), 0.02, 42)
    z = np.zeros((d_out, d_in), np.float32)
    out = oracle.linear_backward(X, dY, W, z, z, moment_dtype=MOMENT_F32, step=1, **HP)
    assert np.array_equal(out["dX"], oracle.input_grad(dY, W))
    assert not np.array_equal(out["dX"], oracle.input_grad(dY, out["W"]))


# ------------------------------------------------------------------------- AdamW update

def _state(d_out, d_in, dtype, seed, warm):
    if not warm:
        z = np.zeros((d_out, d_in), np.float32 if dtype == MOMENT_F32 else np.uint16)
        return z, z.copy()
    g = torch.Generator().manual_seed(seed)
    m = torch.randn((d_out, d_in), generator=g) * 1e-4
    v = (torch.randn((d_out, d_in), generator=g) * 1e-6).abs()
    if dtype == MOMENT_F32:
        return m.numpy().copy(), v.numpy().copy()
    return (m.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16).copy(),
            v.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16).copy())


def _decode(a, dtype):
    return a.astype(np.float64) if dtype == MOMENT_F32 else oracle.bf16_bits_to_f64(a)


@pytest.mark.parametrize("dtype", [MOMENT_F32, MOMENT_BF16])
def test_step1_from_zero_state_closed_form(dtype):
    """t=1, m=v=0: m'=(1-b1)g, v'=(1-b2)g^2, mhat=g, vhat=g^2, W'=(1-lr*wd)W - lr*g/(|g|+eps)."""
    rng = np.random.default_rng(3)
    G = rng.standard_normal((16, 40)) * 0.1
    W = bf16_rand((16, 40), 0.02, 31)
    m, v = _state(16, 40, dtype, 0, warm=False)
    out = oracle.adamw(G, W, m, v, moment_dtype=dtype, step=1, **HP)
    b1, b2, lr, wd, eps = f32(0.9), f32(0.999), f32(1e-3), f32(0.1), f32(1e-8)
    W0 = oracle.bf16_bits_to_f64(W)
    np.testing.assert_allclose(out["m64"], (1 - b1) * G, rtol=1e-15, atol=0)
    np.testing.assert_allclose(out["v64"], (1 - b2) * G * G, rtol=1e-15, atol=0)
    np.testing.assert_allclose(out["W64"], (1 - lr * wd) * W0 - lr * G / (np.abs(G) + eps),
                               rtol=1e-14, atol=1e-18)
    # the update is ~ -lr*sign(g): W moves opposite to the gradient
    assert np.all(np.sign((1 - lr * wd) * W0 - out["W64"]) == np.sign(G))
    assert np.array_equal(out["W"], oracle.f64_to_bf16_bits(out["W64"]))


def test_zero_gradient_cold_state_is_pure_decay():
    W = bf16_rand((8, 24), 0.02, 41)
    z = np.zeros((8, 24), np.float32)
    hp = dict(HP, lr=0.5, weight_decay=0.1)            # lr*wd = 0.05: visible after bf16 rounding
    out = oracle.adamw(np.zeros((8, 24)), W, z, z, moment_dtype=MOMENT_F32, step=7, **hp)
    W0 = oracle.bf16_bits_to_f64(W)
    assert np.array_equal(out["W64"], (1 - f32(0.5) * f32(0.1)) * W0)
    assert not out["m64"].any() and not out["v64"].any()
    assert np.array_equal(out["W"], oracle.f64_to_bf16_bits((1 - f32(0.5) * f32(0.1)) * W0))
    assert not np.array_equal(out["W"], W)


def test_zero_gradient_warm_state_closed_form():
    W = bf16_rand((8, 24), 0.02, 42)
    m, v = _state(8, 24, MOMENT_F32, 5, warm=True)
    t = 100
    out = oracle.adamw(np.zeros((8, 24)), W, m, v, moment_dtype=MOMENT_F32, step=t, **HP)
    b1, b2 = f32(0.9), f32(0.999)
    m0, v0 = m.astype(np.float64), v.astype(np.float64)
    np.testing.assert_allclose(out["m64"], b1 * m0, rtol=1e-15)
    np.testing.assert_allclose(out["v64"], b2 * v0, rtol=1e-15)
    want = ((1 - f32(1e-3) * f32(0.1)) * oracle.bf16_bits_to_f64(W)
            - f32(1e-3) * (b1 * m0 / (1 - b1 ** t)) / (np.sqrt(b2 * v0 / (1 - b2 ** t)) + f32(1e-8)))
    np.testing.assert_allclose(out["W64"], want, rtol=1e-13, atol=1e-18)


def test_beta_zero_is_normalised_gradient_step():
    """b1 = b2 = 0: mhat = G, vhat = G^2 at every step, whatever the state."""
    rng = np.random.default_rng(4)
    G = rng.standard_normal((8, 16)) * 1e-2
    W = bf16_rand((8, 16), 0.02, 43)
    m, v = _state(8, 16, MOMENT_F32, 6, warm=True)
    out = oracle.adamw(G, W, m, v, moment_dtype=MOMENT_F32, step=13,
                       **dict(HP, beta1=0.0, beta2=0.0))
    W0 = oracle.bf16_bits_to_f64(W)
    want = (1 - f32(1e-3) * f32(0.1)) * W0 - f32(1e-3) * G / (np.abs(G) + f32(1e-8))
    np.testing.assert_allclose(out["W64"], want, rtol=1e-14, atol=1e-18)
    np.testing.assert_allclose(out["m64"], G, rtol=1e-15)


def test_lr_zero_leaves_weight_unchanged():
    rng = np.random.default_rng(5)
    G = rng.standard_normal((8, 16))
    W = bf16_rand((8, 16), 0.02, 44)
    m, v = _state(8, 16, MOMENT_BF16, 7, warm=True)
    out = oracle.adamw(G, W, m, v, moment_dtype=MOMENT_BF16, step=3, **dict(HP, lr=0.0))
    assert np.array_equal(out["W"], W)
    assert not np.array_equal(out["m"], m)


@pytest.mark.parametrize("step", [1, 2, 100, 5000])
def test_matches_torch_adamw_fp64(step):
    """torch.optim.AdamW (foreach=False, fp64) is an independent implementation of the update."""
    rng = np.random.default_rng(step)
    d_out, d_in = 12, 20
    G = rng.standard_normal((d_out, d_in)) * 0.02
    W = bf16_rand((d_out, d_in), 0.02, 50 + step)
    m, v = _state(d_out, d_in, MOMENT_F32, 8, warm=True)
    out = oracle.adamw(G, W, m, v, moment_dtype=MOMENT_F32, step=step, **HP)

    p = torch.nn.Parameter(torch.from_numpy(oracle.bf16_bits_to_f64(W)))
    opt = torch.optim.AdamW([p], lr=f32(1e-3), betas=(f32(0.9), f32(0.999)), eps=f32(1e-8),
                            weight_decay=f32(0.1), foreach=False, fused=False)
    p.grad = torch.from_numpy(G.copy())
    st = opt.state[p]
    st["step"] = torch.tensor(float(step - 1), dtype=torch.float64)
    st["exp_avg"] = torch.from_numpy(m.astype(np.float64))
    st["exp_avg_sq"] = torch.from_numpy(v.astype(np.float64))
    opt.step()
    np.testing.assert_allclose(out["m64"], st["exp_avg"].numpy(), rtol=1e-14, atol=0)
    np.testing.assert_allclose(out["v64"], st["exp_avg_sq"].numpy(), rtol=1e-14, atol=0)
    np.testing.assert_allclose(out["W64"], p.detach().numpy(), rtol=1e-13, atol=1e-17)


def test_bf16_moment_storage_is_rne_of_fp64():
    rng = np.random.default_rng(6)
    G = rng.standard_normal((8, 32)) * 0.02
    W = bf16_rand((8, 32), 0.02, 45)
    m, v = _state(8, 32, MOMENT_BF16, 9, warm=True)
    out = oracle.adamw(G, W, m, v, moment_dtype=MOMENT_BF16, step=100, **HP)
    assert np.array_equal(out["m"], oracle.f64_to_bf16_bits(out["m64"]))
    assert np.array_equal(out["v"], oracle.f64_to_bf16_bits(out["v64"]))
    # warm state decoded from bf16 enters the recurrence
    np.testing.assert_allclose(out["m64"], f32(0.9) * _decode(m, MOMENT_BF16) + (1 - f32(0.9)) * G,
                               rtol=1e-15)


def test_round_grad_to_bf16_variant():
    """The two-kernel path with a bf16 gradient buffer sees RNE(G) (App. B truncation)."""
    rng = np.random.default_rng(7)
    G = rng.standard_normal((8, 16)) * 0.02
    W = bf16_rand((8, 16), 0.02, 46)
    z = np.zeros((8, 16), np.float32)
    out = oracle.adamw(G, W, z, z, moment_dtype=MOMENT_F32, step=1, round_grad_to_bf16=True, **HP)
    Gr = oracle.bf16_bits_to_f64(oracle.f64_to_bf16_bits(G))
    assert not np.array_equal(Gr, G)
    np.testing.assert_allclose(out["m64"], (1 - f32(0.9)) * Gr, rtol=1e-15)


# ------------------------------------------------------------------------- int8 moments

def test_i8_quantizer_invariants():
    rng = np.random.default_rng(8)
    d_out, d_in = 512 + 100, 24          # two full blocks and a ragged 100-row block
    x = rng.standard_normal((d_out, d_in)) * 1e-3
    x[256:512, 5] = 0.0                  # an all-zero block column
    codes, scales = oracle.quantize_i8(x, second_moment=False)
    assert scales.shape == (3, d_in)
    assert codes.min() >= -127 and codes.max() <= 127
    for b in range(3):
        rows = slice(256 * b, min(256 * (b + 1), d_out))
        for q in range(d_in):
            col, cq, s = x[rows, q], codes[rows, q], float(scales[b, q])
            a = np.abs(col.astype(np.float32)).max()
            assert s == float(np.float32(a) / np.float32(127))
            if a == 0:
                assert s == 0 and not cq.any()
                continue
            assert np.abs(cq).max() == 127
            assert np.abs(cq[np.argmax(np.abs(col))]) == 127
            assert np.all(np.abs(col - s * cq.astype(np.float64)) <= s / 2 * (1 + 1e-6))


def test_i8_second_moment_floor_and_sqrt_storage():
    rng = np.random.default_rng(9)
    v = np.abs(rng.standard_normal((256, 16)) * 1e-6)
    v[3, 2] = 0.0
    v[7, 2] = 1e-20                         # would quantize to 0 without the floor
    codes, scales = oracle.quantize_i8(v, second_moment=True)
    assert codes.min() >= 1 and codes.max() <= 127
    r = np.sqrt(v)
    np.testing.assert_allclose(scales[0], np.abs(r.astype(np.float32)).max(0) / np.float32(127), rtol=0)
    dec = oracle.dequantize_i8(codes, scales, second_moment=True)
    assert np.all(dec > 0)
    big = r >= scales[0]                     # away from the floor the error is at most half a step
    assert np.all(np.abs(np.sqrt(dec) - r)[big] <= (scales[0] / 2 * (1 + 1e-6) * np.ones_like(r))[big])


def test_i8_first_moment_accumulated_error_bound():
    """App. B: re-quantizing every step keeps |m_q - m| <= s/(2(1-b1)), s the largest scale."""
    rng = np.random.default_rng(10)
    d_out, d_in, b1 = 256, 8, 0.9
    W = bf16_rand((d_out, d_in), 0.02, 47)
    m_exact = np.zeros((d_out, d_in))
    mq, ms = oracle.quantize_i8(m_exact, second_moment=False)
    vq, vs = oracle.quantize_i8(np.full((d_out, d_in), 1e-6), second_moment=True)
    smax = np.zeros(d_in)
    for t in range(1, 41):
        G = rng.standard_normal((d_out, d_in)) * 0.02
        out = oracle.adamw(G, W, mq, vq, m_scale=ms, v_scale=vs, moment_dtype=MOMENT_I8, step=t,
                           **dict(HP, beta1=b1))
        m_exact = f32(b1) * m_exact + (1 - f32(b1)) * G
        mq, vq, ms, vs = out["m"], out["v"], out["m_scale"], out["v_scale"]
        smax = np.maximum(smax, ms[0])
        err = np.abs(oracle.dequantize_i8(mq, ms, False) - m_exact)
        assert np.all(err <= smax / (2 * (1 - f32(b1))) * (1 + 1e-4))


def test_i8_step_weight_update_reads_unquantized_state():
    """int8 mode: the new codes decode near m', and W' is the same as with fp32 moments."""
    rng = np.random.default_rng(11)
    d_out, d_in = 300, 16
    G = rng.standard_normal((d_out, d_in)) * 0.02
    W = bf16_rand((d_out, d_in), 0.02, 48)
    m0 = rng.standard_normal((d_out, d_in)) * 1e-4
    v0 = np.abs(rng.standard_normal((d_out, d_in))) * 1e-6
    mq, ms = oracle.quantize_i8(m0, False)
    vq, vs = oracle.quantize_i8(v0, True)
    out8 = oracle.adamw(G, W, mq, vq, m_scale=ms, v_scale=vs, moment_dtype=MOMENT_I8, step=100,
                        want_quotients=True, **HP)
    # same decoded state as fp64 moments through the fp32-storage path -> same W64
    md = oracle.dequantize_i8(mq, ms, False)
    vd = oracle.dequantize_i8(vq, vs, True)
    ref = oracle.adamw(G, W, md.astype(np.float32), vd.astype(np.float32), moment_dtype=MOMENT_F32,
                       step=100, **HP)
    # fp32 storage of the decoded state rounds it: allow that rounding only
    np.testing.assert_allclose(out8["W64"], ref["W64"], rtol=1e-6, atol=1e-9)
    dec = oracle.dequantize_i8(out8["m"], out8["m_scale"], False)
    s = np.repeat(out8["m_scale"], 256, axis=0)[:d_out]
    assert np.all(np.abs(dec - out8["m64"]) <= s / 2 * (1 + 1e-5))
    assert np.all(np.abs(out8["qm"] - out8["m"]) <= 0.5 + 1e-6)


# ------------------------------------------------------------------------- other update rules

from oracle import (OPT_ADAGRAD, OPT_ADAMAX, OPT_LION, OPT_MUON, OPT_NADAM, OPT_RADAM, OPT_RMSPROP,  # noqa: E402
                    OPT_SGD, OPT_SGD_MOMENTUM)

RHP = dict(lr=f32(2e-3), beta1=f32(0.9), beta2=f32(0.99), eps=f32(1e-8), weight_decay=f32(0.05),
           lr_decay=f32(0.01), momentum_decay=f32(0.004))


def _rule_inputs(seed, d_out=10, d_in=16):
    rng = np.random.default_rng(seed)
    G = rng.standard_normal((d_out, d_in)) * 0.02
    W = bf16_rand((d_out, d_in), 0.02, 60 + seed)
    s1 = (rng.standard_normal((d_out, d_in)) * 1e-3).astype(np.float32)
    s2 = np.abs(rng.standard_normal((d_out, d_in)) * 1e-4).astype(np.float32)
    return G, W, s1, s2


def _torch_param(W):
    return torch.nn.Parameter(torch.from_numpy(oracle.bf16_bits_to_f64(W)))


def _t(a):
    return torch.from_numpy(np.asarray(a, dtype=np.float64).copy())


def _torch_step(opt_code, W, G, s1, s2, step, h):
    """The same step by torch.optim (fp64, foreach=False): returns (W, state1, state2)."""
    p = _torch_param(W)
    ts = lambda: torch.tensor(float(step - 1), dtype=torch.float64)
    if opt_code == OPT_SGD:
        o = torch.optim.SGD([p], lr=h["lr"], weight_decay=h["weight_decay"], foreach=False)
        names = ()
    elif opt_code == OPT_SGD_MOMENTUM:
        o = torch.optim.SGD([p], lr=h["lr"], momentum=h["beta1"], weight_decay=h["weight_decay"], foreach=False)
        o.state[p]["momentum_buffer"] = _t(s1)
        names = ("momentum_buffer",)
    elif opt_code == OPT_ADAGRAD:
        o = torch.optim.Adagrad([p], lr=h["lr"], lr_decay=h["lr_decay"], weight_decay=h["weight_decay"],
                                eps=h["eps"], foreach=False)
        o.state[p].update(step=ts(), sum=_t(s1))
        names = ("sum",)
    elif opt_code == OPT_RMSPROP:
        o = torch.optim.RMSprop([p], lr=h["lr"], alpha=h["beta2"], eps=h["eps"], weight_decay=h["weight_decay"],
                                foreach=False)
        o.state[p].update(step=ts(), square_avg=_t(s1))
        names = ("square_avg",)
    elif opt_code == OPT_NADAM:
        kw = dict(lr=h["lr"], betas=(h["beta1"], h["beta2"]), eps=h["eps"], weight_decay=h["weight_decay"],
                  momentum_decay=h["momentum_decay"], foreach=False)
        # torch's own momentum-schedule product after step - 1 steps (it depends on the step only)
        q = torch.nn.Parameter(torch.zeros(1, dtype=torch.float64))
        oq = torch.optim.NAdam([q], **kw)
        for _ in range(step - 1):
            q.grad = torch.ones(1, dtype=torch.float64)
            oq.step()
        mu_product = oq.state[q]["mu_product"].clone() if step > 1 else torch.tensor(1.0, dtype=torch.float64)
        o = torch.optim.NAdam([p], **kw)
        o.state[p].update(step=ts(), mu_product=mu_product, exp_avg=_t(s1), exp_avg_sq=_t(s2))
        names = ("exp_avg", "exp_avg_sq")
    elif opt_code == OPT_RADAM:
        o = torch.optim.RAdam([p], lr=h["lr"], betas=(h["beta1"], h["beta2"]), eps=h["eps"],
                              weight_decay=h["weight_decay"], foreach=False)
        o.state[p].update(step=ts(), exp_avg=_t(s1), exp_avg_sq=_t(s2))
        names = ("exp_avg", "exp_avg_sq")
    elif opt_code == OPT_ADAMAX:
        o = torch.optim.Adamax([p], lr=h["lr"], betas=(h["beta1"], h["beta2"]), eps=h["eps"],
                               weight_decay=h["weight_decay"], foreach=False)
        o.state[p].update(step=ts(), exp_avg=_t(s1), exp_inf=_t(s2))
        names = ("exp_avg", "exp_inf")
    p.grad = torch.from_numpy(G.copy())
    o.step()
    st = [o.state[p][n].numpy() for n in names]
    return p.detach().numpy(), (st + [None, None])[0], (st + [None, None])[1]


@pytest.mark.parametrize("step", [1, 3, 100])
@pytest.mark.parametrize("opt_code", [OPT_SGD, OPT_SGD_MOMENTUM, OPT_ADAGRAD, OPT_RMSPROP, OPT_NADAM, OPT_RADAM,
                                      OPT_ADAMAX],
                         ids=["sgd", "sgd_momentum", "adagrad", "rmsprop", "nadam", "radam", "adamax"])
def test_rules_match_torch_optim_fp64(opt_code, step):
    """torch.optim (fp64) is the reference implementation each family was checked against."""
    G, W, s1, s2 = _rule_inputs(step + 10 * opt_code)
    hp = dict(RHP)
    if opt_code in (OPT_NADAM, OPT_RADAM):
        hp["beta2"] = f32(0.999)     # RAdam's rectification switches on within the steps tested
    out = oracle.rule_step(G, W, s1, s2, opt=opt_code, state_dtype=MOMENT_F32, step=step, **hp)
    prev = torch.get_default_dtype()
    torch.set_default_dtype(torch.float64)     # torch's scalar state (NAdam's product) in fp64 too
    try:
        wt, a, b = _torch_step(opt_code, W, G, s1, s2, step, hp)
    finally:
        torch.set_default_dtype(prev)
    np.testing.assert_allclose(out["W64"], wt, rtol=1e-13, atol=1e-18)
    if a is not None:
        np.testing.assert_allclose(out["s1_64"], a, rtol=1e-13, atol=1e-20)
    if b is not None:
        np.testing.assert_allclose(out["s2_64"], b, rtol=1e-13, atol=1e-20)


def test_radam_takes_both_branches():
    """rho_t > 5 decides RAdam's rectification: off at t = 1, on at t = 100 (beta2 = 0.999)."""
    G, W, s1, s2 = _rule_inputs(5)
    hp = dict(RHP, beta2=f32(0.999), weight_decay=0.0)
    a = oracle.rule_step(G, W, s1, s2, opt=OPT_RADAM, state_dtype=MOMENT_F32, step=1, **hp)
    # unrectified: w' = w - lr m' / (1 - beta1)
    w = oracle.bf16_bits_to_f64(W)
    np.testing.assert_allclose(a["W64"], w - f32(2e-3) * a["s1_64"] / (1 - f32(0.9)), rtol=1e-14)
    b = oracle.rule_step(G, W, s1, s2, opt=OPT_RADAM, state_dtype=MOMENT_F32, step=100, **hp)
    assert not np.allclose(b["W64"], w - f32(2e-3) * b["s1_64"] / (1 - f32(0.9) ** 100), rtol=1e-6)


def test_lion_zero_betas_is_sign_descent():
    """beta1 = beta2 = 0: Lion is sign descent with decoupled decay, and m' = g."""
    G, W, s1, _ = _rule_inputs(6)
    G[0, :3] = 0.0
    out = oracle.rule_step(G, W, s1, opt=OPT_LION, state_dtype=MOMENT_F32, step=7,
                           **dict(RHP, beta1=0.0, beta2=0.0))
    w = oracle.bf16_bits_to_f64(W)
    lr, wd = f32(2e-3), f32(0.05)
    np.testing.assert_allclose(out["W64"], w * (1 - lr * wd) - lr * np.sign(G), rtol=1e-15, atol=1e-20)
    np.testing.assert_array_equal(out["s1_64"], G)


def test_lion_update_magnitude_and_momentum_closed_form():
    G, W, s1, _ = _rule_inputs(7)
    out = oracle.rule_step(G, W, s1, opt=OPT_LION, state_dtype=MOMENT_F32, step=3, **RHP)
    w = oracle.bf16_bits_to_f64(W)
    lr, wd = f32(2e-3), f32(0.05)
    # every weight moves by exactly lr beyond its decay (no element has c == 0 here)
    np.testing.assert_allclose(np.abs(out["W64"] - w * (1 - lr * wd)), lr, rtol=1e-12)
    # the sign follows the beta1 interpolation, not beta2's
    m = s1.astype(np.float64)
    assert np.array_equal(np.sign(w * (1 - lr * wd) - out["W64"]), np.sign(out["aux"]))
    # constant gradient from m = 0: after k steps m_k = (1 - beta2^k) g (EMA closed form)
    m = np.zeros_like(s1)
    for _ in range(5):
        m = oracle.rule_step(G, W, m, opt=OPT_LION, state_dtype=MOMENT_F32, step=1, **RHP)["s1"]
    np.testing.assert_allclose(m, (1 - f32(0.99) ** 5) * G, rtol=1e-6)


def test_lion_beta1_and_beta2_roles_on_exact_values():
    W = to_bits([[1.0, 1.0]])
    G = np.array([[-1.0, 1.0]])
    m = np.array([[1.0, -1.0]], dtype=np.float32)
    out = oracle.rule_step(G, W, m, opt=OPT_LION, state_dtype=MOMENT_F32, step=1,
                           lr=0.25, beta1=0.25, beta2=0.75, weight_decay=0.0)
    # c = 0.25 m + 0.75 g = (-0.5, 0.5): the sign of g wins; m' = 0.75 m + 0.25 g = (0.5, -0.5)
    np.testing.assert_array_equal(out["W64"], [[1.25, 0.75]])
    np.testing.assert_array_equal(out["s1_64"], [[0.5, -0.5]])


def test_muon_accumulate_is_heavy_ball_buffer_and_leaves_w():
    """B' = mu B + G is the heavy-ball recurrence of torch.optim.SGD's momentum buffer
    (dampening 0, no decay); W is not touched."""
    G, W, s1, _ = _rule_inputs(8)
    out = oracle.rule_step(G, W, s1, opt=OPT_MUON, state_dtype=MOMENT_F32, step=4, lr=0.0, beta1=f32(0.95))
    p = _torch_param(W)
    o = torch.optim.SGD([p], lr=0.0, momentum=f32(0.95), foreach=False)
    o.state[p]["momentum_buffer"] = _t(s1)
    p.grad = torch.from_numpy(G.copy())
    o.step()
    np.testing.assert_allclose(out["s1_64"], o.state[p]["momentum_buffer"].numpy(), rtol=1e-15)
    assert np.array_equal(out["W"], W)


def test_muon_accumulate_over_micro_batches_is_the_whole_batch_gradient():
    """Accumulating micro-batches with beta = mu, then 1, gives mu B + G over all tokens
    (Prop. 1: G is additive over a partition of the token axis)."""
    T, d_in, d_out = 48, 16, 8
    X = bf16_rand((T, d_in), 1.0, 70)
    dY = bf16_rand((T, d_out), 0.01, 71)
    W = bf16_rand((d_out, d_in), 0.02, 72)
    B = np.zeros((d_out, d_in), np.float32) + np.float32(0.5)
    mu = f32(0.95)
    b1 = oracle.rule_step(oracle.wgrad(X[:20], dY[:20]), W, B, opt=OPT_MUON, state_dtype=MOMENT_F32, step=1,
                          lr=0.0, beta1=mu)["s1_64"]
    b2 = oracle.rule_step(oracle.wgrad(X[20:], dY[20:]), W, b1.astype(np.float32), opt=OPT_MUON,
                          state_dtype=MOMENT_F32, step=1, lr=0.0, beta1=1.0)["s1_64"]
    want = mu * 0.5 + oracle.wgrad(X, dY)
    # the first call's B' is rounded to fp32 before the second: allow that rounding
    np.testing.assert_allclose(b2, want, rtol=2 ** -23, atol=2 ** -24 * np.abs(b1).max())


def test_unrounded_adamw_reference_equals_the_oracle_before_rounding():
    """adamw_f64 (the fidelity experiment's reference, no storage rounding) computes the
    same fp64 values as the C oracle's AdamW before it rounds them to storage."""
    rng = np.random.default_rng(9)
    G = rng.standard_normal((12, 20)) * 0.02
    W = bf16_rand((12, 20), 0.02, 90)
    m, v = _state(12, 20, MOMENT_F32, 91, warm=True)
    for step in (1, 7):
        ora = oracle.adamw(G, W, m, v, moment_dtype=MOMENT_F32, step=step, **HP)
        W1, m1, v1 = oracle.adamw_f64(G, oracle.bf16_bits_to_f64(W), m.astype(np.float64), v.astype(np.float64),
                                      step=step, **HP)
        np.testing.assert_allclose(W1, ora["W64"], rtol=1e-15, atol=0)
        np.testing.assert_allclose(m1, ora["m64"], rtol=1e-15, atol=0)
        np.testing.assert_allclose(v1, ora["v64"], rtol=1e-15, atol=0)


# ------------------------------------------------------------------------- int8, 64-wide row blocks

from oracle import MOMENT_I8_ROW64  # noqa: E402


def test_i8_row64_quantizer_invariants():
    """App. B's layout: one scale per 64 consecutive elements of a row (a ragged last block
    when d_in is not a multiple of 64), s = absmax/127, |code| <= 127 with the absmax at
    +-127, and every element within half a step of its code."""
    rng = np.random.default_rng(11)
    d_out, d_in = 5, 200                    # blocks of 64, 64, 64, 8 per row
    x = rng.standard_normal((d_out, d_in)) * 10.0 ** rng.integers(-6, 0, (d_out, 1))
    x[2, 64:128] = 0.0                      # an all-zero block
    codes, scales = oracle.quantize_i8_row64(x, second_moment=False)
    assert scales.shape == (d_out, 4)
    for p in range(d_out):
        for b in range(4):
            blk = slice(64 * b, min(64 * b + 64, d_in))
            a = np.float32(np.abs(x[p, blk].astype(np.float32)).max())
            assert scales[p, b] == np.float32(a / np.float32(127.0))
            if a > 0:
                assert np.abs(codes[p, blk]).max() == 127
                err = np.abs(scales[p, b] * codes[p, blk].astype(np.float64) - x[p, blk])
                assert np.all(err <= 0.5 * scales[p, b] * (1 + 1e-6) + 1e-7 * np.abs(x[p, blk]))
            else:
                assert not codes[p, blk].any()
    # a change in one element moves only its own block's scale
    y = x.copy()
    y[1, 70] *= 100.0
    _, s2 = oracle.quantize_i8_row64(y, second_moment=False)
    changed = np.argwhere(s2 != scales)
    assert changed.tolist() == [[1, 1]]


def test_i8_row64_second_moment_floor_and_no_square_root():
    v = np.abs(np.random.default_rng(12).standard_normal((3, 128))) * 1e-6
    v[0, :64] = 0.0
    v[1, 5] = 1e-20                          # tiny next to its block's max
    codes, scales = oracle.quantize_i8_row64(v, second_moment=True)
    assert not codes[0, :64].any() and scales[0, 0] == 0.0
    assert codes[1, 5] == 1                  # floored away from zero
    assert np.all(codes[np.repeat(scales, 64, axis=1) > 0] >= 1)
    # v itself is stored: the block max maps to 127 and decodes to v (no sqrt)
    np.testing.assert_allclose(oracle.dequantize_i8_row64(codes, scales).max(axis=1)[1:],
                               v.max(axis=1)[1:], rtol=1e-6)


def test_i8_row64_first_moment_accumulated_error_bound():
    """App. B: re-quantising every step keeps |m_q - m| <= s/(2(1-b1)), s the largest scale
    the block has had."""
    rng = np.random.default_rng(13)
    d_out, d_in, b1 = 4, 192, 0.9
    W = bf16_rand((d_out, d_in), 0.02, 48)
    m_exact = np.zeros((d_out, d_in))
    mq, ms = oracle.quantize_i8_row64(m_exact, second_moment=False)
    vq, vs = oracle.quantize_i8_row64(np.full((d_out, d_in), 1e-6), second_moment=True)
    smax = np.zeros_like(ms)
    for t in range(1, 41):
        G = rng.standard_normal((d_out, d_in)) * 0.02
        out = oracle.adamw(G, W, mq, vq, m_scale=ms, v_scale=vs, moment_dtype=MOMENT_I8_ROW64, step=t,
                           **dict(HP, beta1=b1))
        m_exact = f32(b1) * m_exact + (1 - f32(b1)) * G
        mq, vq, ms, vs = out["m"], out["v"], out["m_scale"], out["v_scale"]
        smax = np.maximum(smax, ms)
        err = np.abs(oracle.dequantize_i8_row64(mq, ms) - m_exact)
        assert np.all(err <= np.repeat(smax, 64, axis=1) / (2 * (1 - f32(b1))) * (1 + 1e-4))


def test_i8_row64_step_reads_unquantized_state_for_the_weight():
    rng = np.random.default_rng(14)
    d_out, d_in = 6, 136
    G = rng.standard_normal((d_out, d_in)) * 0.02
    W = bf16_rand((d_out, d_in), 0.02, 49)
    mq, ms = oracle.quantize_i8_row64(rng.standard_normal((d_out, d_in)) * 1e-3, second_moment=False)
    vq, vs = oracle.quantize_i8_row64(np.abs(rng.standard_normal((d_out, d_in))) * 1e-6, second_moment=True)
    out = oracle.adamw(G, W, mq, vq, m_scale=ms, v_scale=vs, moment_dtype=MOMENT_I8_ROW64, step=5, **HP)
    W1, m1, v1 = oracle.adamw_f64(G, oracle.bf16_bits_to_f64(W), oracle.dequantize_i8_row64(mq, ms),
                                  oracle.dequantize_i8_row64(vq, vs), step=5, **HP)
    np.testing.assert_allclose(out["W64"], W1, rtol=1e-15)
    np.testing.assert_allclose(out["m64"], m1, rtol=1e-15)
    np.testing.assert_allclose(out["v64"], v1, rtol=1e-15)
    # and the stored state is that unquantised state, re-quantised
    qm, sm = oracle.quantize_i8_row64(m1, second_moment=False)
    assert np.array_equal(qm, out["m"]) and np.array_equal(sm, out["m_scale"])


# ------------------------------------------------------------------------- fp8 (E4M3) encodings

def test_e4m3_code_table_facts():
    """OCP E4M3: codes 0..126 are the finite non-negative values in increasing order, from 0
    through the smallest subnormal 2^-9 and the smallest normal 2^-6 (code 8) to 448 (code
    126); 127 is NaN; the sign bit mirrors them; every finite code round-trips."""
    vals = oracle.e4m3_decode(np.arange(256, dtype=np.uint8))
    pos = vals[:127]
    assert pos[0] == 0.0 and pos[1] == 2.0 ** -9 and pos[8] == 2.0 ** -6 and pos[126] == 448.0
    assert np.all(np.diff(pos) > 0)
    assert np.isnan(vals[127]) and np.isnan(vals[255])
    np.testing.assert_array_equal(vals[128:255], -pos)
    codes = np.concatenate([np.arange(127), np.arange(128, 255)]).astype(np.uint8)
    assert np.array_equal(oracle.e4m3_encode(vals[codes].astype(np.float32)), codes)


def test_e4m3_encode_is_nearest_even_by_brute_force():
    rng = np.random.default_rng(15)
    pos = oracle.e4m3_decode(np.arange(127, dtype=np.uint8))
    mids = (0.5 * (pos[1:] + pos[:-1])).astype(np.float32)           # exact ties (representable in fp32)
    x = np.concatenate([mids, -mids, (rng.random(4000) * 448).astype(np.float32),
                        (2.0 ** rng.uniform(-14, 8.8, 4000)).astype(np.float32)])
    got = oracle.e4m3_encode(x)
    for xi, c in zip(x, got):
        a = abs(float(xi))
        d = np.abs(pos - a)
        best = np.flatnonzero(d == d.min())
        want = best[0] if len(best) == 1 else best[best % 2 == 0][0]   # tie: even code
        assert (c & 0x7F) == want and (c >> 7) == (1 if np.signbit(xi) else 0), (xi, c, want)


def _fp8_state(d_out, d_in, seed):
    rng = np.random.default_rng(seed)
    G = rng.standard_normal((d_out, d_in)) * 0.02
    W = bf16_rand((d_out, d_in), 0.02, seed)
    z = np.zeros((d_out, d_in), np.uint8)
    return G, W, z, z.copy(), np.zeros(4, np.float32), np.zeros(4, np.float32)


def test_fp8_cold_start_and_ring_slots():
    """Step 1 from a zero ring encodes with scale 1, records max|m'| and max sqrt(v') into
    slot 1 and clears slot 2; step 2 encodes with slot 1's scale, so the tensor's largest
    value lands on 448 (or saturates there)."""
    G, W, m, v, mr, vr = _fp8_state(6, 40, 16)
    mr[2] = vr[2] = 123.0                      # stale content the step must clear
    o1 = oracle.adamw_fp8(G, W, m, v, w_fp8=False, m_fp8=True, m_ring=mr, v_ring=vr, step=1, **HP)
    m1 = o1["m64"].astype(np.float32)
    assert o1["m_ring"][1] == np.abs(m1).max() and o1["v_ring"][1] == np.sqrt(o1["v64"]).astype(np.float32).max()
    assert o1["m_ring"][2] == 0.0 and o1["v_ring"][2] == 0.0
    np.testing.assert_array_equal(o1["m"], oracle.e4m3_encode(np.clip(m1, -448, 448)))   # scale 1
    o2 = oracle.adamw_fp8(G, o1["W"], o1["m"], o1["v"], w_fp8=False, m_fp8=True, m_ring=o1["m_ring"],
                          v_ring=o1["v_ring"], step=2, **HP)
    s = np.float32(o1["m_ring"][1] / np.float32(448.0))
    np.testing.assert_array_equal(o2["qm"], (o2["m64"].astype(np.float32) / s).astype(np.float64))
    big = np.abs(o2["qm"]) >= 448.0
    assert np.all((o2["m"][big] & 0x7F) == 126)          # at or beyond last step's amax: the top code
    # step 2 decoded step 1's codes with scale 1 (slot 0 empty)
    dec = oracle.e4m3_decode(o1["m"])
    np.testing.assert_allclose(o2["m64"], f32(0.9) * dec + (1 - f32(0.9)) * G, rtol=1e-15)


def test_fp8_second_moment_floor_and_sqrt_storage():
    G, W, m, v, mr, vr = _fp8_state(4, 24, 17)
    G[0, 0] = 1e-12                            # sqrt(v') ~ 3e-14: far below the smallest code
    o = oracle.adamw_fp8(G, W, m, v, w_fp8=False, m_fp8=True, m_ring=mr, v_ring=vr, step=1, **HP)
    assert o["v"][0, 0] == 1
    ok = o["v"] != 1
    np.testing.assert_array_equal(o["v"][ok], oracle.e4m3_encode(np.sqrt(o["v64"]).astype(np.float32))[ok])


def test_fp8_weight_update_reads_decoded_state():
    G, W, m, v, mr, vr = _fp8_state(5, 32, 18)
    wr = np.zeros(4, np.float32)
    Wc = oracle.e4m3_encode(np.clip(oracle.bf16_bits_to_f64(W).astype(np.float32) * 100, -448, 448))
    wr[3] = np.float32(448.0 / 100 * 448) / 1.0        # slot (t-2)%4 for t = 5: scale 448/100
    wr[0] = wr[3]
    mc = oracle.e4m3_encode(np.full((5, 32), 0.5, np.float32))
    vc = oracle.e4m3_encode(np.full((5, 32), 0.25, np.float32))
    mr[3] = vr[3] = np.float32(448.0 * 1e-3)             # decode scale 1e-3
    o = oracle.adamw_fp8(G, Wc, mc, vc, w_fp8=True, m_fp8=True, w_ring=wr, m_ring=mr, v_ring=vr, step=5, **HP)
    sw = np.float32(wr[3] / np.float32(448.0))
    W0 = sw * oracle.e4m3_decode(Wc)
    m0 = np.float32(1e-3) * oracle.e4m3_decode(mc)
    v0 = (np.float32(1e-3) * oracle.e4m3_decode(vc)) ** 2
    W1, m1, v1 = oracle.adamw_f64(G, W0, m0, v0, step=5, **HP)
    np.testing.assert_allclose(o["W64"], W1, rtol=1e-14)
    np.testing.assert_allclose(o["m64"], m1, rtol=1e-14)
    np.testing.assert_allclose(o["v64"], v1, rtol=1e-14)


# ------------------------------------------------------------------------- int8 rounding ties

# App. B rounds x/s to an integer code; the oracle reads "round" as round half to even
# (ties to the even integer).  With a block absmax of exactly 127 the fp32 scale is exactly
# 1 and every quotient is its value, so exact half-integers are ties.  Round half away from
# zero (roundf), round half up (floor(x + 1/2)) and truncation each give different codes on
# at least one of these.
TIE_VALUES = [127.0, 0.5, 1.5, 2.5, 3.5, -0.5, -1.5, -2.5, -3.5, 126.5, -126.5, 4.5, -4.5, 0.0, 1.0]
TIE_CODES_EVEN = [127, 0, 2, 2, 4, 0, -2, -2, -4, 126, -126, 4, -4, 0, 1]


def test_round_half_even_codes_differ_from_other_tie_rules():
    """The expected codes above are not those of the other plausible rounding rules."""
    x = np.array(TIE_VALUES)
    away = np.sign(x) * np.floor(np.abs(x) + 0.5)
    up = np.floor(x + 0.5)
    assert not np.array_equal(away, TIE_CODES_EVEN)
    assert not np.array_equal(up, TIE_CODES_EVEN)
    assert not np.array_equal(np.trunc(x), TIE_CODES_EVEN)


def test_i8_column_quantizer_rounds_ties_to_even():
    """256-row column blocks: one column holds the tie values (rest zero), absmax 127."""
    d_out, d_in = 256, 3
    x = np.zeros((d_out, d_in))
    x[:len(TIE_VALUES), 1] = TIE_VALUES
    x[::-1][:len(TIE_VALUES), 2] = TIE_VALUES       # the same values at the block's far end
    codes, scales = oracle.quantize_i8(x, second_moment=False)
    assert scales[0, 1] == 1.0 and scales[0, 2] == 1.0 and scales[0, 0] == 0.0
    assert codes[:len(TIE_VALUES), 1].tolist() == TIE_CODES_EVEN
    assert codes[::-1][:len(TIE_VALUES), 2].tolist() == TIE_CODES_EVEN
    assert not codes[len(TIE_VALUES):, 1].any()


def test_i8_column_quantizer_second_moment_ties_through_the_square_root():
    """sqrt(v) is stored: v = r^2 for the non-negative tie values r (exact squares, exact
    roots), so the codes are round-half-even(r), floored at 1 in a non-zero block."""
    r = np.array([127.0, 0.5, 1.5, 2.5, 3.5, 126.5, 4.5, 0.0, 1.0])
    v = np.zeros((256, 1))
    v[:len(r), 0] = r * r
    codes, scales = oracle.quantize_i8(v, second_moment=True)
    assert scales[0, 0] == 1.0
    # 0.5 -> 0 -> floored to 1; 0 -> 0 -> floored to 1
    assert codes[:len(r), 0].tolist() == [127, 1, 2, 2, 4, 126, 4, 1, 1]


def test_i8_row64_quantizer_rounds_ties_to_even():
    """64-wide row blocks: the tie values in one block of a row, absmax 127; a second row
    holds them at the end of a ragged last block."""
    d_out, d_in = 2, 64 + 20
    x = np.zeros((d_out, d_in))
    x[0, 3:3 + len(TIE_VALUES)] = TIE_VALUES
    x[1, 64 + 20 - len(TIE_VALUES):] = TIE_VALUES
    codes, scales = oracle.quantize_i8_row64(x, second_moment=False)
    assert scales[0, 0] == 1.0 and scales[1, 1] == 1.0
    assert codes[0, 3:3 + len(TIE_VALUES)].tolist() == TIE_CODES_EVEN
    assert codes[1, 64 + 20 - len(TIE_VALUES):].tolist() == TIE_CODES_EVEN


def _tie_step(moment_dtype, layout_shape):
    """One AdamW step with beta1 = beta2 = 0, so m' = G and v' = G^2 exactly; G holds the
    tie values in one int8 block, which therefore has absmax 127 and scale 1."""
    d_out, d_in = layout_shape
    G = np.zeros((d_out, d_in))
    W = np.zeros((d_out, d_in), dtype=np.uint16)
    if moment_dtype == MOMENT_I8:
        G[:len(TIE_VALUES), 0] = TIE_VALUES
        mq, ms = oracle.quantize_i8(np.zeros((d_out, d_in)), False)
        vq, vs = oracle.quantize_i8(np.zeros((d_out, d_in)), True)
    else:
        G[0, :len(TIE_VALUES)] = TIE_VALUES
        mq, ms = oracle.quantize_i8_row64(np.zeros((d_out, d_in)), False)
        vq, vs = oracle.quantize_i8_row64(np.zeros((d_out, d_in)), True)
    out = oracle.adamw(G, W, mq, vq, m_scale=ms, v_scale=vs, moment_dtype=moment_dtype, step=1,
                       want_quotients=True, **dict(HP, beta1=0.0, beta2=0.0))
    return G, out


def test_i8_column_step_rounds_ties_to_even():
    G, out = _tie_step(MOMENT_I8, (256, 2))
    n = len(TIE_VALUES)
    np.testing.assert_array_equal(out["m64"][:n, 0], TIE_VALUES)
    assert out["m_scale"][0, 0] == 1.0 and out["v_scale"][0, 0] == 1.0
    assert out["m"][:n, 0].tolist() == TIE_CODES_EVEN
    # sqrt(v') = |G|: codes round-half-even(|G|), floored at 1
    want_v = [max(1, abs(c)) for c in TIE_CODES_EVEN]
    assert out["v"][:n, 0].tolist() == want_v
    np.testing.assert_array_equal(out["qm"][:n, 0], TIE_VALUES)


def test_i8_row64_step_rounds_ties_to_even():
    G, out = _tie_step(MOMENT_I8_ROW64, (1, 64))
    n = len(TIE_VALUES)
    assert out["m_scale"][0, 0] == 1.0
    assert out["m"][0, :n].tolist() == TIE_CODES_EVEN
    # v itself is stored (no square root): v' = G^2 with absmax 127^2, scale 127^2/127 = 127;
    # quotients G^2/127 are not ties, so only check the floor and the absmax code here
    assert out["v_scale"][0, 0] == np.float32(127.0 * 127.0) / np.float32(127.0)
    assert out["v"][0, 0] == 127 and out["v"][0, n - 2] >= 1 and out["v"][0, n - 2] == 1
