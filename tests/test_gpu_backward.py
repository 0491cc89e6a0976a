"""GPU parity of the layer-level backward: dX = dY W from the pre-update W, then the fused step.

* ``forge_input_grad`` against the oracle's fp64 dX on ragged and multi-tile shapes, all
  three tile shapes (64 and 128 token rows by 128 columns, and 256 x 256 with eight waves),
  and the masking of the K tail (a chunk past a segment's d_out must read zeros, not the
  next dY row or memory past W);
* ``forge_linear_backward`` equals ``forge_input_grad`` on the pre-update W followed by
  ``forge_linear_step``, bit for bit, and matches the oracle;
* ``forge_linear_backward_grouped`` sums the projections of one input (q, k, v) into one
  dX and steps them like ``forge_linear_step_grouped``.

The dX bar, derived from the arithmetic: the kernel accumulates exact bf16 x bf16 products
in fp32 in some order over K = sum of d_out, then rounds once to bf16.  So
|dX_gpu - dX| <= 2^-8 (|dX| + E) + E with E = K 2^-24 (|dY| |W|) per element (bf16
rounding is at most half an ulp, 2^-8 relative; fp32 summation errs by at most
gamma_K times the sum of magnitudes).  On top, at least 99% of the elements must equal the
oracle's value rounded to bf16 exactly (the fp32 error is far below half a bf16 ulp).
"""
import numpy as np
import pytest
import torch

import oracle
from compare import check_step
from gpu_util import HP, bits, dev, make_problem, run_oracle
from paper_2606_22932_amd import forge, synth

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)


def check_dx(gpu_bits, terms, frac_exact=0.99):
    """gpu_bits: bf16 bits [T, d_in]; terms: list of (dY bits, W bits) whose products sum to dX."""
    exact = sum(oracle.input_grad(y, w) for y, w in terms)
    scale = sum(np.abs(oracle.bf16_bits_to_f64(y)) @ np.abs(oracle.bf16_bits_to_f64(w)) for y, w in terms)
    K = sum(y.shape[1] for y, _ in terms)
    E = K * 2.0 ** -24 * scale + 2.0 ** -50 * scale
    got = oracle.bf16_bits_to_f64(gpu_bits)
    tol = 2.0 ** -8 * (np.abs(exact) + E) + E
    err = np.abs(got - exact)
    bad = ~(err <= tol)
    assert not bad.any(), (f"dX: {int(bad.sum())} elements outside the bound; worst at "
                           f"{np.unravel_index(np.argmax(err - tol), err.shape)}")
    n_exact = int((gpu_bits == oracle.f64_to_bf16_bits(exact)).sum())
    assert n_exact >= frac_exact * gpu_bits.size, f"dX: only {n_exact}/{gpu_bits.size} equal to RNE(oracle)"
    return dict(n=gpu_bits.size, exact=n_exact, max_rel_to_tol=float((err / np.maximum(tol, 1e-300)).max(initial=0)))


def _rand(shape, std, seed):
    return synth.gaussian(shape, std, seed)


# (T, d_in, d_out): multi-tile, ragged in every axis, a lone token row, the 128-row tiles
# (4096 x 2048 gives 512 tiles of 128 x 128, two per compute unit), a single 8-wide tile,
# 128-row tiles again at the sizes just below the 256 x 256 grid (16 x 32 of them, and 17 x 32
# ragged on both axes), and the 256 x 256 tiles (16 x 16 and 17 x 17 of them, ragged on both
# axes and, with d_out = 1032, in the last K chunk).  On a 256-CU device each shape past the
# first few selects the tile named.
DX_SHAPES = [(128, 256, 256), (200, 136, 40), (1000, 520, 776), (1, 128, 4096), (4096, 2048, 264),
             (64, 8, 8), (77, 1032, 1000), (2048, 4096, 264), (2100, 4040, 200), (4000, 4040, 200),
             (4100, 4104, 1032)]


@pytest.mark.parametrize("shape", DX_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_input_grad_matches_oracle(shape):
    T, d_in, d_out = shape
    _say(f"input_grad T={T} d_in={d_in} d_out={d_out}")
    dY = _rand((T, d_out), 1e-3, 9100 + T)
    W = _rand((d_out, d_in), 0.02, 9200 + d_in)
    dYg, Wg = dY.cuda(), W.cuda()
    dX = torch.full((T, d_in), float("nan"), dtype=torch.bfloat16, device="cuda")
    forge.forge_input_grad(dYg, Wg, dX)
    torch.cuda.synchronize()
    assert torch.equal(dYg.cpu(), dY) and torch.equal(Wg.cpu(), W), "inputs were modified"
    _say(check_dx(bits(dX), [(bits(dY), bits(W))]))


def test_input_grad_zero_dout_fills_zeros():
    T, d_in = 100, 264
    dY = torch.empty((T, 0), dtype=torch.bfloat16, device="cuda")
    W = torch.empty((0, d_in), dtype=torch.bfloat16, device="cuda")
    dX = torch.full((T, d_in), float("nan"), dtype=torch.bfloat16, device="cuda")
    forge.forge_input_grad(dY, W, dX)
    torch.cuda.synchronize()
    assert torch.equal(dX.cpu(), torch.zeros((T, d_in), dtype=torch.bfloat16))


def test_input_grad_k_tail_reads_zeros():
    """d_out = 40: the second 32-row chunk holds 8 real rows.  dY's row t+1 follows row t in
    memory and W sits inside a larger buffer whose next rows are +Inf: a chunk that read
    either instead of zeros would put Inf * 0 = NaN into dX."""
    T, d_in, d_out = 96, 264, 40
    dY = _rand((T, d_out), 1e-3, 9301)
    W_big = torch.full((d_out + 64, d_in), float("inf"), dtype=torch.bfloat16)
    W_big[:d_out] = _rand((d_out, d_in), 0.02, 9302)
    t_inf = 37
    dY_inf = dY.clone()
    dY_inf[t_inf, 0] = float("inf")
    dYg, Wg = dY_inf.cuda(), W_big.cuda()
    dX = torch.empty((T, d_in), dtype=torch.bfloat16, device="cuda")
    forge.forge_input_grad(dYg, Wg[:d_out], dX)
    torch.cuda.synchronize()
    got = bits(dX)
    rows = [t for t in range(T) if t != t_inf]
    assert np.isfinite(oracle.bf16_bits_to_f64(got[rows])).all(), "a non-finite value leaked across rows"
    check_dx(got[rows], [(bits(dY)[rows], bits(W_big[:d_out]))])
    # the row holding the Inf gets Inf * W[0, :] (W finite and mostly non-zero)
    assert np.isinf(oracle.bf16_bits_to_f64(got[t_inf])).sum() >= d_in // 2


def same(x, y):
    """Bitwise equality of two device tensors of one dtype."""
    return torch.equal(x.contiguous().view(torch.uint8), y.contiguous().view(torch.uint8))


def _gpu_state(p):
    st = [dev(a) for a in (p.X, p.dY, p.W, p.m, p.v)]
    st += [dev(p.m_scale), dev(p.v_scale)] if p.m_scale is not None else [None, None]
    return st


@pytest.mark.parametrize("moment", ["f32", "bf16", "i8", "i8r64"])
def test_backward_equals_input_grad_then_step_bitwise(moment):
    p = make_problem(300, 392, 520, moment, seed=41)
    T, d_in, d_out = p.shape
    a = _gpu_state(p)
    b = [t.clone() if t is not None else None for t in a]
    dX_a = torch.empty((T, d_in), dtype=torch.bfloat16, device="cuda")
    dX_b = torch.empty_like(dX_a)
    forge.forge_linear_backward(*a, dX=dX_a, step=7, **p.hp)
    forge.forge_input_grad(b[1], b[2], dX_b)
    forge.forge_linear_step(*b, step=7, **p.hp)
    torch.cuda.synchronize()
    assert same(dX_a, dX_b)
    for x, y in zip(a[2:], b[2:]):
        if x is not None:
            assert same(x, y)
    # the weight did change, so dX really came from the pre-update W
    assert not torch.equal(a[2], dev(p.W))


@pytest.mark.parametrize("moment", ["f32", "bf16", "i8", "i8r64"])
def test_backward_matches_oracle(moment):
    p = make_problem(256, 264, 328, moment, seed=42)
    T, d_in, d_out = p.shape
    ora = run_oracle(p, 100)
    g = _gpu_state(p)
    dX = torch.empty((T, d_in), dtype=torch.bfloat16, device="cuda")
    forge.forge_linear_backward(*g, dX=dX, step=100, **p.hp)
    torch.cuda.synchronize()
    _say(check_dx(bits(dX), [(p.dY, p.W)]))
    out = dict(W=bits(g[2]), m=bits(g[3]), v=bits(g[4]))
    if g[5] is not None:
        out.update(m_scale=bits(g[5]), v_scale=bits(g[6]))
    _say(check_step(out, ora, moment, hp=p.hp))


def _qkv(moment, T=200, d_in=264, outs=(264, 72, 72), seed=50):
    """Projections of one input X: per member (X, dY, W, m, v[, scales]) on the host (bits)."""
    X = _rand((T, d_in), 1.0, 1000 * seed + 1)
    mats = []
    for i, d_out in enumerate(outs):
        p = make_problem(T, d_in, d_out, moment, seed=seed + 1 + i)
        p.X = bits(X)
        mats.append(p)
    return mats


@pytest.mark.parametrize("moment", ["bf16", "i8", "i8r64"])
def test_backward_grouped_sums_projections_of_one_input(moment):
    ps = _qkv(moment)
    T, d_in = ps[0].X.shape
    Xg = dev(ps[0].X)
    A, B = [], []
    for p in ps:
        st = _gpu_state(p)
        st[0] = Xg
        A.append(tuple(t for t in st if t is not None))
        B.append(tuple(t.clone() if t is not Xg else Xg for t in A[-1]))
    dX = torch.full((T, d_in), float("nan"), dtype=torch.bfloat16, device="cuda")
    forge.forge_linear_backward_grouped(A, dX=dX, step=5, **HP)
    forge.forge_linear_step_grouped(B, step=5, **HP)
    torch.cuda.synchronize()
    _say(check_dx(bits(dX), [(p.dY, p.W) for p in ps]))
    for a, b in zip(A, B):
        for x, y in zip(a[2:], b[2:]):
            assert same(x, y)
    # and the state against the oracle, member by member
    for p, a in zip(ps, A):
        ora = run_oracle(p, 5)
        out = dict(W=bits(a[2]), m=bits(a[3]), v=bits(a[4]))
        if len(a) > 5:
            out.update(m_scale=bits(a[5]), v_scale=bits(a[6]))
        check_step(out, ora, moment, hp=p.hp)


def test_backward_grouped_with_empty_member_and_zero_tokens():
    ps = _qkv("bf16", outs=(136, 64), seed=60)
    T, d_in = ps[0].X.shape
    Xg = dev(ps[0].X)
    mats = []
    for p in ps:
        st = _gpu_state(p)
        mats.append((Xg,) + tuple(st[1:5]))
    empty = (Xg, torch.empty((T, 0), dtype=torch.bfloat16, device="cuda"),
             torch.empty((0, d_in), dtype=torch.bfloat16, device="cuda"),
             torch.empty((0, d_in), dtype=torch.bfloat16, device="cuda"),
             torch.empty((0, d_in), dtype=torch.bfloat16, device="cuda"))
    dX = torch.empty((T, d_in), dtype=torch.bfloat16, device="cuda")
    forge.forge_linear_backward_grouped([mats[0], empty, mats[1]], dX=dX, step=3, **HP)
    torch.cuda.synchronize()
    check_dx(bits(dX), [(p.dY, p.W) for p in ps])
    # T = 0: no dX, and the zero-gradient step equals forge_linear_step's
    p = make_problem(0, 136, 72, "bf16", seed=61)
    a = _gpu_state(p)
    b = [t.clone() for t in a[:5]]
    forge.forge_linear_backward(*a[:5], dX=torch.empty((0, 136), dtype=torch.bfloat16, device="cuda"), step=3, **HP)
    forge.forge_linear_step(*b, step=3, **HP)
    torch.cuda.synchronize()
    for x, y in zip(a[2:5], b[2:5]):
        assert same(x, y)
