"""GPU parity: the HIP path through the C ABI against the CPU oracle, element by element.

Sizes span several tiles with ragged tails on every axis; the full-size workloads (the
Llama-3.1-8B o_proj and MLP projections at T=512) are checked on every element.
"""
import numpy as np
import pytest
import torch

import oracle
from compare import bf16_f64, bf16_key, check_moment, check_step, check_weight
from gpu_util import Problem, bits, dev, gemm_error_bound, make_problem, run_gpu, run_oracle, with_state
from paper_2606_22932_amd import forge, synth

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)


# (T, d_in, d_out): several tiles, ragged tiles on both axes, ragged token chunks,
# the empty token axis and the smallest legal shape; long token axes, where the int8
# column-block kernel walks its tiles in raster groups of 2 and of 1 tile rows (a group's
# dY slabs are kept near 2 MB).
SMALL = [
    (128, 256, 256),
    (77, 328, 200),
    (33, 136, 264),
    (1, 8, 8),
    (0, 64, 32),
    (512, 384, 520),
    (200, 1032, 776),
    (2048, 200, 1032),
    (4100, 136, 776),
]


@pytest.mark.parametrize("moment", ["f32", "bf16", "i8", "i8r64"])
@pytest.mark.parametrize("shape", SMALL, ids=lambda s: "x".join(map(str, s)))
def test_fused_matches_oracle(moment, shape):
    T, d_in, d_out = shape
    _say(f"fused {moment} T={T} d_in={d_in} d_out={d_out}")
    p = make_problem(T, d_in, d_out, moment, seed=T + d_in + d_out, warm=True)
    for step in (1, 100):
        ora = run_oracle(p, step)
        gpu = run_gpu(p, step)
        _say(check_step(gpu, ora, moment, hp=p.hp))


def test_cold_start_step1_closed_form_on_gpu():
    """From zero state at t=1 the update is -lr*g/(|g|+eps): W moves against sign(G)."""
    p = make_problem(64, 256, 128, "f32", seed=5, warm=False, dy_std=0.01)
    gpu = run_gpu(p, 1)
    ora = run_oracle(p, 1)
    check_step(gpu, ora, "f32", hp=p.hp)
    G = ora["G"]
    W0 = bf16_f64(p.W)
    Wn = bf16_f64(gpu["W"])
    moved = (1 - np.float32(1e-3) * np.float32(0.1)) * W0 - Wn
    big = np.abs(G) > 1e-6
    assert np.mean(np.sign(moved[big]) == np.sign(G[big])) > 0.999


def test_layer256_three_steps():
    """T=128, 256x256, fp32 moments from zero, steps 1..3 with a fresh dY each step.

    Teacher-forced: each step starts from the oracle's stored state (strict bar).
    Free-running: each side carries its own state (reported; W within 1 ulp on 99.5%).
    """
    wl = synth.WORKLOADS["layer256"]
    mat = wl.matrices[0]
    X0, _ = synth.activations(wl.T, mat, wl, 1)
    W0 = synth.weight(mat, wl)
    m0, v0 = synth.warm_moments(mat, wl)
    st_o = dict(W=bits(W0), m=bits(m0), v=bits(v0))
    st_g = dict(st_o)
    for t in wl.steps:
        _, dY = synth.activations(wl.T, mat, wl, t)
        base = Problem(bits(X0), bits(dY), None, None, None, "f32", hp=dict(wl.hyper))
        p_o = with_state(base, st_o)
        ora = run_oracle(p_o, t)
        gpu_tf = run_gpu(p_o, t)
        _say("teacher-forced step", t, check_step(gpu_tf, ora, "f32", hp=p_o.hp))
        gpu_fr = run_gpu(with_state(base, st_g), t)
        st_o = dict(W=ora["W"], m=ora["m"], v=ora["v"])
        st_g = gpu_fr
    _say("free-running after 3 steps", check_weight(st_g["W"], st_o["W"], frac=0.995))
    check_moment(st_g["m"], st_o["m"], st_o["m"].astype(np.float64), "f32", "m")


def _full_matrix(wl_name, idx, step=100):
    wl = synth.WORKLOADS[wl_name]
    mat = wl.matrices[idx]
    _say(f"{wl_name}:{mat.name} [{mat.d_out}x{mat.d_in}] T={wl.T}")
    X, dY = synth.activations(wl.T, mat, wl, step)
    W = synth.weight(mat, wl)
    m, v = synth.warm_moments(mat, wl)
    p = Problem(bits(X), bits(dY), bits(W), None, None, wl.moment, hp=dict(wl.hyper))
    if wl.moment == "bf16":
        p.m, p.v = bits(m.to(torch.bfloat16)), bits(v.to(torch.bfloat16))
    elif wl.moment == "i8r64":
        p.m, p.m_scale = oracle.quantize_i8_row64(m.double().numpy(), second_moment=False)
        p.v, p.v_scale = oracle.quantize_i8_row64(v.double().numpy(), second_moment=True)
    else:
        p.m, p.m_scale = oracle.quantize_i8(m.double().numpy(), False)
        p.v, p.v_scale = oracle.quantize_i8(v.double().numpy(), True)
    gpu = run_gpu(p, step)
    ora = run_oracle(p, step)
    _say(check_step(gpu, ora, wl.moment, hp=p.hp))


def test_o_proj_full():
    _full_matrix("o_proj", 0)


def test_o_proj_t4096_full():
    """Every element of the o_proj shape at T = 4096 (128 token chunks per tile), the
    compute-bound regime that bench.py times beside the sweep."""
    _full_matrix("o_proj_t4096", 0)


@pytest.mark.parametrize("idx", [0, 1, 2], ids=["gate", "up", "down"])
def test_mlp_bf16_full(idx):
    _full_matrix("mlp", idx)


@pytest.mark.parametrize("idx", [0, 1, 2], ids=["gate", "up", "down"])
def test_mlp_int8_full(idx):
    _full_matrix("mlp_i8", idx)


@pytest.mark.parametrize("idx", [0, 1, 2], ids=["gate", "up", "down"])
def test_mlp_int8_rows_full(idx):
    """The paper's own int8 layout (one scale per 64 elements of a row) on every element of
    the MLP projections, the shapes bench.py times it on."""
    _full_matrix("mlp_i8r64", idx)


@pytest.mark.parametrize("moment", ["f32", "bf16", "i8", "i8r64"])
def test_unfused_fp32_gradient_matches_oracle(moment):
    p = make_problem(96, 392, 264, moment, seed=17)
    ora = run_oracle(p, 9)
    gpu = run_gpu(p, 9, path="unfused", grad="f32")
    _say(check_step(gpu, ora, moment, hp=p.hp))


def _gemm_error_bound(p):
    """Worst-case fp32 accumulation error of G in any order (plus an absolute floor)."""
    return gemm_error_bound(p.X, p.dY) + 1e-30


def _near_bf16_midpoint(G64, bound):
    """Elements whose bf16 rounding can be decided either way within `bound`."""
    k = np.abs(G64).astype(np.float32).view(np.uint32)
    lo = (k & 0xFFFF0000).view(np.float32).astype(np.float64)
    hi = ((k & 0xFFFF0000) + 0x10000).view(np.float32).astype(np.float64)
    mid = 0.5 * (lo + hi)
    return np.abs(np.abs(G64) - mid) <= bound


@pytest.mark.parametrize("moment", ["bf16", "i8", "i8r64"])
def test_unfused_bf16_gradient_matches_rounded_oracle(moment):
    """The two-kernel path with a bf16 gradient buffer equals the oracle that rounds G to
    bf16 first (App. B truncation), except where G sits on a bf16 rounding midpoint."""
    p = make_problem(96, 392, 264, moment, seed=19)
    ora = run_oracle(p, 9, round_grad_to_bf16=True)
    gpu = run_gpu(p, 9, path="unfused", grad="bf16")
    exempt = _near_bf16_midpoint(ora["G"], _gemm_error_bound(p))
    _say(f"near-midpoint gradients exempted: {int(exempt.sum())} of {exempt.size}")
    # the worst-case bound is loose (T 2^-24 sum|terms|), so a few percent sit in its window
    assert exempt.mean() < 0.10
    if moment in ("i8", "i8r64"):
        # a flipped gradient rounding moves a whole block's codes at most by a tie; check W only
        keep = ~exempt
        ulps = np.abs(bf16_key(gpu["W"]) - bf16_key(ora["W"]))[keep]
        assert (ulps <= 1).mean() >= 0.999
        return
    for k in ("W", "m", "v"):
        gpu[k] = np.where(exempt, ora[k], gpu[k])
    _say(check_step(gpu, ora, moment, hp=p.hp))


def test_wgrad_store_gradient():
    p = make_problem(200, 264, 136, "bf16", seed=23)
    G64 = oracle.wgrad(p.X, p.dY)
    bound = _gemm_error_bound(p)
    X, dY = dev(p.X), dev(p.dY)
    G32 = torch.empty((136, 264), dtype=torch.float32, device="cuda")
    G16 = torch.empty((136, 264), dtype=torch.bfloat16, device="cuda")
    forge.forge_wgrad(X, dY, G32)
    forge.forge_wgrad(X, dY, G16)
    torch.cuda.synchronize()
    g32 = G32.cpu().double().numpy()
    assert np.all(np.abs(g32 - G64) <= bound)
    g16 = bits(G16)
    want = oracle.f64_to_bf16_bits(G64)
    ok = (g16 == want) | _near_bf16_midpoint(G64, bound)
    assert ok.all()


def test_deterministic_bitwise():
    """No atomics and a fixed summation order: two runs agree bit for bit (cf. App. A FP remark)."""
    for moment in ("bf16", "i8"):
        p = make_problem(256, 512, 512, moment, seed=29)
        a, b = run_gpu(p, 50), run_gpu(p, 50)
        for k in a:
            assert np.array_equal(a[k], b[k]), (moment, k)


def test_stream_argument_is_honoured():
    p = make_problem(64, 256, 256, "bf16", seed=31)
    s = torch.cuda.Stream()
    X, dY, W, m, v = (dev(x) for x in (p.X, p.dY, p.W, p.m, p.v))
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        forge.forge_linear_step(X, dY, W, m, v, step=3, **p.hp)
    s.synchronize()
    ora = run_oracle(p, 3)
    check_step(dict(W=bits(W), m=bits(m), v=bits(v)), ora, "bf16", hp=p.hp)


def _state_on_gpu(p):
    st = [dev(a) for a in (p.W, p.m, p.v)]
    sc = [dev(p.m_scale), dev(p.v_scale)] if p.m_scale is not None else [None, None]
    return st + sc


@pytest.mark.parametrize("moment", ["f32", "bf16", "i8", "i8r64"])
def test_grouped_matches_oracle_and_single_calls(moment):
    """forge_linear_step_grouped: every matrix as the oracle has it, and bit-identical to
    a separate forge_linear_step call on that matrix (Def. 1: tiles are independent)."""
    T = 77
    shapes = [(328, 200), (136, 264), (8, 8), (1032, 776), (392, 520)]
    probs = [make_problem(T, d_in, d_out, moment, seed=40 + i) for i, (d_in, d_out) in enumerate(shapes)]
    _say(f"grouped {moment}: {len(probs)} matrices, T={T}")
    group, single = [], []
    for p in probs:
        X, dY = dev(p.X), dev(p.dY)
        W, m, v, ms, vs = _state_on_gpu(p)
        group.append((X, dY, W, m, v, ms, vs))
        W2, m2, v2, ms2, vs2 = _state_on_gpu(p)
        forge.forge_linear_step(X, dY, W2, m2, v2, ms2, vs2, step=100, **p.hp)
        single.append((W2, m2, v2, ms2, vs2))
    forge.forge_linear_step_grouped(group, step=100, **probs[0].hp)
    torch.cuda.synchronize()
    for p, g, s1 in zip(probs, group, single):
        out = dict(W=bits(g[2]), m=bits(g[3]), v=bits(g[4]))
        if moment in ("i8", "i8r64"):
            out.update(m_scale=bits(g[5]), v_scale=bits(g[6]))
        _say(check_step(out, run_oracle(p, 100), moment, hp=p.hp))
        for a, b in zip(g[2:], s1):
            if a is not None:
                assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), "grouped != single call"


def test_grouped_shared_input_and_empty_member():
    """q, k, v style: three matrices read the same X; an empty matrix in the group is skipped."""
    T, d_in = 96, 264
    X = synth.gaussian((T, d_in), 1.0, 5101, device="cuda")
    members, probs = [], []
    for i, d_out in enumerate((392, 136, 136)):
        dY = synth.gaussian((T, d_out), 1e-3, 5111 + i, device="cuda")
        W = synth.gaussian((d_out, d_in), 0.02, 5121 + i, device="cuda")
        m = synth.gaussian((d_out, d_in), 1e-4, 5131 + i, device="cuda")
        v = synth.gaussian((d_out, d_in), 1e-6, 5141 + i, device="cuda", absolute=True)
        probs.append(Problem(bits(X), bits(dY), bits(W), bits(m), bits(v), "bf16"))
        members.append((X, dY, W, m, v))
    e = torch.empty((0, d_in), dtype=torch.bfloat16, device="cuda")
    members.insert(1, (X, torch.empty((T, 0), dtype=torch.bfloat16, device="cuda"), e, e.clone(), e.clone()))
    forge.forge_linear_step_grouped(members, step=7, **probs[0].hp)
    torch.cuda.synchronize()
    for p, (_, _, W, m, v) in zip(probs, [members[0], members[2], members[3]]):
        _say(check_step(dict(W=bits(W), m=bits(m), v=bits(v)), run_oracle(p, 7), "bf16", hp=p.hp))


def test_long_launch_prefetch_depth_bitwise():
    """A launch of at least 8 waves of resident tiles (4096 tiles of 128x128 on 256 CUs)
    prefetches all eight row passes of a tile's state, a shorter one six (at T < 1024; from
    T = 1024 every launch takes eight, which the T = 4096 tests cover).  The depth changes
    when loads are issued, not what is computed: four o_proj-sized matrices in one grouped
    launch (4096 tiles) give the bits of four single launches (1024 tiles each), and the
    first is checked against the oracle on every element."""
    T, d = 512, 4096
    probs = [make_problem(T, d, d, "bf16", seed=70 + k) for k in range(4)]
    _say(f"long launch: 4 x {d}x{d}, T={T}")
    group, single = [], []
    for p in probs:
        X, dY = dev(p.X), dev(p.dY)
        W, m, v, _, _ = _state_on_gpu(p)
        group.append((X, dY, W, m, v))
        W2, m2, v2, _, _ = _state_on_gpu(p)
        forge.forge_linear_step(X, dY, W2, m2, v2, step=100, **p.hp)
        single.append((W2, m2, v2))
    forge.forge_linear_step_grouped(group, step=100, **probs[0].hp)
    torch.cuda.synchronize()
    for g, s1 in zip(group, single):
        for a, b in zip(g[2:], s1):
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), "long launch != short launches"
    g = group[0]
    _say(check_step(dict(W=bits(g[2]), m=bits(g[3]), v=bits(g[4])), run_oracle(probs[0], 100), "bf16",
                    hp=probs[0].hp))


@pytest.mark.parametrize("shape", [(512, 520, 776), (77, 328, 264), (0, 64, 256)], ids=lambda s: "x".join(map(str, s)))
def test_int8_fused_equals_unfused_fp32_gradient_bitwise(shape):
    """The fused int8 step and the two-kernel step through an fp32 G accumulate every
    element of G in the same order and share the epilogue arithmetic: identical bits."""
    T, d_in, d_out = shape
    p = make_problem(T, d_in, d_out, "i8", seed=77 + T)
    a = run_gpu(p, 100)
    b = run_gpu(p, 100, path="unfused", grad="f32")
    for k in ("W", "m", "v", "m_scale", "v_scale"):
        assert np.array_equal(a[k].view(np.uint8), b[k].view(np.uint8)), k


# Exact half-integers through the kernel's int8 quantiser (App. B's "round", read as round
# half to even): beta1 = beta2 = 0 makes m' = G exactly, and one token with a unit input
# side puts the values below into one int8 block whose absmax is 127, so its scale is 1
# and every quotient is its value.
TIE_VALUES = [127.0, 0.5, 1.5, 2.5, 3.5, -0.5, -1.5, -2.5, -3.5, 126.5, -126.5, 4.5, -4.5, 0.0, 1.0]
TIE_CODES_EVEN = [127, 0, 2, 2, 4, 0, -2, -2, -4, 126, -126, 4, -4, 0, 1]


@pytest.mark.parametrize("moment", ["i8", "i8r64"])
def test_int8_exact_ties_round_half_even(moment):
    n = len(TIE_VALUES)
    ties = np.array(TIE_VALUES)
    if moment == "i8":                        # a 256-row block of each column: G[p, q] = dY[0, p]
        d_in, d_out = 64, 256
        X, dY = np.ones((1, d_in)), np.zeros((1, d_out))
        dY[0, :n] = ties
        zeros = np.zeros((d_out, d_in))
        m, ms = oracle.quantize_i8(zeros, False)
        v, vs = oracle.quantize_i8(zeros, True)
    else:                                     # a 64-wide block of each row: G[p, q] = X[0, q]
        d_in, d_out = 64, 8
        X, dY = np.zeros((1, d_in)), np.ones((1, d_out))
        X[0, :n] = ties
        zeros = np.zeros((d_out, d_in))
        m, ms = oracle.quantize_i8_row64(zeros, False)
        v, vs = oracle.quantize_i8_row64(zeros, True)
    b16 = lambda a: oracle.f64_to_bf16_bits(a)
    assert np.array_equal(oracle.bf16_bits_to_f64(b16(ties)), ties)
    hp = dict(lr=1e-3, beta1=0.0, beta2=0.0, eps=1e-8, weight_decay=0.1)
    p = Problem(b16(X), b16(dY), b16(zeros), m, v, moment, ms, vs, hp=hp)
    ora = run_oracle(p, 1)
    gpu = run_gpu(p, 1)
    _say(check_step(gpu, ora, moment, hp=hp))
    assert np.array_equal(gpu["m"], ora["m"]), "m codes differ from the oracle at exact ties"
    got = gpu["m"][:n, :] if moment == "i8" else gpu["m"][:, :n].T
    assert (got == np.array(TIE_CODES_EVEN)[:, None]).all()
    assert (gpu["m_scale"] == 1.0).all()


# The fused bf16 step (one workgroup per 128x128 tile, two resident per CU) against the
# two-kernel path (the store-G GEMM, then the stand-alone optimizer).  Shapes: fewer tiles
# than CUs, ragged edges on both axes, ragged token chunks, the empty token axis, and the
# o_proj shape (1024 tiles, two waves of resident workgroups).
BITWISE = [(512, 520, 776), (77, 1032, 2056), (33, 8, 8), (0, 264, 1032), (1024, 520, 392),
           (512, 4096, 4096)]


@pytest.mark.parametrize("shape", BITWISE, ids=lambda s: "x".join(map(str, s)))
def test_bf16_fused_equals_unfused_fp32_gradient_bitwise(shape):
    """The fused bf16 step and the two-kernel step through an fp32 G accumulate every
    element of G in the same order and share the AdamW arithmetic: identical bits."""
    T, d_in, d_out = shape
    p = make_problem(T, d_in, d_out, "bf16", seed=91 + T)
    _say(f"fused vs unfused: T={T} d_in={d_in} d_out={d_out}")
    a = run_gpu(p, 100)
    b = run_gpu(p, 100, path="unfused", grad="f32")
    for k in ("W", "m", "v"):
        assert np.array_equal(a[k].view(np.uint8), b[k].view(np.uint8)), k


def test_bf16_grouped_mixed_shapes_bitwise():
    """A grouped launch of matrices of different shapes gives the bits of the matrices
    stepped one by one through the two-kernel path."""
    T = 300
    shapes = [(T, 264, 136), (T, 1032, 520), (T, 128, 8), (T, 520, 1160)]
    probs = [make_problem(*s, "bf16", seed=140 + k) for k, s in enumerate(shapes)]
    group = []
    for p in probs:
        X, dY = dev(p.X), dev(p.dY)
        W, m, v, _, _ = _state_on_gpu(p)
        group.append((X, dY, W, m, v))
    forge.forge_linear_step_grouped(group, step=100, **probs[0].hp)
    torch.cuda.synchronize()
    for g, p in zip(group, probs):
        b = run_gpu(p, 100, path="unfused", grad="f32")
        for k, t in zip(("W", "m", "v"), g[2:]):
            assert np.array_equal(bits(t).view(np.uint8), b[k].view(np.uint8)), k
