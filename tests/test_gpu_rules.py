"""GPU parity of the fused step with the other update rules (forge_linear_step_opt).

Each rule of the optimizer-family table (SGD, SGD with momentum, Adagrad, RMSprop, Lion,
NAdam, RAdam, Adamax) and Muon's momentum accumulate runs in the fused kernel's epilogue
on fp32 and bf16 state and is compared with the oracle (exact fp64 G, then the rule in
fp64), with the bar of the AdamW tests and the per-rule state windows of compare.py.
"""
import numpy as np
import pytest
import torch

import oracle
from compare import check_rule_step
from gpu_util import bits, dev, gemm_error_bound
from paper_2606_22932_amd import forge, synth

pytestmark = pytest.mark.gpu

RULES = {"sgd": oracle.OPT_SGD, "sgd_momentum": oracle.OPT_SGD_MOMENTUM, "adagrad": oracle.OPT_ADAGRAD,
         "rmsprop": oracle.OPT_RMSPROP, "lion": oracle.OPT_LION, "nadam": oracle.OPT_NADAM,
         "radam": oracle.OPT_RADAM, "adamax": oracle.OPT_ADAMAX, "muon_accumulate": oracle.OPT_MUON}

# The shared protocol of the family table (betas, eps, weight decay), with learning rates
# large enough that every update moves W by about a bf16 ulp or more.
HP = {
    "sgd": dict(lr=0.5, weight_decay=1e-2),
    "sgd_momentum": dict(lr=0.5, beta1=0.9, weight_decay=1e-2),
    "adagrad": dict(lr=1e-3, eps=1e-10, weight_decay=1e-2, lr_decay=0.01),
    "rmsprop": dict(lr=1e-3, beta2=0.99, eps=1e-8, weight_decay=1e-2),
    "lion": dict(lr=1e-3, beta1=0.9, beta2=0.99, weight_decay=1.0),
    "nadam": dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=1e-2, momentum_decay=0.004),
    "radam": dict(lr=1e-2, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=1e-2),
    "adamax": dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=1e-2),
    "muon_accumulate": dict(lr=0.0, beta1=0.95),
}


def _say(*a):
    print(*a, flush=True)


def _states(name, shape, seed, dtype):
    """Warm states of the rule's kind: signed first-moment-like, positive second-moment-like."""
    signed = synth.gaussian(shape, 1e-3, seed + 3, dtype=torch.float32)
    positive = synth.gaussian(shape, 1e-4, seed + 4, dtype=torch.float32, absolute=True)
    if name in ("adagrad", "rmsprop"):
        s1, s2 = positive, None
    elif name in ("nadam", "radam", "adamax"):
        s1, s2 = signed, positive
    elif name == "sgd":
        s1 = s2 = None
    else:
        s1, s2 = signed, None
    cast = (lambda t: t) if dtype == "f32" else (lambda t: t.to(torch.bfloat16))
    return tuple(cast(t) if t is not None else None for t in (s1, s2))


def run_rule(name, T, d_in, d_out, kind, step, seed=300):
    base = 1000 * seed
    X = synth.gaussian((T, d_in), 1.0, base + 1)
    dY = synth.gaussian((T, d_out), 1e-3, base + 11)
    W = synth.gaussian((d_out, d_in), 0.02, base + 2)
    s1, s2 = _states(name, (d_out, d_in), base, kind)
    hp = HP[name]
    opt = RULES[name]
    h = lambda t: bits(t) if t is not None else None
    G = oracle.wgrad(bits(X), bits(dY))
    EG = gemm_error_bound(bits(X), bits(dY))
    sdt = oracle.MOMENT_F32 if kind == "f32" else oracle.MOMENT_BF16
    ora = oracle.rule_step(G, bits(W), h(s1), h(s2), opt=opt, state_dtype=sdt, step=step, **hp)
    # the oracle's W' at the ends of the interval the kernel's fp32 G lies in
    W_at = lambda sign: oracle.rule_step(G + sign * EG, bits(W), h(s1), h(s2), opt=opt, state_dtype=sdt,
                                         step=step, **hp)["W64"]
    g = [dev(bits(t)) if t is not None else None for t in (X, dY, W, s1, s2)]
    forge.forge_linear_step_opt(g[0], g[1], None if name == "muon_accumulate" else g[2], g[3], g[4],
                                optimizer=name, step=step, **hp)
    torch.cuda.synchronize()
    gpu = dict(W=bits(g[2]), s1=h(g[3]), s2=h(g[4]))
    W64 = oracle.bf16_bits_to_f64(bits(W))
    to64 = lambda t: (oracle.bf16_bits_to_f64(bits(t)) if t.dtype == torch.bfloat16 else bits(t).astype(np.float64)) \
        if t is not None else None
    return check_rule_step(gpu, ora, opt, kind, hp, G, EG, W64, to64(s1), to64(s2), W_at=W_at)


SHAPES = [(77, 328, 200), (256, 264, 520)]


@pytest.mark.parametrize("kind", ["f32", "bf16"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("name", list(RULES))
def test_rule_matches_oracle(name, shape, kind):
    _say(f"{name} {shape} {kind}")
    _say(run_rule(name, *shape, kind, step=100))


@pytest.mark.parametrize("kind", ["bf16", "f32"])
@pytest.mark.parametrize("name", list(RULES))
def test_rule_full_size_o_proj(name, kind):
    """Every element of the Llama-3.1-8B o_proj shape (T=512, 4096 x 4096, bf16 or fp32
    state): the full tile grid of the single-layer configuration, not only a few tiles, and
    for fp32 state every pass of the prefetch (four passes loaded during the mainloop, the
    rest four passes ahead in the epilogue)."""
    _say(f"{name} full size 512x4096x4096 {kind}")
    _say(run_rule(name, 512, 4096, 4096, kind, step=100, seed=302))


@pytest.mark.parametrize("name", ["adagrad", "nadam", "radam", "adamax"])
def test_rule_first_step(name):
    """Step 1: Adagrad's undecayed rate, NAdam's first schedule terms, RAdam's unrectified
    branch (rho_1 < 5) and the bias corrections at their largest."""
    _say(run_rule(name, 128, 136, 264, "f32", step=1, seed=301))


def test_adamw_through_rule_entry_point_equals_forge_linear_step():
    T, d_in, d_out = 200, 264, 392
    X = synth.gaussian((T, d_in), 1.0, 401, device="cuda")
    dY = synth.gaussian((T, d_out), 1e-3, 411, device="cuda")
    W = synth.gaussian((d_out, d_in), 0.02, 402, device="cuda")
    for dt in (torch.float32, torch.bfloat16):
        m = synth.gaussian((d_out, d_in), 1e-4, 403, device="cuda", dtype=dt)
        v = synth.gaussian((d_out, d_in), 1e-6, 404, device="cuda", dtype=dt, absolute=True)
        a = [W.clone(), m.clone(), v.clone()]
        b = [W.clone(), m.clone(), v.clone()]
        hp = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.1)
        forge.forge_linear_step_opt(X, dY, *a, optimizer="adamw", step=9, **hp)
        forge.forge_linear_step(X, dY, *b, step=9, **hp)
        torch.cuda.synchronize()
        for x, y in zip(a, b):
            assert torch.equal(x.view(torch.uint8), y.view(torch.uint8))


def test_muon_accumulate_over_micro_batches():
    """beta = mu on the first micro-batch and 1 on the second gives mu B + G of all tokens,
    within the fp32 accumulation bound of the two partial gradients."""
    T, d_in, d_out = 192, 264, 136
    X = synth.gaussian((T, d_in), 1.0, 501, device="cuda")
    dY = synth.gaussian((T, d_out), 1e-3, 511, device="cuda")
    B0 = synth.gaussian((d_out, d_in), 1e-3, 503, device="cuda", dtype=torch.float32)
    B = B0.clone()
    forge.forge_linear_step_opt(X[:80].contiguous(), dY[:80].contiguous(), None, B, optimizer="muon_accumulate",
                                lr=0.0, beta1=0.95, step=1)
    forge.forge_linear_step_opt(X[80:].contiguous(), dY[80:].contiguous(), None, B, optimizer="muon_accumulate",
                                lr=0.0, beta1=1.0, step=1)
    torch.cuda.synchronize()
    want = float(np.float32(0.95)) * bits(B0).astype(np.float64) + oracle.wgrad(bits(X), bits(dY))
    bound = gemm_error_bound(bits(X), bits(dY)) + 2 ** -22 * np.abs(want) + 2 ** -23 * np.abs(bits(B0))
    err = np.abs(bits(B).astype(np.float64) - want)
    assert (err <= bound).all(), float((err / bound).max())
