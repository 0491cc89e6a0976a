"""The numerical-fidelity experiment of App. E (and Sec. 3.1) on the GPU path.

Twenty optimizer steps of one [V, H] = [1024, 4096] weight at BT = 2048 tokens, with
identical seeded inputs in every arm, each arm's weight compared after the last step with
two references, both from the oracle's exact fp64 gradient:
* unrounded   Algorithm 1 with no storage rounding at all (fp64 W, m, v carried across
              steps; the paper compares against an fp32 reference, which this reads as);
* same-storage  the oracle's step with the arm's own storage (bf16 W, the arm's moment
              type), so that what remains is the gradient the arm's optimizer read.
Metrics: rms-rel(W) = rms(W_arm - W_ref) / rms(W_ref), and max |W_arm - W_ref|.  Against
the unrounded reference all bf16-weight arms share the random walk of rounding W each
step (updates of several ulps at lr 1e-3), which dominates; against the same-storage
reference only the gradient's path differs.

Arms (W is bf16 in all of them):
* fused         forge_linear_step (G stays in fp32 registers), fp32 or bf16 moments
* standard      the two-kernel path with the gradient stored as bf16 (the common
                bf16 pipeline), fp32 or bf16 moments
* decomposed    the two-kernel path with an fp32 gradient: the control that differs from
                the fused arm only in where G lives, not in its value
* int8          forge_linear_step with int8 block-absmax moments: 256-row column blocks
                with sqrt(v) stored, and the paper's 64-wide row blocks with v stored

The paper's claim checked here: the fused arm's rms weight error is below the standard
arm's, because the standard arm rounds every gradient to bf16 before the moments read it
(App. B: that truncation passes through the moving averages undamped), and the fp32-G
control matches the fused arm.  Inputs: X ~ N(0, 1), dY ~ N(0, 1e-3) per step,
W0 ~ N(0, 0.02), cold moments, AdamW lr 1e-3, betas (0.9, 0.999), eps 1e-8, wd 0.1.

Run with -s to see the table (it is also written to gpurun_out/fidelity_app_e.json when
that folder exists).
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle
from gpu_util import bits
from paper_2606_22932_amd import forge, synth

pytestmark = pytest.mark.gpu

V, H, BT, STEPS = 1024, 4096, 2048, 20
HP = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.1)


def _say(*a):
    print(*a, flush=True)


def _inputs(step, device):
    X = synth.gaussian((BT, H), 1.0, 880_000 + 2 * step, device=device)
    dY = synth.gaussian((BT, V), 1e-3, 880_001 + 2 * step, device=device)
    return X, dY


def test_fidelity_twenty_steps():
    dev = torch.device("cuda:0")
    W0 = synth.gaussian((V, H), 0.02, 879_999, device=dev)

    def state(dt):
        if dt in ("i8", "i8r64"):
            z8 = torch.zeros((V, H), dtype=torch.int8, device=dev)
            shape = ((V + 255) // 256, H) if dt == "i8" else (V, (H + 63) // 64)
            zs = torch.zeros(shape, dtype=torch.float32, device=dev)
            return [W0.clone(), z8, z8.clone(), zs, zs.clone()]
        t = torch.float32 if dt == "f32" else torch.bfloat16
        z = torch.zeros((V, H), dtype=t, device=dev)
        return [W0.clone(), z, z.clone(), None, None]

    arms = {
        "fused_f32m": ("fused", "f32", None),
        "fused_bf16m": ("fused", "bf16", None),
        "standard_bf16G_f32m": ("unfused", "f32", torch.bfloat16),
        "standard_bf16G_bf16m": ("unfused", "bf16", torch.bfloat16),
        "decomposed_f32G_f32m": ("unfused", "f32", torch.float32),
        "fused_int8m": ("fused", "i8", None),
        "fused_int8r64m": ("fused", "i8r64", None),
    }
    st = {k: state(v[1]) for k, v in arms.items()}
    ws = {torch.bfloat16: torch.empty((V, H), dtype=torch.bfloat16, device=dev),
          torch.float32: torch.empty((V, H), dtype=torch.float32, device=dev)}

    Wr = oracle.bf16_bits_to_f64(bits(W0))
    mr = np.zeros((V, H))
    vr = np.zeros((V, H))
    # same-storage references: bf16 W and the arm's moment storage, exact G
    MK = {"f32": oracle.MOMENT_F32, "bf16": oracle.MOMENT_BF16, "i8": oracle.MOMENT_I8,
          "i8r64": oracle.MOMENT_I8_ROW64}
    zeros = {"f32": lambda: np.zeros((V, H), np.float32), "bf16": lambda: np.zeros((V, H), np.uint16),
             "i8": lambda: np.zeros((V, H), np.int8), "i8r64": lambda: np.zeros((V, H), np.int8)}
    sshape = {"i8": ((V + 255) // 256, H), "i8r64": (V, (H + 63) // 64)}
    ss = {dt: dict(W=bits(W0), m=zeros[dt](), v=zeros[dt](),
                   ms=np.zeros(sshape[dt], np.float32) if dt in sshape else None,
                   vs=np.zeros(sshape[dt], np.float32) if dt in sshape else None)
          for dt in ("f32", "bf16", "i8", "i8r64")}
    for t in range(1, STEPS + 1):
        X, dY = _inputs(t, dev)
        for k, (path, _, gdt) in arms.items():
            W, m, v, ms, vs = st[k]
            if path == "fused":
                forge.forge_linear_step(X, dY, W, m, v, ms, vs, step=t, **HP)
            else:
                forge.forge_linear_step_unfused(X, dY, W, m, v, ms, vs, G_ws=ws[gdt], step=t, **HP)
        G = oracle.wgrad(bits(X), bits(dY))
        Wr, mr, vr = oracle.adamw_f64(G, Wr, mr, vr, step=t, **HP)
        for dt, r in ss.items():
            o = oracle.adamw(G, r["W"], r["m"], r["v"], moment_dtype=MK[dt], step=t, m_scale=r["ms"],
                             v_scale=r["vs"], **HP)
            r.update(W=o["W"], m=o["m"], v=o["v"], ms=o["m_scale"], vs=o["v_scale"])
        torch.cuda.synchronize()
        _say(f"step {t} done")

    def metrics(W_bits, ref64):
        d = oracle.bf16_bits_to_f64(W_bits) - ref64
        return dict(rms_rel=float(np.sqrt(np.mean(d * d)) / np.sqrt(np.mean(ref64 * ref64))),
                    max_abs=float(np.abs(d).max()))

    table = {}
    for k, (_, dt, _) in arms.items():
        Wk = bits(st[k][0])
        table[k] = dict(vs_unrounded=metrics(Wk, Wr),
                        vs_same_storage=metrics(Wk, oracle.bf16_bits_to_f64(ss[dt]["W"])))
    # the floor of any bf16-weight arm against the unrounded reference: that reference
    # rounded once to bf16 at the end
    table["unrounded_reference_rounded_once"] = dict(vs_unrounded=metrics(oracle.f64_to_bf16_bits(Wr), Wr))
    out = dict(V=V, H=H, BT=BT, steps=STEPS, hyper=HP, arms=table)
    _say(json.dumps(out, indent=1))
    if os.path.isdir("gpurun_out"):
        with open("gpurun_out/fidelity_app_e.json", "w") as f:
            json.dump(out, f, indent=1)

    u = lambda k: table[k]["vs_unrounded"]["rms_rel"]
    s_ = lambda k: table[k]["vs_same_storage"]["rms_rel"]
    # Sec. 3.1 / App. E: the fused arm's weights are closer to the reference than the arm that
    # rounds G to bf16, at either moment precision and against either reference
    for mom in ("f32m", "bf16m"):
        assert u(f"fused_{mom}") < u(f"standard_bf16G_{mom}")
        assert s_(f"fused_{mom}") < 0.5 * s_(f"standard_bf16G_{mom}")
    # the fp32-G two-kernel control differs from the fused arm only in summation order
    assert abs(u("decomposed_f32G_f32m") - u("fused_f32m")) <= 0.01 * u("fused_f32m")
    assert s_("decomposed_f32G_f32m") < 0.5 * s_("standard_bf16G_f32m")
