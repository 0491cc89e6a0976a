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
* fp8           E4M3 moments with per-tensor delayed scales (App. E's fp8 mode), and fp8
                weights with bf16 or fp8 moments (Sec. 3's w and w+m recipes); fp8 weights
                start from W0 encoded with its own amax as the scale

The paper's claim checked here: the fused arm's rms weight error is below the standard
arm's, because the standard arm rounds every gradient to bf16 before the moments read it
(App. B: that truncation passes through the moving averages undamped), and the fp32-G
control matches the fused arm.  Inputs: X ~ N(0, 1), dY ~ N(0, 1e-3) per step,
W0 ~ N(0, 0.02), cold moments, AdamW lr 1e-3, betas (0.9, 0.999), eps 1e-8, wd 0.1.

Run with -s to see the table (it is also written as fidelity_app_e.json into the directory
that FORGE_RESULTS_DIR names, when that is set).
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

    a0 = np.float32(np.abs(oracle.bf16_bits_to_f64(bits(W0))).max())
    W0_codes = oracle.e4m3_encode(np.clip(oracle.bf16_bits_to_f64(bits(W0)).astype(np.float32) / (a0 / np.float32(448)),
                                          -448, 448))

    def w_ring0():
        r = np.zeros(4, np.float32)
        r[3] = r[0] = a0          # step 1 decodes with slot 3 and encodes with slot 0
        return r

    def fp8(a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint8)).view(torch.float8_e4m3fn).to(dev)

    def state(dt, wfp8=False):
        if wfp8:
            Wq = fp8(W0_codes)
            wr = torch.from_numpy(w_ring0()).to(dev)
            if dt == "fp8":
                z = fp8(np.zeros((V, H), np.uint8))
                return [Wq, z, fp8(np.zeros((V, H), np.uint8)), torch.zeros(4, device=dev), torch.zeros(4, device=dev), wr]
            z = torch.zeros((V, H), dtype=torch.bfloat16, device=dev)
            return [Wq, z, z.clone(), None, None, wr]
        if dt == "fp8":
            z = fp8(np.zeros((V, H), np.uint8))
            return [W0.clone(), z, fp8(np.zeros((V, H), np.uint8)), torch.zeros(4, device=dev),
                    torch.zeros(4, device=dev)]
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
        "fused_fp8m": ("fused", "fp8", None),
        "fused_fp8w_bf16m": ("wfp8", "bf16", None),
        "fused_fp8w_fp8m": ("wfp8", "fp8", None),
    }
    st = {k: state(v[1], wfp8=v[0] == "wfp8") for k, v in arms.items()}
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
    z8 = lambda: np.zeros((V, H), np.uint8)
    z16 = lambda: np.zeros((V, H), np.uint16)
    ss8 = {"fused_fp8m": dict(W=bits(W0), m=z8(), v=z8(), w8=False, m8=True, wr=None, mr=np.zeros(4, np.float32),
                              vr=np.zeros(4, np.float32)),
           "fused_fp8w_bf16m": dict(W=W0_codes.copy(), m=z16(), v=z16(), w8=True, m8=False, wr=w_ring0(), mr=None,
                                    vr=None),
           "fused_fp8w_fp8m": dict(W=W0_codes.copy(), m=z8(), v=z8(), w8=True, m8=True, wr=w_ring0(),
                                   mr=np.zeros(4, np.float32), vr=np.zeros(4, np.float32))}
    for t in range(1, STEPS + 1):
        X, dY = _inputs(t, dev)
        for k, (path, _, gdt) in arms.items():
            W, m, v, ms, vs = st[k][:5]
            if path == "fused":
                forge.forge_linear_step(X, dY, W, m, v, ms, vs, step=t, **HP)
            elif path == "wfp8":
                forge.forge_linear_step_wfp8(X, dY, W, st[k][5], m, v, ms, vs, step=t, **HP)
            else:
                forge.forge_linear_step_unfused(X, dY, W, m, v, ms, vs, G_ws=ws[gdt], step=t, **HP)
        G = oracle.wgrad(bits(X), bits(dY))
        Wr, mr, vr = oracle.adamw_f64(G, Wr, mr, vr, step=t, **HP)
        for dt, r in ss.items():
            o = oracle.adamw(G, r["W"], r["m"], r["v"], moment_dtype=MK[dt], step=t, m_scale=r["ms"],
                             v_scale=r["vs"], **HP)
            r.update(W=o["W"], m=o["m"], v=o["v"], ms=o["m_scale"], vs=o["v_scale"])
        for key, r in ss8.items():
            o = oracle.adamw_fp8(G, r["W"], r["m"], r["v"], w_fp8=r["w8"], m_fp8=r["m8"], w_ring=r["wr"],
                                 m_ring=r["mr"], v_ring=r["vr"], step=t, **HP)
            r.update(W=o["W"], m=o["m"], v=o["v"], wr=o["w_ring"], mr=o["m_ring"], vr=o["v_ring"])
        torch.cuda.synchronize()
        _say(f"step {t} done")

    def weight64(k):
        """An arm's W as fp64 values (fp8 weights decoded with the scale they were encoded with)."""
        if arms[k][0] == "wfp8":
            ring = bits(st[k][5])
            scale = np.float32(ring[(STEPS + 3) % 4]) / np.float32(448) if ring[(STEPS + 3) % 4] > 0 else np.float32(1)
            return float(scale) * oracle.e4m3_decode(st[k][0].view(torch.uint8).cpu().numpy())
        return oracle.bf16_bits_to_f64(bits(st[k][0]))

    def ref64(k, dt):
        if k in ss8:
            r = ss8[k]
            if r["w8"]:
                a = r["wr"][(STEPS + 3) % 4]
                scale = np.float32(a) / np.float32(448) if a > 0 else np.float32(1)
                return float(scale) * oracle.e4m3_decode(r["W"])
            return oracle.bf16_bits_to_f64(r["W"])
        return oracle.bf16_bits_to_f64(ss[dt]["W"])

    def metrics64(W64, ref):
        d = W64 - ref
        return dict(rms_rel=float(np.sqrt(np.mean(d * d)) / np.sqrt(np.mean(ref * ref))),
                    max_abs=float(np.abs(d).max()))

    table = {}
    for k, (_, dt, _) in arms.items():
        Wk = weight64(k)
        table[k] = dict(vs_unrounded=metrics64(Wk, Wr), vs_same_storage=metrics64(Wk, ref64(k, dt)))
    # the floor of any bf16-weight arm against the unrounded reference: that reference
    # rounded once to bf16 at the end
    table["unrounded_reference_rounded_once"] = dict(
        vs_unrounded=metrics64(oracle.bf16_bits_to_f64(oracle.f64_to_bf16_bits(Wr)), Wr))
    out = dict(V=V, H=H, BT=BT, steps=STEPS, hyper=HP, arms=table)
    _say(json.dumps(out, indent=1))
    results_dir = os.environ.get("FORGE_RESULTS_DIR")
    if results_dir and os.path.isdir(results_dir):
        with open(os.path.join(results_dir, "fidelity_app_e.json"), "w") as f:
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
    # fp8 arms: reported (a tie decided the other way moves an fp8 weight by a whole E4M3 step,
    # and the free-running trajectories then part); only that they stay finite and bounded
    for k in ("fused_fp8m", "fused_fp8w_bf16m", "fused_fp8w_fp8m"):
        assert np.isfinite(u(k)) and u(k) < 0.2, k
