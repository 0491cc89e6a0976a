"""Helpers shared by the GPU parity tests: seeded problems, a HIP run and an oracle run.

Inputs come from ``paper_2606_22932_amd.synth`` (random numbers only); the oracle never
sees a value produced by the HIP path.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np
import torch

import oracle
from paper_2606_22932_amd import forge, synth

HP = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.1)
MOMENT_CODE = {"f32": oracle.MOMENT_F32, "bf16": oracle.MOMENT_BF16, "i8": oracle.MOMENT_I8,
               "i8r64": oracle.MOMENT_I8_ROW64}


def bits(t: torch.Tensor) -> np.ndarray:
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16).copy()
    return t.numpy().copy()


def dev(a: np.ndarray, device="cuda") -> torch.Tensor:
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(a).copy()).to(device)


@dataclass
class Problem:
    X: np.ndarray
    dY: np.ndarray
    W: np.ndarray
    m: np.ndarray
    v: np.ndarray
    moment: str
    m_scale: np.ndarray = None
    v_scale: np.ndarray = None
    hp: dict = field(default_factory=lambda: dict(HP))

    @property
    def shape(self):
        return self.X.shape[0], self.X.shape[1], self.dY.shape[1]

    def state(self):
        return dict(W=self.W, m=self.m, v=self.v, m_scale=self.m_scale, v_scale=self.v_scale)


def make_problem(T, d_in, d_out, moment, seed, *, warm=True, x_std=1.0, dy_std=1e-3, w_std=0.02,
                 m_std=1e-4, v_std=1e-6):
    base = 1000 * seed
    X = synth.gaussian((T, d_in), x_std, base + 1)
    dY = synth.gaussian((T, d_out), dy_std, base + 11)
    W = synth.gaussian((d_out, d_in), w_std, base + 2)
    if warm:
        m = synth.gaussian((d_out, d_in), m_std, base + 3, dtype=torch.float32)
        v = synth.gaussian((d_out, d_in), v_std, base + 4, dtype=torch.float32, absolute=True)
    else:
        m = torch.zeros((d_out, d_in), dtype=torch.float32)
        v = torch.zeros((d_out, d_in), dtype=torch.float32)
    p = Problem(bits(X), bits(dY), bits(W), None, None, moment)
    if moment == "f32":
        p.m, p.v = bits(m), bits(v)
    elif moment == "bf16":
        p.m, p.v = bits(m.to(torch.bfloat16)), bits(v.to(torch.bfloat16))
    elif moment == "i8":
        p.m, p.m_scale = oracle.quantize_i8(m.double().numpy(), second_moment=False)
        p.v, p.v_scale = oracle.quantize_i8(v.double().numpy(), second_moment=True)
    else:
        p.m, p.m_scale = oracle.quantize_i8_row64(m.double().numpy(), second_moment=False)
        p.v, p.v_scale = oracle.quantize_i8_row64(v.double().numpy(), second_moment=True)
    return p


def with_state(p: Problem, st: dict, dY=None) -> Problem:
    q = Problem(p.X, p.dY if dY is None else dY, st["W"], st["m"], st["v"], p.moment,
                st.get("m_scale"), st.get("v_scale"), dict(p.hp))
    return q


def gemm_error_bound(X: np.ndarray, dY: np.ndarray) -> np.ndarray:
    """Bound on the fp32 accumulation error of any summation order of G: T 2^-24 |dY|^T |X|.

    (A numpy product of absolute values, used only as an error scale.)"""
    T = X.shape[0]
    ax = np.abs(oracle.bf16_bits_to_f64(X))
    ay = np.abs(oracle.bf16_bits_to_f64(dY))
    return T * 2.0 ** -24 * (ay.T @ ax)


def run_oracle(p: Problem, step: int, round_grad_to_bf16=False):
    out = oracle.linear_step(p.X, p.dY, p.W, p.m, p.v, moment_dtype=MOMENT_CODE[p.moment], step=step,
                             m_scale=p.m_scale, v_scale=p.v_scale, round_grad_to_bf16=round_grad_to_bf16,
                             want_quotients=True, **p.hp)
    out["EG"] = gemm_error_bound(p.X, p.dY)
    return out


def run_gpu(p: Problem, step: int, *, path="fused", grad="f32"):
    """One step through the C ABI on cuda:0; returns the new state on the host."""
    X, dY, W, m, v = (dev(a) for a in (p.X, p.dY, p.W, p.m, p.v))
    ms = dev(p.m_scale) if p.m_scale is not None else None
    vs = dev(p.v_scale) if p.v_scale is not None else None
    X0, dY0 = X.clone(), dY.clone()
    if path == "fused":
        forge.forge_linear_step(X, dY, W, m, v, ms, vs, step=step, **p.hp)
    else:
        G = torch.empty(W.shape, dtype=torch.float32 if grad == "f32" else torch.bfloat16, device=W.device)
        forge.forge_linear_step_unfused(X, dY, W, m, v, ms, vs, G_ws=G, step=step, **p.hp)
    torch.cuda.synchronize()
    assert torch.equal(X, X0) and torch.equal(dY, dY0), "X / dY were modified"
    out = dict(W=bits(W), m=bits(m), v=bits(v))
    if ms is not None:
        out.update(m_scale=bits(ms), v_scale=bits(vs))
    return out
