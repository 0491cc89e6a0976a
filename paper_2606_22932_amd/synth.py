"""Seeded synthetic inputs for the fused weight-gradient + AdamW step.

This module only draws random numbers; it holds none of the method's arithmetic, and
both the GPU path's tests and the CPU oracle take their inputs from it.

Workloads (Llama-3.1-8B linear layers at batch 1, sequence 512, BF16 everywhere, the
setting of the paper's single-GPU experiments, Sec. 3; random data stands in for real
activations and gradients):

* ``layer256``   T=128, 256x256, X~N(0,1), dY~N(0,0.01) (fresh each step), W~N(0,0.02),
                 fp32 moments starting at zero, steps 1..3.
* ``o_proj``     T=512, 4096x4096, X std 1, dY std 1e-3, W std 0.02, bf16 moments from a
                 warm state m~N(0,1e-4), v=|N(0,1e-6)|, step 100.
* ``o_proj_t4096``  ``o_proj`` at T=4096 tokens, where the GEMM (2T flop per parameter)
                 outweighs the state traffic: the compute-bound regime.
* ``mlp``        T=512, gate/up [14336x4096], down [4096x14336], as ``o_proj``.
* ``mlp_i8``     ``mlp`` with int8 block-absmax moments (256-row column blocks, sqrt(v)).
* ``mlp_i8r64``  ``mlp`` with int8 moments in 64-wide row blocks (v stored).
* ``mlp_fp8``, ``mlp_wfp8``, ``mlp_wfp8_fp8``  ``mlp`` with fp8 E4M3 moments (m and sqrt(v)),
                 fp8 E4M3 weights with bf16 moments, and both (per-tensor delayed scales).
* ``sweep``      32 decoder layers x {q,k,v,o,gate,up,down} + lm_head [128256x4096], bf16 moments.

"N(0, s)" means standard deviation s.  Per-tensor seeds are ``1000*base + id`` with ids
X=1, W=2, m=3, v=4 and dY at step t = 10+t.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import torch

ID_X, ID_W, ID_M, ID_V = 1, 2, 3, 4


def seed_of(base: int, ident: int) -> int:
    return 1000 * base + ident


def gaussian(shape, std: float, seed: int, *, device="cpu", dtype=torch.bfloat16, absolute=False):
    """std * N(0,1) drawn in fp32 from a seeded torch generator, then cast (RNE) to ``dtype``."""
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    x = torch.randn(tuple(shape), generator=g, device=device, dtype=torch.float32)
    x.mul_(std)
    if absolute:
        x.abs_()
    return x.to(dtype)


@dataclass(frozen=True)
class Matrix:
    """One linear layer's weight-gradient problem: W is [d_out, d_in], X [T, d_in], dY [T, d_out]."""
    name: str
    d_out: int
    d_in: int
    base: int


@dataclass(frozen=True)
class Workload:
    name: str
    T: int
    matrices: tuple
    moment: str                  # "f32" | "bf16" | "i8" | "i8r64" | "fp8"
    x_std: float = 1.0
    dy_std: float = 1e-3
    w_std: float = 0.02
    m_std: float = 1e-4          # warm first moment (0 -> cold start at zero)
    v_std: float = 1e-6          # warm second moment |N(0, v_std)|
    steps: tuple = (100,)
    weight: str = "bf16"         # "bf16" | "fp8"
    hyper: dict = field(default_factory=lambda: dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8,
                                                     weight_decay=0.1))


LLAMA8B_PROJ = (("q", 4096, 4096), ("k", 1024, 4096), ("v", 1024, 4096), ("o", 4096, 4096),
                ("gate", 14336, 4096), ("up", 14336, 4096), ("down", 4096, 14336))
LM_HEAD = ("lm_head", 128256, 4096)


def _sweep_matrices():
    mats = []
    for layer in range(32):
        for j, (nm, do, di) in enumerate(LLAMA8B_PROJ):
            mats.append(Matrix(f"L{layer}.{nm}", do, di, 100 + 8 * layer + j))
    mats.append(Matrix(LM_HEAD[0], LM_HEAD[1], LM_HEAD[2], 100 + 8 * 32))
    return tuple(mats)


def launch_groups(wl: "Workload", schedule: str = "backward"):
    """Indices into ``wl.matrices`` per fused launch, in the order a backward pass makes
    the weight gradients available.

    For the sweep: lm_head first, then each decoder layer from the last to the first as
    [down], [gate, up], [o], [q, k, v] -- gate and up (and q, k, v) read the same input and
    receive their upstream gradients together, so one grouped launch steps them.  Other
    workloads: one matrix per launch.
    """
    if wl.name != "sweep":
        return [[i] for i in range(len(wl.matrices))]
    per = len(LLAMA8B_PROJ)
    idx = {nm: j for j, (nm, _, _) in enumerate(LLAMA8B_PROJ)}
    groups = [[32 * per]]
    if schedule == "layer":
        # one launch per decoder layer, last layer first: the layer's input gradients are
        # formed first (each from its pre-update weight), then its seven weights are stepped
        return groups + [[layer * per + j for j in range(per)] for layer in reversed(range(32))]
    for layer in reversed(range(32)):
        b = layer * per
        groups += [[b + idx["down"]], [b + idx["gate"], b + idx["up"]], [b + idx["o"]],
                   [b + idx["q"], b + idx["k"], b + idx["v"]]]
    return groups


WORKLOADS = {
    "layer256": Workload("layer256", 128, (Matrix("layer256", 256, 256, 0),), "f32",
                         x_std=1.0, dy_std=0.01, m_std=0.0, v_std=0.0, steps=(1, 2, 3)),
    "o_proj": Workload("o_proj", 512, (Matrix("o_proj", 4096, 4096, 2),), "bf16"),
    "o_proj_t4096": Workload("o_proj_t4096", 4096, (Matrix("o_proj", 4096, 4096, 2),), "bf16"),
    "mlp": Workload("mlp", 512, (Matrix("gate", 14336, 4096, 3), Matrix("up", 14336, 4096, 4),
                                 Matrix("down", 4096, 14336, 5)), "bf16"),
    "mlp_i8": Workload("mlp_i8", 512, (Matrix("gate", 14336, 4096, 6), Matrix("up", 14336, 4096, 7),
                                       Matrix("down", 4096, 14336, 8)), "i8"),
    "mlp_i8r64": Workload("mlp_i8r64", 512, (Matrix("gate", 14336, 4096, 6), Matrix("up", 14336, 4096, 7),
                                             Matrix("down", 4096, 14336, 8)), "i8r64"),
    "mlp_fp8": Workload("mlp_fp8", 512, (Matrix("gate", 14336, 4096, 6), Matrix("up", 14336, 4096, 7),
                                         Matrix("down", 4096, 14336, 8)), "fp8"),
    "mlp_wfp8": Workload("mlp_wfp8", 512, (Matrix("gate", 14336, 4096, 6), Matrix("up", 14336, 4096, 7),
                                           Matrix("down", 4096, 14336, 8)), "bf16", weight="fp8"),
    "mlp_wfp8_fp8": Workload("mlp_wfp8_fp8", 512, (Matrix("gate", 14336, 4096, 6), Matrix("up", 14336, 4096, 7),
                                                   Matrix("down", 4096, 14336, 8)), "fp8", weight="fp8"),
    "sweep": Workload("sweep", 512, _sweep_matrices(), "bf16"),
}


def activations(T, mat: Matrix, wl: Workload, step: int, device="cpu"):
    """X [T, d_in] and dY [T, d_out] (bf16) for ``mat`` at optimizer step ``step``."""
    X = gaussian((T, mat.d_in), wl.x_std, seed_of(mat.base, ID_X), device=device)
    dY = gaussian((T, mat.d_out), wl.dy_std, seed_of(mat.base, 10 + step), device=device)
    return X, dY


def weight(mat: Matrix, wl: Workload, device="cpu"):
    return gaussian((mat.d_out, mat.d_in), wl.w_std, seed_of(mat.base, ID_W), device=device)


def warm_moments(mat: Matrix, wl: Workload, device="cpu", dtype=torch.float32):
    """First/second moment draws (zeros for a cold start); int8 callers quantize these themselves."""
    shape = (mat.d_out, mat.d_in)
    if wl.m_std == 0.0:
        return (torch.zeros(shape, device=device, dtype=dtype),
                torch.zeros(shape, device=device, dtype=dtype))
    m = gaussian(shape, wl.m_std, seed_of(mat.base, ID_M), device=device, dtype=dtype)
    v = gaussian(shape, wl.v_std, seed_of(mat.base, ID_V), device=device, dtype=dtype, absolute=True)
    return m, v


def random_i8_state(mat: Matrix, wl: Workload, device="cpu", layout="col256"):
    """Random int8 moment codes and positive fp32 scales of warm-state magnitude.

    Used where only the cost of a step matters (timing): the codes are uniform, m in
    [-127, 127] and the second-moment code in [1, 127]; scales are m_std*3/127 and, for the
    256-row column layout (which stores sqrt(v)), sqrt(v_std)*3/127, for the 64-wide row
    layout (which stores v) v_std*3/127.  Scales are [ceil(d_out/256), d_in] (col256) or
    [d_out, ceil(d_in/64)] (row64).
    """
    g = torch.Generator(device=device)
    g.manual_seed(seed_of(mat.base, 5))
    shape = (mat.d_out, mat.d_in)
    mq = torch.randint(-127, 128, shape, generator=g, device=device, dtype=torch.int8)
    vq = torch.randint(1, 128, shape, generator=g, device=device, dtype=torch.int8)
    if layout == "col256":
        sshape = ((mat.d_out + 255) // 256, mat.d_in)
        v_scale = (wl.v_std ** 0.5) * 3 / 127
    else:
        sshape = (mat.d_out, (mat.d_in + 63) // 64)
        v_scale = wl.v_std * 3 / 127
    ms = torch.full(sshape, wl.m_std * 3 / 127, device=device, dtype=torch.float32)
    vs = torch.full(sshape, v_scale, device=device, dtype=torch.float32)
    return mq, vq, ms, vs


def random_fp8_codes(shape, seed: int, *, signed: bool, device="cpu"):
    """Uniform random E4M3 codes (float8_e4m3fn) over the finite values: magnitude bytes
    0x00-0x7E (0x7F is NaN), with a random sign when ``signed``."""
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    b = torch.randint(0, 0x7F, tuple(shape), generator=g, device=device, dtype=torch.int32)
    if signed:
        b |= torch.randint(0, 2, tuple(shape), generator=g, device=device, dtype=torch.int32) << 7
    return b.to(torch.uint8).view(torch.float8_e4m3fn)


def random_fp8_state(mat: Matrix, wl: Workload, device="cpu"):
    """Random fp8 state for timing: E4M3 codes of W (fp8 weights) and of m and sqrt(v) (fp8
    moments), each with an amax ring of 4 float32 slots filled with 3 standard deviations
    of the tensor's warm magnitude (w_std, m_std, sqrt(v_std)).  Returns (W, w_ring, m,
    m_ring, v, v_ring); the entries of the parts in bf16 are None."""
    shape = (mat.d_out, mat.d_in)
    ring = lambda a: torch.full((4,), float(a), device=device, dtype=torch.float32)
    W = w_ring = m = m_ring = v = v_ring = None
    if wl.weight == "fp8":
        W = random_fp8_codes(shape, seed_of(mat.base, 7), signed=True, device=device)
        w_ring = ring(3 * wl.w_std)
    if wl.moment == "fp8":
        m = random_fp8_codes(shape, seed_of(mat.base, 8), signed=True, device=device)
        v = random_fp8_codes(shape, seed_of(mat.base, 9), signed=False, device=device)
        m_ring, v_ring = ring(3 * wl.m_std), ring(3 * wl.v_std ** 0.5)
    return W, w_ring, m, m_ring, v, v_ring


def bf16_bits(t: torch.Tensor):
    """A CPU bf16 tensor as a numpy uint16 array of its bit patterns."""
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view("uint16")


def from_bf16_bits(a, device="cpu"):
    import numpy as np
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(device)
