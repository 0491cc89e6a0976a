"""Algorithmic HBM bytes and flops of one step (what the method must move and compute).

Sec. 2.2, "Memory and bandwidth": a step reads and writes the weight and both moments
once; the conventional two-kernel step also writes the gradient and reads it back.  The
weight-gradient GEMM reads X and dY once and costs 2*T flops per parameter.
"""
from __future__ import annotations

MOMENT_BYTES = {"f32": 4, "bf16": 2, "i8": 1, "i8r64": 1, "fp8": 1}
WEIGHT_BYTES = {"bf16": 2, "fp8": 1}
GRAD_BYTES = {"bf16": 2, "f32": 4}
I8_BLOCK = 256          # rows of d_out per scale, 256-row column layout
I8_ROW_BLOCK = 64       # elements of a row per scale, 64-wide row layout


def state_bytes_per_param(moment: str, weight: str = "bf16") -> float:
    """Bytes of W and m, v moved per parameter by a step: each read once and written once."""
    return 2 * (WEIGHT_BYTES[weight] + 2 * MOMENT_BYTES[moment])


def fused_bytes(T: int, d_in: int, d_out: int, moment: str, weight: str = "bf16") -> int:
    """fp8 tensors' per-tensor amax rings (16 bytes each) are not counted."""
    P = d_in * d_out
    b = P * state_bytes_per_param(moment, weight) + 2 * T * (d_in + d_out)
    if moment == "i8":
        nblk = (d_out + I8_BLOCK - 1) // I8_BLOCK
        b += 2 * 2 * 4 * nblk * d_in          # two fp32 scale tensors, read and written
    elif moment == "i8r64":
        b += 2 * 2 * 4 * d_out * ((d_in + I8_ROW_BLOCK - 1) // I8_ROW_BLOCK)
    return int(b)


def unfused_bytes(T: int, d_in: int, d_out: int, moment: str, grad: str = "bf16") -> int:
    """The fused bytes plus the gradient's round trip (written by the GEMM, read by the optimizer)."""
    return fused_bytes(T, d_in, d_out, moment) + 2 * GRAD_BYTES[grad] * d_in * d_out


def gemm_flops(T: int, d_in: int, d_out: int) -> int:
    return 2 * T * d_in * d_out
